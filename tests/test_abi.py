"""C ABI contract on the CPU: the library loads, exports every function the
header declares, sizes workspaces as pure functions, and rejects bad
arguments before any HIP call (so these calls never touch a device)."""
import ctypes

import pytest

from paper_2608_02474_amd import _lib

FAKE = ctypes.c_void_p(0x10000)        # 16-byte aligned host-side stand-in, never dereferenced
MISALIGNED = ctypes.c_void_p(0x10004)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_every_header_function_is_exported(lib):
    names = _lib.header_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib._SIGNATURES)


def test_status_strings_and_version(lib):
    for s in range(5):
        assert lib.echo_status_str(s)
    assert lib.echo_status_str(99) == b"unknown status"
    assert lib.echo_version().decode().count(".") == 2
    assert lib.echo_last_hip_error() == 0


def test_workspace_queries(lib):
    e = _lib.EnergyCfg(21, 16000, 512, 160, 8)
    ws = lib.echo_energy_workspace(ctypes.byref(e), 81000)
    assert ws >= 21 * 21 * 8 * 8
    assert lib.echo_energy_workspace(ctypes.byref(_lib.EnergyCfg(0, 16000, 512, 160, 8)), 81000) == 0
    s = _lib.SelectCfg(21, 1560, 5120, _lib.ECHO_BF16, 13104, 0.0, 1e-6)
    assert lib.echo_select_workspace(ctypes.byref(s)) >= 32760 * 20
    b = _lib.BlockCfg(32760, 5120, 40, 13824, _lib.ECHO_BF16, 1e-6)
    w0 = lib.echo_block_workspace(ctypes.byref(b), 0)
    w1 = lib.echo_block_workspace(ctypes.byref(b), 13104)
    assert w0 >= 32760 * 5120 * 2 * 3                   # LN output + K/V for all rows
    assert w1 - w0 >= 13104 * (5120 * 2 * 3 + 5120 * 4 + 13824 * 2)
    assert lib.echo_block_workspace(ctypes.byref(b), -1) == 0


def test_energy_rejects_before_launch(lib):
    good = _lib.EnergyCfg(2, 16000, 512, 160, 8)
    run = lambda cfg, n=8000, ws=FAKE, wsb=1 << 20, a=FAKE: lib.echo_energy(
        ctypes.byref(cfg) if cfg else None, a, n, FAKE, FAKE, FAKE, ws, wsb, None)
    assert run(None) == _lib.ECHO_EINVAL
    assert run(_lib.EnergyCfg(2, 16000, 511, 160, 8)) == _lib.ECHO_EINVAL   # odd n_fft
    assert run(_lib.EnergyCfg(2, 16000, 512, 0, 8)) == _lib.ECHO_EINVAL     # hop 0
    assert run(good, n=1) == _lib.ECHO_EINVAL                                # fewer samples than T
    assert run(good, a=None) == _lib.ECHO_EINVAL
    assert run(good, a=MISALIGNED) == _lib.ECHO_EINVAL
    assert run(good, wsb=8) == _lib.ECHO_EWORKSPACE
    assert run(good, ws=None) == _lib.ECHO_EWORKSPACE


def test_select_rejects_before_launch(lib):
    def run(cfg, x=FAKE, wsb=1 << 30):
        return lib.echo_select(ctypes.byref(cfg), x, FAKE, FAKE, FAKE, FAKE, FAKE, None, None,
                               FAKE, wsb, None)
    assert run(_lib.SelectCfg(2, 16, 64, 0, 33, 0.0, 1e-6)) == _lib.ECHO_EINVAL     # k > L
    assert run(_lib.SelectCfg(2, 16, 60, 0, 3, 0.0, 1e-6)) == _lib.ECHO_EINVAL      # D % 8
    assert run(_lib.SelectCfg(2, 16, 64, 7, 3, 0.0, 1e-6)) == _lib.ECHO_EINVAL      # dtype
    assert run(_lib.SelectCfg(2, 16, 64, 0, 3, 0.0, -1.0)) == _lib.ECHO_EINVAL      # xi < 0
    assert run(_lib.SelectCfg(2, 16, 64, 0, -1, float("nan"), 1e-6)) == _lib.ECHO_EINVAL
    assert run(_lib.SelectCfg(2, 16, 64, 0, 3, 0.0, 1e-6), x=MISALIGNED) == _lib.ECHO_EINVAL
    assert run(_lib.SelectCfg(2, 16, 64, 0, 3, 0.0, 1e-6), wsb=16) == _lib.ECHO_EWORKSPACE


def test_select_noalloc_rejects_before_launch(lib):
    def run(cfg, x=FAKE):
        return lib.echo_select_noalloc(ctypes.byref(cfg), x, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None)
    lim = _lib.ECHO_SELECT_NOALLOC_MAX_TOKENS
    assert run(_lib.SelectCfg(2, lim // 2 + 1, 64, 0, 3, 0.0, 1e-6)) == _lib.ECHO_ELIMIT
    assert run(_lib.SelectCfg(1, lim + 1, 64, 1, 3, 0.0, 1e-6)) == _lib.ECHO_ELIMIT
    assert run(_lib.SelectCfg(2, 16, 64, 0, 33, 0.0, 1e-6)) == _lib.ECHO_EINVAL     # k > L
    assert run(_lib.SelectCfg(2, 16, 64, 0, 3, 0.0, 1e-6), x=MISALIGNED) == _lib.ECHO_EINVAL
    assert lib.echo_status_str(_lib.ECHO_ELIMIT) == b"size above the allocation-free limit"


def test_mfma_ceiling_rejects_before_launch(lib):
    out = ctypes.c_double(-1.0)
    run = lambda pat, dat, secs, o=ctypes.byref(out): lib.echo_mfma_ceiling(pat, dat, secs, o, None)
    assert run(2, 1, 1.0) == _lib.ECHO_EINVAL                    # unknown pattern
    assert run(0, 2, 1.0) == _lib.ECHO_EINVAL                    # unknown data kind
    assert run(1, 1, 0.0) == _lib.ECHO_EINVAL                    # no time
    assert run(1, 1, 61.0) == _lib.ECHO_EINVAL                   # above the limit
    assert run(0, 0, float("nan")) == _lib.ECHO_EINVAL
    assert run(0, 1, 1.0, None) == _lib.ECHO_EINVAL              # no output
    assert out.value == -1.0


def test_block_rejects_before_launch(lib):
    w = _lib.BlockWeights(*([0x20000] * 13))
    def run(cfg, n=4, wsb=1 << 40, weights=w):
        return lib.echo_block_partial(ctypes.byref(cfg), ctypes.byref(weights), FAKE, FAKE, n,
                                      FAKE, FAKE, wsb, None)
    bf = _lib.ECHO_BF16
    assert run(_lib.BlockCfg(32, 64, 3, 256, 0, 1e-6)) == _lib.ECHO_EINVAL           # D % H
    assert run(_lib.BlockCfg(32, 256, 4, 512, bf, 1e-6)) == _lib.ECHO_EUNSUPPORTED   # dh 64 on bf16
    assert run(_lib.BlockCfg(32, 384, 3, 512, bf, 1e-6)) == _lib.ECHO_EUNSUPPORTED   # D % 256
    assert run(_lib.BlockCfg(32, 1024, 4, 512, 0, 1e-6)) == _lib.ECHO_EUNSUPPORTED   # fp32 dh 256
    assert run(_lib.BlockCfg(32, 256, 2, 512, bf, 1e-6), n=-1) == _lib.ECHO_EINVAL
    assert run(_lib.BlockCfg(32, 256, 2, 512, bf, 1e-6), wsb=64) == _lib.ECHO_EWORKSPACE
    bad = _lib.BlockWeights(*([0x20000] * 12 + [0x20008]))                            # misaligned mod
    assert run(_lib.BlockCfg(32, 256, 2, 512, bf, 1e-6), weights=bad) == _lib.ECHO_EINVAL
    assert run(_lib.BlockCfg(32, 256, 2, 512, bf, 1e-6, 2)) == _lib.ECHO_EINVAL      # unknown flag
    # n_sel == 0 is a successful no-op that launches nothing
    assert run(_lib.BlockCfg(32, 256, 2, 512, bf, 1e-6), n=0) == _lib.ECHO_OK


def test_cache_rejects_before_launch(lib):
    def run(cfg, n=4, y=FAKE):
        return lib.echo_cache_update(ctypes.byref(cfg), FAKE, FAKE, FAKE, n, FAKE, FAKE, FAKE,
                                     FAKE, y, None)
    assert run(_lib.CacheCfg(32, 60, 0)) == _lib.ECHO_EINVAL
    assert run(_lib.CacheCfg(32, 64, 0), n=33) == _lib.ECHO_EINVAL
    assert run(_lib.CacheCfg(32, 64, 0), y=None) == _lib.ECHO_EINVAL
    assert run(_lib.CacheCfg(32, 64, 2)) == _lib.ECHO_EINVAL


def test_profile_read_empty(lib):
    arr = (_lib.KernelTime * 4)()
    assert lib.echo_profile_read(arr, 4) == 0
    assert lib.echo_profile_read(None, -1) == -_lib.ECHO_EINVAL


def test_refcache_rejects_before_launch(lib):
    st = _lib.RefCacheState(*([0x20000] * 9))
    def run(cfg, n=4, state=st, x=FAKE):
        return lib.echo_refcache_update(ctypes.byref(cfg), ctypes.byref(state), x, FAKE, FAKE, n,
                                        FAKE, FAKE, FAKE, None)
    ok = _lib.RefCacheCfg(40, 64, 0, 8, 45, 0.5)
    assert run(_lib.RefCacheCfg(40, 64, 0, 7, 46, 0.5)) == _lib.ECHO_EINVAL            # L % chain_len
    assert run(_lib.RefCacheCfg(40, 64, 0, 8, 44, 0.5)) == _lib.ECHO_EINVAL            # capacity < L + chains
    assert run(_lib.RefCacheCfg(40, 60, 0, 8, 45, 0.5)) == _lib.ECHO_EINVAL            # D % 8
    assert run(_lib.RefCacheCfg(40, 64, 0, 8, 45, float("nan"))) == _lib.ECHO_EINVAL   # tau
    assert run(_lib.RefCacheCfg(40, 64, 5, 8, 45, 0.5)) == _lib.ECHO_EINVAL            # dtype
    assert run(ok, n=41) == _lib.ECHO_EINVAL
    assert run(ok, x=MISALIGNED) == _lib.ECHO_EINVAL
    bad = _lib.RefCacheState(*([0x20000] * 8 + [0]))                                   # null scale
    assert run(ok, state=bad) == _lib.ECHO_EINVAL
    assert lib.echo_refcache_init(ctypes.byref(_lib.RefCacheCfg(40, 64, 0, 8, 44, 0.5)),
                                  ctypes.byref(st), None) == _lib.ECHO_EINVAL


def test_anchors_and_segments_reject_before_launch(lib):
    def anc(keys=FAKE, T=21, k=7, mode=_lib.ECHO_ANCHOR_TOPK, out=FAKE):
        return lib.echo_anchors(keys, T, k, mode, out, None)
    assert anc(T=0, k=0) == _lib.ECHO_EINVAL
    assert anc(T=4097, k=1) == _lib.ECHO_EINVAL
    assert anc(k=22) == _lib.ECHO_EINVAL
    assert anc(k=-1) == _lib.ECHO_EINVAL
    assert anc(mode=2) == _lib.ECHO_EINVAL
    assert anc(keys=None) == _lib.ECHO_EINVAL                   # top-k needs keys
    assert anc(keys=MISALIGNED) == _lib.ECHO_EINVAL
    assert anc(out=None, mode=_lib.ECHO_ANCHOR_UNIFORM) == _lib.ECHO_EINVAL

    def seg(s=FAKE, T=21, N=1560, k=10, idx=FAKE, n=FAKE):
        return lib.echo_topk_segments(s, FAKE, T, N, k, idx, FAKE, n, None)
    assert seg(T=0) == _lib.ECHO_EINVAL
    assert seg(N=0) == _lib.ECHO_EINVAL
    assert seg(k=-1) == _lib.ECHO_EINVAL
    assert seg(T=65535, N=40000) == _lib.ECHO_EINVAL            # T * N >= 2^31
    assert seg(s=MISALIGNED) == _lib.ECHO_EINVAL
    assert seg(n=None) == _lib.ECHO_EINVAL


def test_cache_codec_rejects_before_launch(lib):
    def run(codec, store=FAKE, codes=FAKE, scale=FAKE, cfg=_lib.CacheCfg(32, 64, 1), n=4):
        return lib.echo_cache_update_codec(ctypes.byref(cfg), codec, FAKE, FAKE, FAKE, n, FAKE, FAKE,
                                           store, codes, scale, FAKE, None)
    assert run(3) == _lib.ECHO_EINVAL
    assert run(_lib.ECHO_CODEC_FULL, store=None) == _lib.ECHO_EINVAL
    assert run(_lib.ECHO_CODEC_NAIVE_INT8, codes=None) == _lib.ECHO_EINVAL
    assert run(_lib.ECHO_CODEC_RESIDUAL_INT8, scale=MISALIGNED) == _lib.ECHO_EINVAL
    assert run(_lib.ECHO_CODEC_FULL, cfg=_lib.CacheCfg(32, 60, 1)) == _lib.ECHO_EINVAL
    assert run(_lib.ECHO_CODEC_FULL, n=33) == _lib.ECHO_EINVAL


def test_wan_block_rejects_before_launch(lib):
    w = _lib.WanBlockWeights(_lib.BlockWeights(*([0x20000] * 13)), *([0x20000] * 14))
    counts = (ctypes.c_int32 * 2)(10, 12)

    def run(cfg, weights=w, n=counts, x=FAKE):
        return lib.echo_wan_block_partial(ctypes.byref(cfg), ctypes.byref(weights), x, FAKE, FAKE, n, FAKE,
                                          FAKE, 1 << 40, None)

    def cfg(**kw):
        base = dict(B=2, L=300, D=256, H=2, F=512, Lc=77, T=3, gh=10, gw=10, dtype=1, ln_eps=1e-6,
                    rms_eps=1e-6, rope_base=1e4, flags=0)
        base.update(kw)
        return _lib.WanBlockCfg(**base)
    assert run(cfg(gw=11)) == _lib.ECHO_EINVAL                     # T * gh * gw != L
    assert run(cfg(Lc=0)) == _lib.ECHO_EINVAL
    assert run(cfg(rope_base=float("nan"))) == _lib.ECHO_EINVAL
    assert run(cfg(flags=2)) == _lib.ECHO_EINVAL
    assert run(cfg(dtype=0)) == _lib.ECHO_EUNSUPPORTED              # bf16 only
    assert run(cfg(D=192, H=2)) == _lib.ECHO_EUNSUPPORTED           # head width 96
    assert run(cfg(), n=(ctypes.c_int32 * 2)(10, 301)) == _lib.ECHO_EINVAL
    assert run(cfg(), x=MISALIGNED) == _lib.ECHO_EINVAL
    bad = _lib.WanBlockWeights(_lib.BlockWeights(*([0x20000] * 13)), *([0x20000] * 13 + [0]))   # null b3
    assert run(cfg(), weights=bad) == _lib.ECHO_EINVAL
    assert lib.echo_wan_block_workspace(ctypes.byref(cfg()), 100) > 0
    assert lib.echo_wan_block_workspace(ctypes.byref(cfg(T=2)), 100) == 0
