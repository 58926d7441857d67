"""GPU parity: every C-ABI call against the CPU oracle on the same seeded
inputs, at sizes the oracle finishes in seconds (element by element) and at
the full 32760- and 75600-token block shapes (sampled rows the oracle computes
one by one, plus properties that hold at any size)."""
import numpy as np
import pytest
import torch

import synth
from oracle import block as OB
from oracle import cache as OC
from oracle import energy as OE
from oracle import select as OS
from oracle import step as OST
from paper_2608_02474_amd import api

from gpu_util import (check_block, check_selection, device, down, params_to_device, say, tdtype,
                      up, TOL_BF16_ABS, TOL_BF16_REL_L2, TOL_F32_ABS)

pytestmark = pytest.mark.gpu

# a small bf16 shape that is ragged against every tile size (GEMM 256, attention 128/64)
RAGGED = synth.Workload("ragged_bf16_300tok", T=3, grid=(10, 10), D=256, H=2, F=512,
                        n_samples=4000, ratio=0.37, dtype="bf16", audio="bursts", seed=21)
RAGGED_F32 = RAGGED.with_(name="ragged_f32_300tok", dtype="f32", H=4, seed=22)


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


# ------------------------------------------------------------------- energy

@pytest.mark.parametrize("profile,n,T", [
    ("bursts", 8000, 2), ("bursts", 20000, 5), ("speech", 81000, 21), ("noise", 81000, 21),
    ("half_silence", 81000, 21), ("speech", 1000, 3), ("speech", 4000, 1)])
def test_energy_matches_oracle(profile, n, T):
    say(f"energy {profile} n={n} T={T}")
    audio = synth.make_audio(profile, n, 16000, seed=11)
    Eb, e, w = OE.energy(audio, T)
    gb, ge, gw = api.energy(up(audio), T)
    torch.cuda.synchronize()
    gb, ge, gw = down(gb), down(ge), down(gw)
    for got, want, name in ((gb, Eb, "band"), (ge, e, "frame"), (gw, w, "weight")):
        err = np.abs(got.astype(np.float64) - want)
        assert (err <= 1e-6 * np.abs(want.astype(np.float64))).all(), (name, float(err.max()))
    if profile == "half_silence":
        assert (ge[: T // 2] == 0).all()


@pytest.mark.parametrize("n_fft,hop,bands", [(514, 160, 8), (256, 100, 6), (2048, 512, 16), (18, 7, 3)])
def test_energy_other_stft_sizes(n_fft, hop, bands):
    """Window lengths that are not a multiple of 4 (the DFT's four-way
    unrolled sum then has a two-term tail), short and long windows."""
    say(f"energy n_fft={n_fft} hop={hop} bands={bands}")
    audio = synth.make_audio("speech", 20000, 16000, seed=12)
    Eb, e, w = OE.energy(audio, 5, 16000, n_fft, hop, bands)
    gb, ge, gw = api.energy(up(audio), 5, 16000, n_fft, hop, bands)
    torch.cuda.synchronize()
    for got, want, name in ((down(gb), Eb, "band"), (down(ge), e, "frame"), (down(gw), w, "weight")):
        err = np.abs(got.astype(np.float64) - want)
        assert (err <= 1e-6 * np.abs(want.astype(np.float64))).all(), (name, float(err.max()))


# ------------------------------------------------------------------- select

def _frame_weight(w, profile=None):
    audio = synth.make_audio(profile or w.audio, w.n_samples, 16000, w.seed)
    return OE.energy(audio, w.T)[2]


def _select_case(w, ks, fw=None, profile=None):
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w, profile) if fw is None else fw
    s, num, den = OS.saliency(x, xref, fw, w.N)
    dt = tdtype(w.dtype)
    X, XR, FW = up(x, dt), up(xref, dt), up(fw)
    for K in ks:
        say(f"select {w.name} profile={profile or w.audio} K={K}")
        sel = api.select(X, XR, FW, w.N, k=K)
        torch.cuda.synchronize()
        gs = down(sel.saliency)
        assert (np.abs(gs.astype(np.float64) - s) <= 1e-6 * np.abs(s.astype(np.float64))).all()
        gi = down(sel.idx)[:K]
        nd = check_selection(gi, OS.select_topk(s, K), s, K) if K else 0
        if K == 0:
            assert len(gi) == 0
        m = down(sel.mask)
        assert m.sum() == K and (m[gi] == 1).all()
        assert int(down(sel.n_sel_dev)[0]) == K
        sd = float(down(sel.step_delta)[0])
        assert sd == pytest.approx(OS.step_delta(num, den), rel=1e-12)
        say(f"  ok ({nd} tie-excluded differences)")
    return s, X, XR, FW


def test_select_tiny_f32():
    w = synth.TINY
    _select_case(w, [0, 1, w.K, w.L - 1, w.L])


def test_select_ragged_with_ties():
    # frame weights with zeros: exact zero-saliency ties resolved by index
    w = RAGGED_F32
    fw = np.array([0.0, 0.6, 0.0], np.float32)
    _select_case(w, [0, 1, 99, 100, 101, 150, 299, 300], fw=fw)


def test_select_small_bf16():
    w = synth.SMALL
    _select_case(w, [w.K, 1, w.L])


def test_select_threshold_mode():
    w = synth.SMALL
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w)
    s, _, _ = OS.saliency(x, xref, fw, w.N)
    dt = tdtype(w.dtype)
    for th in (float(np.median(s)), float(np.quantile(s, 0.9)), 0.0, 1e9):
        sel = api.select(up(x, dt), up(xref, dt), up(fw), w.N, threshold=th)
        torch.cuda.synchronize()
        n = sel.count()
        want = OS.select_threshold(s, th)
        got = down(sel.idx)[:n]
        # identical saliencies (checked above to 1e-6) decide identically except at the threshold
        diff = set(got.tolist()) ^ set(want.tolist())
        for i in diff:
            assert abs(float(s[i]) - th) <= 1e-6 * max(abs(th), 1e-30)
        assert list(got) == sorted(got)


@pytest.mark.parametrize("profile", synth.SWEEP_AUDIO)
def test_select_14b_shape_sweep(profile):
    w = synth.WAN14B_480P.with_(audio=profile, seed=3)
    ks = [synth.WAN14B_480P.with_(ratio=r).K for r in synth.SWEEP_RATIOS] + [w.K]
    _select_case(w, ks)


def test_select_720p_shape():
    w = synth.WAN14B_720P
    _select_case(w, [w.K])


@pytest.mark.parametrize("grid", [(64, 64), (60, 64)], ids=["81920tok", "96000tok"])
def test_select_register_limit(grid):
    # 81920 keys is the most the register-resident selection holds (80 per
    # thread); 96000 takes the variant that re-reads the keys on every pass
    w = synth.TINY.with_(name=f"select_{grid[0]}x{grid[1]}", T=20 if grid == (64, 64) else 25,
                         grid=grid, ratio=0.3)
    _select_case(w, [1, w.K, w.L - 1, w.L])


# -------------------------------------------------------------------- cache

@pytest.mark.parametrize("w", [synth.TINY, RAGGED, synth.SMALL, synth.WAN14B_480P, synth.WAN14B_720P],
                         ids=lambda w: w.name)
def test_cache_update_bit_exact(w):
    say(f"cache {w.name}")
    xref, x = synth.make_latents(w)
    rng = np.random.default_rng(5)
    L, D, K = w.L, w.D, w.K
    idx = np.sort(rng.choice(L, K, replace=False)).astype(np.int32)
    y_sel = (x[idx] + 0.1 * rng.standard_normal((K, D))).astype(np.float32)
    y_sel[0] = x[idx[0]]                                   # zero residual -> scale 0, codes 0
    y_sel[-1] = x[idx[-1]]
    y_sel[-1, 7] += 3.0                                    # one-hot residual -> +127
    codes0 = rng.integers(-127, 128, (L, D)).astype(np.int8)
    scale0 = rng.uniform(0, 0.02, L).astype(np.float32)
    y_o, xr_o, c_o, s_o = OC.cache_update(x, idx, y_sel, xref, codes0, scale0, w.dtype)
    dt = tdtype(w.dtype)
    XR, C, S = up(xref, dt), up(codes0), up(scale0)
    mask = OS.mask_of(idx, L)
    Y = api.cache_update(up(x, dt), up(idx), up(mask), K, up(y_sel), XR, C, S)
    torch.cuda.synchronize()
    assert np.array_equal(down(C), c_o)
    assert np.array_equal(_bits(down(S)), _bits(s_o))
    assert np.array_equal(_bits(down(XR)), _bits(xr_o))
    assert np.array_equal(_bits(down(Y)), _bits(y_o))
    assert down(S)[idx[0]] == 0 and (down(C)[idx[0]] == 0).all()
    assert down(C)[idx[-1], 7] == 127


def test_cache_update_empty_and_full():
    w = synth.SMALL
    xref, x = synth.make_latents(w)
    rng = np.random.default_rng(6)
    codes0 = rng.integers(-127, 128, (w.L, w.D)).astype(np.int8)
    scale0 = rng.uniform(0, 0.02, w.L).astype(np.float32)
    dt = tdtype(w.dtype)
    # K = 0: output is the dequantized cache everywhere
    y_o, _, _, _ = OC.cache_update(x, np.zeros(0, np.int64), np.zeros((0, w.D), np.float32), xref,
                                   codes0, scale0, w.dtype)
    Y = api.cache_update(up(x, dt), None, up(np.zeros(w.L, np.uint8)), 0, None, up(xref, dt),
                         up(codes0), up(scale0))
    torch.cuda.synchronize()
    assert np.array_equal(_bits(down(Y)), _bits(y_o))
    # K = L: every row fresh
    idx = np.arange(w.L, dtype=np.int32)
    y_sel = (x + 0.05 * rng.standard_normal(x.shape)).astype(np.float32)
    y_o, xr_o, c_o, s_o = OC.cache_update(x, idx, y_sel, xref, codes0, scale0, w.dtype)
    C = up(codes0)
    Y = api.cache_update(up(x, dt), up(idx), up(np.ones(w.L, np.uint8)), w.L, up(y_sel),
                         up(xref, dt), C, up(scale0))
    torch.cuda.synchronize()
    assert np.array_equal(down(C), c_o)
    assert np.array_equal(_bits(down(Y)), _bits(y_o))


# -------------------------------------------------------------------- block

def _block_gpu(w, p, x, idx):
    P = params_to_device(p, w.dtype)
    ys = api.block_partial(P, up(x, tdtype(w.dtype)), up(np.asarray(idx, np.int32)), len(idx), w.H)
    torch.cuda.synchronize()
    return down(ys)


@pytest.mark.parametrize("w", [synth.TINY, RAGGED_F32, RAGGED, synth.SMALL], ids=lambda w: w.name)
def test_block_partial_full_compare(w):
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    rng = np.random.default_rng(7)
    cases = {"topK": np.sort(rng.choice(w.L, w.K, replace=False)),
             "one": np.array([w.L - 1]), "all": np.arange(w.L)}
    if w.L <= 300:
        cases["unsorted_repeats"] = np.array([5, 3, 3, w.L - 1, 0])
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    for name, idx in cases.items():
        say(f"block {w.name} {name} n={len(idx)}")
        got = _block_gpu(w, p, x, idx)
        want = OB.block_partial(p, x, idx, w.H, kv=kv)
        check_block(got, want, w.dtype, f"{w.name}/{name}")


# widths whose second LayerNorm (over fp32 rows) runs one row per workgroup of
# D / 512 waves: the widths the kernel is built for other than 5120 (which the
# full-size tests cover), bf16 and fp32 block
WIDE = [synth.Workload(f"width{D}_{dt}_60tok", T=1, grid=(6, 10), D=D, H=D // 128, F=512,
                       n_samples=4000, ratio=0.5, dtype=dt, audio="bursts", seed=90 + D // 512)
        for D, dt in [(2048, "bf16"), (4096, "bf16"), (2048, "f32")]]


@pytest.mark.parametrize("w", WIDE, ids=lambda w: w.name)
def test_block_partial_ln2_widths(w):
    p = synth.make_block_weights(w)
    _, x = synth.make_latents(w)
    rng = np.random.default_rng(13)
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    for name, idx in {"half": np.sort(rng.choice(w.L, w.L // 2, replace=False)), "one": np.array([w.L - 1])}.items():
        say(f"block {w.name} {name} n={len(idx)}")
        got = _block_gpu(w, p, x, idx)
        want = OB.block_partial(p, x, idx, w.H, kv=kv)
        check_block(got, want, w.dtype, f"{w.name}/{name}")


# bf16 shapes at the edges of the attention tiling: one ragged key tile, exactly
# one tile, one tile plus one key, three tiles, and query sets that cross a
# 384-query workgroup (with the key-split tail of a few items)
EDGE = [synth.Workload(f"edge_bf16_{T * gh * gw}tok", T=T, grid=(gh, gw), D=256, H=2, F=512,
                       n_samples=4000, ratio=0.5, dtype="bf16", audio="bursts", seed=30 + T * gh * gw)
        for T, gh, gw in [(2, 4, 5), (1, 8, 8), (5, 1, 13), (2, 5, 13), (4, 10, 12)]]


@pytest.mark.parametrize("w", EDGE, ids=lambda w: w.name)
def test_block_partial_attention_edges(w):
    p = synth.make_block_weights(w)
    _, x = synth.make_latents(w)
    rng = np.random.default_rng(11)
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    for name, idx in {"half": np.sort(rng.choice(w.L, w.L // 2, replace=False)),
                      "one": np.array([0]), "all": np.arange(w.L)}.items():
        say(f"block {w.name} {name} n={len(idx)}")
        got = _block_gpu(w, p, x, idx)
        want = OB.block_partial(p, x, idx, w.H, kv=kv)
        check_block(got, want, w.dtype, f"{w.name}/{name}")


# bf16 shapes whose attention runs the balanced key ranges (at least 32 key
# tiles): few items, so that every item is cut into many pieces merged by the
# combine; query counts that leave the last query tile of a head with 48, 160
# and 288 queries (one, two and three waves with queries on the busiest
# SIMD: the three costs of a short item), whole tiles only, and every token;
# the 2100-token shape ends in a ragged key tile
BALANCED = [synth.Workload(f"balanced_bf16_{T * gh * gw}tok", T=T, grid=(gh, gw), D=256, H=2, F=512,
                           n_samples=8000, ratio=0.3, dtype="bf16", audio="speech", seed=70 + T)
            for T, gh, gw in [(5, 16, 32), (3, 20, 35)]]


@pytest.mark.parametrize("w", BALANCED, ids=lambda w: w.name)
def test_block_partial_balanced_ranges(w):
    p = synth.make_block_weights(w)
    _, x = synth.make_latents(w)
    rng = np.random.default_rng(13)
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    for n in (48, 432, 544, 672, 768, w.L):
        idx = np.sort(rng.choice(w.L, n, replace=False))
        say(f"block {w.name} n={n}")
        got = _block_gpu(w, p, x, idx)
        want = OB.block_partial(p, x, idx, w.H, kv=kv)
        check_block(got, want, w.dtype, f"{w.name}/n={n}")


def _reference_moves(q, k, H):
    """Per (query, head) row: how often a lazily rescaled streaming softmax
    moves its reference over the keys in 32-key halves (the reference starts
    at the first half's maximum and moves when a half's largest exp2
    argument exceeds it by more than 8), in fp64 from the oracle's q and k."""
    dh = q.shape[1] // H
    c = np.log2(np.e) / np.sqrt(dh)
    moves = []
    for h in range(H):
        s = (q[:, h * dh:(h + 1) * dh] @ k[:, h * dh:(h + 1) * dh].T) * c
        ref = s[:, :32].max(axis=1)
        n = np.zeros(s.shape[0], np.int64)
        for j in range(32, s.shape[1], 32):
            m = s[:, j:j + 32].max(axis=1)
            grow = m - ref > 8.0
            ref = np.where(grow, m, ref)
            n += grow
        moves.append(n)
    return np.concatenate(moves)


def test_block_partial_attention_rescale():
    """Peaked scores (query and key projections scaled by 10, score std about
    10): most rows move their softmax reference along the keys, in waves that
    also hold rows that do not move, which drives the attention's lazy
    rescale path; the block matches the oracle as the other blocks do."""
    w = synth.Workload("rescale_bf16_2600tok", T=5, grid=(20, 26), D=256, H=2, F=512,
                       n_samples=4000, ratio=0.5, dtype="bf16", audio="bursts", seed=77)
    p = synth.make_block_weights(w)
    for name in ("wq", "wk"):
        p[name] = synth.storage_round(p[name] * 10.0, w.dtype)
    _, x = synth.make_latents(w)
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    rng = np.random.default_rng(12)
    idx = np.sort(rng.choice(w.L, 1000, replace=False))
    q = OB.linear(kv[0][idx], OB._f64(p)["wq"], OB._f64(p)["bq"])
    moves = _reference_moves(q, kv[1], w.H)
    say(f"rescale: rows whose reference moves {np.mean(moves > 0):.2f}, moves per row up to {moves.max()}")
    assert np.mean(moves > 0) > 0.5 and np.mean(moves == 0) > 0.01
    got = _block_gpu(w, p, x, idx)
    want = OB.block_partial(p, x, idx, w.H, kv=kv)
    check_block(got, want, w.dtype, "rescale")


def test_block_gates_one_informational():
    # gates ~ N(1, 0.1): larger bf16 error budget; reported, bounded loosely
    w = RAGGED
    p = synth.make_block_weights(w, gate_mean=1.0, gate_std=0.1)
    _, x = synth.make_latents(w)
    idx = np.arange(w.L)
    got = _block_gpu(w, p, x, idx)
    want = OB.block_partial(p, x, idx, w.H)
    err = np.abs(got - want)
    say(f"  gates~N(1,0.1): max|err| {err.max():.3e}")
    assert err.max() < 0.1


_KV = {}


def _kv_shared(w, p, x, tag="x"):
    """The oracle's all-row LN + K/V projection of one input (`tag` names it),
    kept for the tests of one workload (it does not depend on the selection);
    at most two projections are held at a time."""
    key = (w.name, tag)
    if key not in _KV:
        while len(_KV) >= 2:
            _KV.pop(next(iter(_KV)))
        _KV[key] = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    return _KV[key]


ATTN_Q_TILE = 384   # queries of one attention workgroup
GEMM_TILE = 256     # rows of one GEMM tile


def _tile_rows(K, rng):
    """Positions in the selection that the full-size tests compare: one from
    every 384-query attention tile (each spans all heads, so the key-split
    tail items of the last round are reached too), every row of the last
    partial query tile, 16 rows of the last (partial) 256-row GEMM tile, and
    the first and last rows."""
    rows = [int(rng.integers(t, min(t + ATTN_Q_TILE, K))) for t in range(0, K, ATTN_Q_TILE)]
    rows += list(range((K // ATTN_Q_TILE) * ATTN_Q_TILE, K))
    last_g = ((K - 1) // GEMM_TILE) * GEMM_TILE
    rows += rng.choice(np.arange(last_g, K), min(16, K - last_g), replace=False).tolist()
    rows += [0, K - 1]
    return np.unique(np.asarray(rows, np.int64))


def test_block_partial_full_size_sampled():
    """Full-size block (32760 tokens) in the launch configuration the
    benchmark times; the oracle computes the all-row K/V projection and then
    the rows of every query tile."""
    w = synth.WAN14B_480P
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w)
    s, _, _ = OS.saliency(x, xref, fw, w.N)
    idx = OS.select_topk(s, w.K)
    say(f"block {w.name} K={w.K} (GPU)")
    got = _block_gpu(w, p, x, idx)
    rows = _tile_rows(w.K, np.random.default_rng(8))
    say(f"block {w.name}: oracle on {len(rows)} rows (every query tile)")
    want = OB.block_partial(p, x, idx[rows], w.H, kv=_kv_shared(w, p, x))
    check_block(got[rows], want, w.dtype, f"{w.name}/tile rows")


@pytest.mark.parametrize("ratio", synth.SWEEP_RATIOS, ids=lambda r: f"r{r}")
def test_block_partial_ratio_sweep_sampled(ratio):
    """The 32760-token block at every recompute ratio of the sweep (K from
    3276 to all 32760 tokens: other GEMM and attention grids and split tails
    than the 0.4 case), the rows of every query tile against the oracle."""
    w = synth.WAN14B_480P.with_(ratio=ratio)
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w)
    s, _, _ = OS.saliency(x, xref, fw, w.N)
    idx = OS.select_topk(s, w.K)
    say(f"block {w.name} r={ratio} K={w.K} (GPU)")
    got = _block_gpu(w, p, x, idx)
    rows = _tile_rows(w.K, np.random.default_rng(10))
    say(f"block r={ratio}: oracle on {len(rows)} rows (every query tile)")
    want = OB.block_partial(p, x, idx[rows], w.H, kv=_kv_shared(w, p, x))
    check_block(got[rows], want, w.dtype, f"{w.name}/r{ratio}/tile rows")


@pytest.mark.parametrize("w", [synth.WAN14B_480P, synth.WAN14B_720P], ids=lambda w: w.name)
def test_cached_step_end_to_end_full_size(w):
    """One whole cached step at full size through CachedBlock (the benchmark's
    calls and launch configuration), after the init step on xref:
      - the init step stores xref itself as the reference;
      - the selection equals the oracle's (ties within 1e-6 excluded);
      - codes, scales, references and the fused output equal the oracle's
        cache update bit for bit, given the GPU's fresh rows and init cache;
      - fresh rows of every query tile equal the oracle block, over the tokens
        both selections contain;
      - reused rows are within the block bar plus one quantization step of
        the oracle's own init-then-reuse output, and the init step's rows
        (every token recomputed: the dense block) match the oracle."""
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w)
    dt = tdtype(w.dtype)
    L, K = w.L, w.K
    rng = np.random.default_rng(12)
    blk = api.CachedBlock(params_to_device(p, w.dtype), w.H, L, w.D, device(), dt)
    say(f"step {w.name}: init on xref, then K={K} (GPU)")
    blk.init(up(xref, dt))
    torch.cuda.synchronize()
    xref0, codes0, scale0 = down(blk.xref).copy(), down(blk.codes).copy(), down(blk.scale).copy()
    # reused rows to check: a sample of tokens the oracle leaves unselected
    s, _, _ = OS.saliency(x, xref, fw, w.N)
    want_idx = OS.select_topk(s, K)
    rest_o = np.setdiff1d(np.arange(L), want_idx)
    reuse = np.sort(rng.choice(rest_o, 48, replace=False))
    ys_init = down(blk.y_sel)[reuse].copy()
    y = blk.step(up(x, dt), up(fw), w.N, k=K)
    torch.cuda.synchronize()

    assert np.array_equal(_bits(xref0), _bits(xref))
    gi = down(blk.sel.idx)[:K].astype(np.int64)
    nd = check_selection(gi, want_idx, s, K)
    say(f"  selection: {nd} tie-excluded differences")

    ys = down(blk.y_sel)[:K]
    y_o, xr_o, c_o, s_o = OC.cache_update(x, gi, ys, xref0, codes0, scale0, w.dtype)
    assert np.array_equal(down(blk.codes), c_o)
    assert np.array_equal(_bits(down(blk.scale)), _bits(s_o))
    assert np.array_equal(_bits(down(blk.xref)), _bits(xr_o))
    gy = down(y)
    assert np.array_equal(_bits(gy), _bits(y_o))
    del y_o, xr_o, c_o, s_o
    say("  cache state and fused output bit-exact")

    pos = _tile_rows(K, rng)
    pos = pos[np.isin(gi[pos], want_idx)]
    say(f"  fresh rows: oracle on {len(pos)} rows (every query tile)")
    want = OB.block_partial(p, x, gi[pos], w.H, kv=_kv_shared(w, p, x, "x"))
    check_block(ys[pos], want, w.dtype, f"{w.name}/step fresh rows")

    keep = ~np.isin(reuse, gi)                   # unselected on the GPU side too
    reuse, ys_init = reuse[keep], ys_init[keep]
    say(f"  reused rows: oracle init block on {len(reuse)} rows")
    yi = OB.block_partial(p, xref, reuse, w.H, kv=_kv_shared(w, p, xref, "xref")).astype(np.float32)
    check_block(ys_init, yi, w.dtype, f"{w.name}/init rows")
    c_i, s_i = OC.quantize_rows((yi - xref[reuse]).astype(np.float32))
    y_reuse_o = OC.cast_act(OC.dequantize_rows(xref[reuse], c_i, s_i), w.dtype)
    tol = TOL_BF16_ABS if w.dtype == "bf16" else TOL_F32_ABS
    sc = np.maximum(down(blk.scale)[reuse], s_i)[:, None]
    cast = np.abs(y_reuse_o) * (2.0 ** -8 if w.dtype == "bf16" else 2.0 ** -23)
    err = np.abs(gy[reuse].astype(np.float64) - y_reuse_o)
    say(f"  reused rows: max|err| {err.max():.3e}")
    assert (err <= tol + sc + cast).all(), float((err - (tol + sc + cast)).max())


def test_block_row_independence_full_size():
    """With the batch-invariant flag any selection gives exactly the rows of
    the all-token block (GPU vs GPU, bit-exact): holds at any size, checked at
    32760 tokens."""
    w = synth.WAN14B_480P
    p = synth.make_block_weights(w)
    _, x = synth.make_latents(w)
    P = params_to_device(p, w.dtype)
    X = up(x, tdtype(w.dtype))
    all_idx = torch.arange(w.L, dtype=torch.int32, device=device())
    ys_all = api.block_partial(P, X, all_idx, w.L, w.H, batch_invariant=True).clone()
    rng = np.random.default_rng(9)
    sub = np.sort(rng.choice(w.L, w.K, replace=False)).astype(np.int32)
    ys_sub = api.block_partial(P, X, up(sub), w.K, w.H, batch_invariant=True).clone()
    # the default path may split the attention of the last partial round
    # along the keys: same rows within the block tolerance
    ys_def = api.block_partial(P, X, up(sub), w.K, w.H)
    torch.cuda.synchronize()
    a = down(ys_all)[sub]
    b = down(ys_sub)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c = down(ys_def)
    err = np.abs(c.astype(np.float64) - b)
    assert err.max() <= TOL_BF16_ABS, float(err.max())
    assert np.linalg.norm(c - b) <= TOL_BF16_REL_L2 * np.linalg.norm(b)


# --------------------------------------------------------------- whole step

@pytest.mark.parametrize("w", [synth.TINY, RAGGED, synth.SMALL], ids=lambda w: w.name)
def test_cached_step_end_to_end(w):
    say(f"step {w.name}")
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w) if w is not RAGGED else np.array([0.3, 1.0, 0.0], np.float32)
    o_init = OST.init_step(p, xref, w.H, w.dtype)
    o_step = OST.cached_step(p, x, o_init["cache"], fw, w.N, w.H, w.K, w.dtype)
    dt = tdtype(w.dtype)
    P = params_to_device(p, w.dtype)
    blk = api.CachedBlock(P, w.H, w.L, w.D, device(), dt)
    blk.init(up(xref, dt))
    y = blk.step(up(x, dt), up(fw), w.N, k=w.K)
    torch.cuda.synchronize()
    gi = down(blk.sel.idx)[: w.K]
    nd = check_selection(gi, o_step["idx"], o_step["s"], w.K)
    gy = down(y)
    tol = TOL_F32_ABS if w.dtype == "f32" else TOL_BF16_ABS
    # fresh rows over the tokens both selections contain (all of them unless a
    # tie within 1e-6 of the K-th saliency went the other way)
    both, g_pos, o_pos = np.intersect1d(gi, o_step["idx"], return_indices=True)
    assert len(both) == w.K - nd // 2
    check_block(down(blk.y_sel)[: w.K][g_pos], o_step["y_sel"][o_pos], w.dtype, f"{w.name}/step y_sel")
    # reused rows: each side dequantizes its own cache; allow the block tolerance,
    # one quantization step of either cache, and the final cast
    rest = np.setdiff1d(np.arange(w.L), gi)
    sc = np.maximum(down(blk.scale)[rest], o_step["cache"][2][rest])[:, None]
    cast = np.abs(o_step["y"][rest]) * (2.0 ** -8 if w.dtype == "bf16" else 2.0 ** -23)
    err = np.abs(gy[rest].astype(np.float64) - o_step["y"][rest])
    assert (err <= tol + sc + cast).all(), float((err - (tol + sc + cast)).max())


def test_cached_step_deterministic():
    w = synth.SMALL
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = _frame_weight(w)
    dt = tdtype(w.dtype)
    P = params_to_device(p, w.dtype)
    outs = []
    for _ in range(2):
        blk = api.CachedBlock(P, w.H, w.L, w.D, device(), dt)
        blk.init(up(xref, dt))
        y = blk.step(up(x, dt), up(fw), w.N, ratio=w.ratio)
        torch.cuda.synchronize()
        outs.append([down(t).copy() for t in (blk.sel.idx[: w.K], blk.sel.mask, blk.codes,
                                              blk.scale, y)])
    for a, b in zip(*outs):
        assert np.array_equal(_bits(a), _bits(b))
