"""Seeded random sweep of tiny shapes on the GPU against the oracle: every
C-ABI call of the path at L in [1, 300] tokens and 1 to 8 latent frames, with
K in {0, 1, L - 1, L} and random counts, silent frames (exact saliency ties),
unchanged tokens (zero relative change) and duplicated rows.  The top-K is
checked against a pure-Python brute-force ranking, the rest against the
oracle with the bars of the other parity tests."""
import numpy as np
import pytest
import torch

from oracle import block as OB
from oracle import cache as OC
from oracle import energy as OE
from oracle import select as OS
from paper_2608_02474_amd import api

from gpu_util import check_block, check_selection, down, params_to_device, say, tdtype, up

pytestmark = pytest.mark.gpu

SEEDS = range(24)


def _brute_topk(s, K):
    """The K tokens first by (saliency desc, index asc), by sorting pairs."""
    order = sorted(range(len(s)), key=lambda i: (-float(s[i]), i))
    return np.array(sorted(order[:K]), np.int64)


def _shape(rng, max_tokens=300):
    T = int(rng.integers(1, 9))
    N = int(rng.integers(1, max_tokens // T + 1))
    return T, N


def _counts(rng, L):
    return sorted({0, 1, max(L - 1, 0), L, int(rng.integers(0, L + 1))})


def _latents(rng, L, D, dtype, T, N):
    xref = rng.standard_normal((L, D)).astype(np.float32)
    x = xref + rng.uniform(0.01, 0.3, (T, 1, 1)).astype(np.float32).repeat(N, 1).reshape(L, 1) * \
        rng.standard_normal((L, D)).astype(np.float32)
    same = rng.random(L) < 0.15                      # unchanged tokens: delta = 0
    x[same] = xref[same]
    if L >= 4:                                       # duplicated rows: equal saliency in one frame
        x[1] = x[0]
        xref[1] = xref[0]
    cast = OC.cast_act
    return cast(xref, dtype), cast(x, dtype)


@pytest.mark.parametrize("seed", SEEDS)
def test_fuzz_select(seed):
    rng = np.random.default_rng(1000 + seed)
    T, N = _shape(rng)
    L = T * N
    D = int(rng.choice([8, 16, 24, 64, 136]))
    dtype = "bf16" if seed % 2 else "f32"
    xref, x = _latents(rng, L, D, dtype, T, N)
    fw = rng.uniform(0.0, 1.0, T).astype(np.float32)
    fw[rng.random(T) < 0.3] = 0.0                    # silent frames: exact zero ties
    s, num, den = OS.saliency(x, xref, fw, N)
    dt = tdtype(dtype)
    X, XR, FW = up(x, dt), up(xref, dt), up(fw)
    for K in _counts(rng, L):
        say(f"fuzz select seed={seed} T={T} N={N} D={D} {dtype} K={K}")
        sel = api.select(X, XR, FW, N, k=K)
        torch.cuda.synchronize()
        gs = down(sel.saliency)
        assert (np.abs(gs.astype(np.float64) - s) <= 1e-6 * np.abs(s.astype(np.float64))).all()
        gi = down(sel.idx)[:K]
        if K:
            check_selection(gi, _brute_topk(s, K), s, K)
        m = down(sel.mask)
        assert m.sum() == K and (m[gi] == 1).all()
        assert int(down(sel.n_sel_dev)[0]) == K
        assert float(down(sel.step_delta)[0]) == pytest.approx(OS.step_delta(num, den), rel=1e-12)
    th = float(rng.choice(s)) if L else 0.0
    sel = api.select(X, XR, FW, N, threshold=th)
    torch.cuda.synchronize()
    n = sel.count()
    got = set(down(sel.idx)[:n].tolist())
    want = {i for i in range(L) if float(s[i]) > th}
    for i in got ^ want:
        assert abs(float(s[i]) - th) <= 1e-6 * max(abs(th), 1e-30)


@pytest.mark.parametrize("seed", SEEDS)
def test_fuzz_block(seed):
    rng = np.random.default_rng(2000 + seed)
    T, N = _shape(rng)
    L = T * N
    if seed % 2:
        dtype, D, H, F = "bf16", 256, 2, 512
    else:
        dtype, D, H, F = "f32", 64, 2, 128
    p = {"wq": (D, D), "wk": (D, D), "wv": (D, D), "wo": (D, D), "w1": (F, D), "w2": (D, F),
         "bq": (D,), "bk": (D,), "bv": (D,), "bo": (D,), "b1": (F,), "b2": (D,)}
    p = {k: OC.cast_act(rng.normal(0, 0.02, v).astype(np.float32), dtype) for k, v in p.items()}
    mod = rng.normal(0, 0.1, (6, D)).astype(np.float32)
    mod[[2, 5]] = rng.normal(0.25, 0.05, (2, D)).astype(np.float32)
    p["mod"] = mod
    _, x = _latents(rng, L, D, dtype, T, N)
    P = params_to_device(p, dtype)
    X = up(x, tdtype(dtype))
    kv = OB.kv_projection(OB._f64(p), np.asarray(x, np.float64))
    for K in _counts(rng, L):
        if K == 0:
            continue
        idx = np.sort(rng.choice(L, K, replace=False))
        say(f"fuzz block seed={seed} L={L} {dtype} K={K}")
        got = down(api.block_partial(P, X, up(idx.astype(np.int32)), K, H))
        torch.cuda.synchronize()
        want = OB.block_partial(p, x, idx, H, kv=kv)
        check_block(got, want, dtype, f"fuzz/{seed}/K{K}")


@pytest.mark.parametrize("seed", SEEDS)
def test_fuzz_cache_update(seed):
    rng = np.random.default_rng(3000 + seed)
    T, N = _shape(rng)
    L = T * N
    D = int(rng.choice([8, 16, 40, 64, 264]))
    dtype = "bf16" if seed % 2 else "f32"
    xref, x = _latents(rng, L, D, dtype, T, N)
    codes0 = rng.integers(-127, 128, (L, D)).astype(np.int8)
    scale0 = rng.uniform(0, 0.02, L).astype(np.float32)
    scale0[rng.random(L) < 0.2] = 0.0
    dt = tdtype(dtype)
    for K in _counts(rng, L):
        say(f"fuzz cache seed={seed} L={L} D={D} {dtype} K={K}")
        idx = np.sort(rng.choice(L, K, replace=False)).astype(np.int32)
        y_sel = (x[idx] + rng.standard_normal((K, D)) * rng.uniform(0, 0.2, (K, 1))).astype(np.float32)
        if K:
            y_sel[0] = x[idx[0]]                     # zero residual
        y_o, xr_o, c_o, s_o = OC.cache_update(x, idx, y_sel, xref, codes0, scale0, dtype)
        XR, C, S = up(xref, dt), up(codes0), up(scale0)
        Y = api.cache_update(up(x, dt), up(idx) if K else None, up(OS.mask_of(idx, L)), K,
                             up(y_sel) if K else None, XR, C, S)
        torch.cuda.synchronize()
        assert np.array_equal(down(C), c_o)
        assert np.array_equal(down(S).view(np.uint32), s_o.view(np.uint32))
        assert np.array_equal(down(XR).view(np.uint32), xr_o.view(np.uint32))
        assert np.array_equal(down(Y).view(np.uint32), y_o.view(np.uint32))


@pytest.mark.parametrize("seed", SEEDS)
def test_fuzz_energy(seed):
    rng = np.random.default_rng(4000 + seed)
    T = int(rng.integers(1, 9))
    n = int(rng.integers(T, 20000))
    n_fft = int(rng.choice([16, 18, 64, 100, 256, 512, 1024]))
    hop = int(rng.integers(max(1, n_fft // 4), n_fft + 1))
    bands = int(rng.integers(1, 17))
    audio = (rng.standard_normal(n) * 0.1).astype(np.float32)
    audio[: n // 3] = 0.0 if seed % 3 == 0 else audio[: n // 3]    # leading silence
    say(f"fuzz energy seed={seed} n={n} T={T} n_fft={n_fft} hop={hop} bands={bands}")
    Eb, e, w = OE.energy(audio, T, 16000, n_fft, hop, bands)
    gb, ge, gw = api.energy(up(audio), T, 16000, n_fft, hop, bands)
    torch.cuda.synchronize()
    for got, want, name in ((down(gb), Eb, "band"), (down(ge), e, "frame"), (down(gw), w, "weight")):
        err = np.abs(got.astype(np.float64) - want)
        assert (err <= 1e-6 * np.abs(want.astype(np.float64))).all(), (name, float(err.max()))
