"""GPU parity of the module-ablation variants (Sec. 3.3 anchors and
k_t = ceil(N r_t); Table 2): anchor segments by energy, random keys and even
spacing (exact), the two-stage selection (exact up to saliency ties), the
16-bit and naive int8 cache codecs (bit-exact) and block stacks that use them
(within the block tolerance)."""
import numpy as np
import pytest
import torch

import synth
from oracle import energy as OE
from oracle import select as OS
from oracle import variants as OV
from oracle.cache import cast_act
from oracle.schedule import Schedule, stack_trajectory
from paper_2608_02474_amd import api

from gpu_util import (TOL_BF16_ABS, TOL_BF16_REL_L2, TOL_F32_ABS, check_selection, device, down,
                      params_to_device, say, tdtype, up)

pytestmark = pytest.mark.gpu

CODEC_NAMES = {OV.CODEC_RESIDUAL_INT8: "residual_int8", OV.CODEC_FULL: "full",
               OV.CODEC_NAIVE_INT8: "naive_int8"}


# ------------------------------------------------------------------ anchors
def test_energy_anchors_480p():
    w = synth.WAN14B_480P
    audio = synth.make_audio(w.audio, w.n_samples, w.sample_rate, w.seed)
    _, e, _ = OE.energy(audio, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
    _, fe, _ = api.energy(up(audio), w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
    se = np.sort(e.astype(np.float64))[::-1]
    # neighbouring energies differ far beyond the energy tolerance, so the ranking is unique
    assert (np.abs(np.diff(se)) > 1e-4 * se[:-1]).all()
    for k in (0, 1, 5, 7, 10, w.T):
        say(f"energy anchors T={w.T} k={k}")
        got = down(api.anchors(w.T, k, "energy", keys=fe))
        assert np.array_equal(got, OV.anchors_topk(e, k)), k


@pytest.mark.parametrize("T", [1, 21, 1000, 1025, 4096])
def test_random_anchors_with_ties(T):
    keys = synth.random_anchor_keys(T, seed=T)
    coarse = (np.round(keys * 8) / 8).astype(np.float32)      # many exact ties
    coarse[:: max(1, T // 5)] = np.nan
    for name, kk in (("random", keys), ("coarse+nan", coarse)):
        for k in sorted({0, 1, T // 3, max(T - 1, 0), T}):
            say(f"top-k anchors {name} T={T} k={k}")
            got = down(api.anchors(T, k, "random", keys=up(kk)))
            assert np.array_equal(got, OV.anchors_topk(kk, k)), (name, k)


@pytest.mark.parametrize("T", [1, 7, 21, 1024, 1025, 4096])
def test_uniform_anchors(T):
    for k in sorted({0, 1, max(T // 3, 1), max(T - 1, 0), T}):
        say(f"uniform anchors T={T} k={k}")
        got = down(api.anchors(T, k, "uniform", device=device()))
        assert np.array_equal(got, OV.anchors_uniform(T, k)), k


# -------------------------------------------------------- two-stage selection
def _segments_case(w, anchors, ks, tie_rows=0):
    xref, x = synth.make_latents(w)
    if tie_rows:
        rows = np.random.default_rng(w.seed).choice(w.L, tie_rows, replace=False)
        x[rows] = xref[rows]                                   # delta 0: exact ties
    unit = np.ones(w.T, np.float32)
    s, _, _ = OS.saliency(x, xref, unit, w.N)
    dt = tdtype(w.dtype)
    sel = api.saliency(up(x, dt), up(xref, dt), up(unit), w.N)
    A = up(anchors.astype(np.uint8))
    torch.cuda.synchronize()
    gs = down(sel.saliency)
    assert (np.abs(gs.astype(np.float64) - s) <= 1e-6 * np.abs(s.astype(np.float64))).all()
    n_anchor = int(anchors.sum())
    for k in ks:
        say(f"segments {w.name} T={w.T} N={w.N} anchors={n_anchor} k={k}")
        api.topk_segments(sel, A, w.N, k)
        torch.cuda.synchronize()
        kk = min(k, w.N)
        n = int(down(sel.n_sel_dev)[0])
        assert n == n_anchor * kk
        got = down(sel.idx)[:n]
        want = OV.select_segments(s, anchors, w.N, k)
        assert list(got) == sorted(got)
        diffs = 0
        for j, t in enumerate(np.flatnonzero(anchors)):
            g = got[j * kk:(j + 1) * kk]
            assert ((g >= t * w.N) & (g < (t + 1) * w.N)).all()
            if kk:
                diffs += check_selection(g - t * w.N, want[j * kk:(j + 1) * kk] - t * w.N,
                                         s[t * w.N:(t + 1) * w.N], kk)
        m = down(sel.mask)
        assert m.sum() == n and (m[got] == 1).all()
        say(f"  ok ({diffs} tie-excluded differences)")


def test_segments_ragged_with_ties():
    w = synth.TINY.with_(name="segments_ragged", T=3, grid=(10, 10), D=64, dtype="f32", seed=31)
    _segments_case(w, np.array([1, 0, 1]), [0, 1, 37, 99, 100, 150], tie_rows=40)


def test_segments_480p_bf16():
    w = synth.WAN14B_480P
    audio = synth.make_audio(w.audio, w.n_samples, w.sample_rate, w.seed)
    _, e, _ = OE.energy(audio, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
    k = OS.topk_count(w.ratio, w.N)
    _segments_case(w, OV.anchors_topk(e, 7), [k, 1, w.N])
    _segments_case(w.with_(seed=5), OV.anchors_uniform(w.T, 7), [k])


@pytest.mark.parametrize("grid,T", [((64, 64), 3), ((200, 200), 2)], ids=["4096tok", "40000tok"])
def test_segments_large_segments(grid, T):
    # 4096 tokens per segment: keys in registers (8 per thread); 40000: re-read per pass
    w = synth.TINY.with_(name=f"segments_{grid[0]}x{grid[1]}", T=T, grid=grid, D=64, dtype="f32", seed=32)
    anchors = np.ones(T, np.uint8)
    anchors[0] = 0
    N = grid[0] * grid[1]
    _segments_case(w, anchors, [1, OS.topk_count(0.3, N), N - 1, N], tie_rows=N // 4)


# ----------------------------------------------------------------- codecs
def _codec_run(codec, L, D, dtype, steps, seed, ratio=0.4):
    rng = np.random.default_rng(seed)
    dt = tdtype(dtype)
    ora = OV.empty_codec_cache(L, D)
    full = codec == OV.CODEC_FULL
    xref = torch.zeros((L, D), dtype=dt, device=device())
    store = torch.zeros((L, D), dtype=dt, device=device()) if full else None
    codes = None if full else torch.zeros((L, D), dtype=torch.int8, device=device())
    scale = None if full else torch.zeros(L, dtype=torch.float32, device=device())
    for step in range(steps):
        k = L if step == 0 else max(1, int(ratio * L))
        idx = np.arange(L) if step == 0 else np.sort(rng.choice(L, k, replace=False))
        x = cast_act(rng.standard_normal((L, D)).astype(np.float32), dtype)
        y_sel = (x[idx] + 0.3 * rng.standard_normal((k, D))).astype(np.float32)
        say(f"codec {CODEC_NAMES[codec]} L={L} D={D} {dtype} step {step} k={k}")
        y_o, *ora = OV.cache_update_codec(codec, x, idx, y_sel, *ora, dtype)
        mask = np.zeros(L, np.uint8)
        mask[idx] = 1
        y_g = api.cache_update_codec(codec, up(x, dt), up(idx.astype(np.int32)), up(mask), k, up(y_sel),
                                     xref, store=store, codes=codes, scale=scale)
        torch.cuda.synchronize()
        bits = lambda a: np.asarray(a, np.float32).view(np.uint32)
        assert np.array_equal(bits(down(y_g)), bits(y_o)), "output"
        assert np.array_equal(bits(down(xref)), bits(ora[0])), "saliency reference"
        if full:
            assert np.array_equal(bits(down(store)), bits(ora[1])), "store"
        else:
            assert np.array_equal(down(codes), ora[2]), "codes"
            assert np.array_equal(bits(down(scale)), bits(ora[3])), "scales"


@pytest.mark.parametrize("codec", [OV.CODEC_FULL, OV.CODEC_NAIVE_INT8, OV.CODEC_RESIDUAL_INT8],
                         ids=lambda c: CODEC_NAMES[c])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_codec_small(codec, dtype):
    # D = 264: one 8-element chunk per lane with idle lanes; D = 8200: the streamed form
    _codec_run(codec, L=300, D=264, dtype=dtype, steps=3, seed=40 + codec)
    _codec_run(codec, L=40, D=8200, dtype=dtype, steps=3, seed=50 + codec)


@pytest.mark.parametrize("codec", [OV.CODEC_FULL, OV.CODEC_NAIVE_INT8], ids=lambda c: CODEC_NAMES[c])
def test_codec_full_size(codec):
    _codec_run(codec, L=32760, D=5120, dtype="bf16", steps=2, seed=60 + codec)


def test_codec_entry_matches_cache_update():
    # codec 0 of the codec entry point is echo_cache_update
    rng = np.random.default_rng(70)
    L, D = 96, 512
    dt = torch.bfloat16
    x = up(rng.standard_normal((L, D)).astype(np.float32), dt)
    idx = np.sort(rng.choice(L, 30, replace=False)).astype(np.int32)
    mask = np.zeros(L, np.uint8)
    mask[idx] = 1
    y_sel = up(rng.standard_normal((30, D)).astype(np.float32))
    outs = []
    for use_codec in (False, True):
        xref = up(rng.standard_normal((L, D)).astype(np.float32), dt) if not outs else outs[0][1].clone()
        st = [xref.clone(), torch.zeros((L, D), dtype=torch.int8, device=device()),
              torch.zeros(L, dtype=torch.float32, device=device())]
        if use_codec:
            y = api.cache_update_codec(0, x, up(idx), up(mask), 30, y_sel, st[0], codes=st[1], scale=st[2])
        else:
            y = api.cache_update(x, up(idx), up(mask), 30, y_sel, st[0], st[1], st[2])
        torch.cuda.synchronize()
        outs.append((y, xref, st))
    (y0, _, s0), (y1, _, s1) = outs
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    for a, b in zip(s0, s1):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))


# ----------------------------------------------------------------- stacks
RAGGED = synth.Workload("ragged_bf16_300tok", T=3, grid=(10, 10), D=256, H=2, F=512,
                        n_samples=4000, ratio=0.37, dtype="bf16", audio="bursts", seed=21)


def _trajectory(w, steps, seed=7):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((w.L, w.D)).astype(np.float32)
    out = []
    for t in range(steps):
        out.append(cast_act(x, w.dtype))
        x = (x + rng.standard_normal(x.shape) * (0.3 / (t + 1))).astype(np.float32)
    return out


def _stack_variant(w, n_blocks, steps, sched, anchors=None, codec=OV.CODEC_RESIDUAL_INT8):
    blocks = [synth.make_block_weights(w.with_(seed=w.seed + 100 * b)) for b in range(n_blocks)]
    xs = _trajectory(w, steps)
    fw = np.linspace(0.3, 1.0, w.T).astype(np.float32)
    want = stack_trajectory(blocks, xs, fw, w.N, w.H, sched, w.dtype, anchors=anchors, codec=codec)
    dt = tdtype(w.dtype)
    stack = api.BlockStack([params_to_device(p, w.dtype) for p in blocks], w.H, w.L, w.D, device(), dt,
                           api.Scheduler(sched.n_full, sched.r_min, sched.r_max, sched.alpha,
                                         sched.refresh_delta),
                           anchor_mask=None if anchors is None else up(anchors.astype(np.uint8)),
                           n_anchors=None if anchors is None else int(np.count_nonzero(anchors)),
                           codec=CODEC_NAMES[codec])
    for t, x in enumerate(xs):
        y = stack.step(up(x, dt), up(fw), w.N)
        torch.cuda.synchronize()
        k, full, delta = stack.history[-1]
        wk, wfull, wdelta, wy = want[t]
        say(f"stack {w.name} x{n_blocks} anchors={anchors} codec={CODEC_NAMES[codec]} step {t}: "
            f"k={k} full={full}")
        assert (k, full) == (wk, wfull)
        if t >= sched.n_full:
            assert delta == pytest.approx(wdelta, rel=1e-12)
        got = down(y).astype(np.float64)
        err = np.abs(got - wy)
        mx, rel = float(err.max()), float(np.linalg.norm(got - wy) / np.linalg.norm(wy))
        say(f"  last block output: max|err| {mx:.3e} rel-L2 {rel:.3e}")
        if w.dtype == "f32":
            assert mx <= TOL_F32_ABS * n_blocks
        else:
            assert mx <= TOL_BF16_ABS * n_blocks and rel <= TOL_BF16_REL_L2 * n_blocks
    return stack


def test_stack_two_stage_f32():
    w = synth.TINY.with_(name="tiny_two_stage", T=4, grid=(4, 4))
    _stack_variant(w, 2, 5, Schedule(1, 0.25, 0.75, 0.6), anchors=np.array([1, 0, 1, 1], np.uint8))


@pytest.mark.parametrize("codec", [OV.CODEC_FULL, OV.CODEC_NAIVE_INT8], ids=lambda c: CODEC_NAMES[c])
def test_stack_codecs_f32(codec):
    _stack_variant(synth.TINY, 2, 5, Schedule(1, 0.3, 0.6, 0.5), codec=codec)


def test_stack_two_stage_bf16_uniform_naive():
    _stack_variant(RAGGED, 3, 4, Schedule(1, 0.2, 0.6, 0.5), anchors=OV.anchors_uniform(RAGGED.T, 2),
                   codec=OV.CODEC_NAIVE_INT8)


def test_stack_step_only_and_latent_only():
    w = synth.TINY
    _stack_variant(w, 2, 6, OV.step_only(n_full=1, refresh_delta=0.2))
    _stack_variant(w, 2, 4, OV.latent_only(n_full=1, ratio=0.4))
