"""Pins of the ablation-variant oracle (Sec. 3.3 anchors and k_t = ceil(N r_t);
Table 2's Uniform / Random anchors, FP16 and naive INT8 caches, step-only and
latent-only schedules): brute-force subset search for the rankings, hand
values for the uniform spacing, the loud segments of a constructed clip as
energy anchors, naive INT8 as the residual codec against a zero reference,
exact reconstruction of representable rows, the rounding bound, torch's bf16
conversion for the 16-bit store, and hand-computed schedules."""
import itertools
import math

import numpy as np
import pytest
import torch

import synth
from oracle import block as OB
from oracle import cache as OC
from oracle import energy as OE
from oracle import variants as OV
from oracle.schedule import Schedule, ScheduleState, schedule_next, stack_trajectory


def _beats(a, i, b, j):
    """(a, i) ranks before (b, j): NaN first, then larger value, then smaller index."""
    an, bn = math.isnan(a), math.isnan(b)
    if an != bn:
        return an
    if not an and a != b:
        return a > b
    return i < j


def _brute_subset(vals, k):
    """The unique k-subset whose every member ranks before every non-member."""
    n = len(vals)
    found = []
    for sub in itertools.combinations(range(n), k):
        inside = set(sub)
        if all(_beats(float(vals[i]), i, float(vals[j]), j)
               for i in inside for j in range(n) if j not in inside):
            found.append(sub)
    assert len(found) == 1
    return list(found[0])


def test_anchors_topk_brute_force():
    rng = np.random.default_rng(0)
    for trial in range(40):
        T = int(rng.integers(1, 9))
        keys = rng.choice(np.array([0.0, 0.25, 0.5, 1.0, 3.0, np.nan], np.float32), size=T)
        if trial % 3 == 0:
            keys = rng.standard_normal(T).astype(np.float32)
        for k in range(T + 1):
            want = np.zeros(T, np.uint8)
            want[_brute_subset(keys, k)] = 1
            assert np.array_equal(OV.anchors_topk(keys, k), want), (keys, k)


def test_energy_anchors_are_the_loud_segments():
    # a silent clip with a bin-centred tone filling segments 2 and 5 (louder in 5)
    T, n, sr, n_fft = 7, 7 * 4000, 16000, 512
    audio = np.zeros(n)
    bounds = OE.segment_bounds(n, T)
    k0 = 40
    for t, amp in ((2, 0.3), (5, 0.6)):
        a, b = bounds[t]
        m = np.arange(b - a)
        audio[a:b] = amp * np.cos(2 * np.pi * k0 * m / n_fft)
    _, e, _ = OE.energy(audio.astype(np.float32), T, sr, n_fft)
    assert np.array_equal(np.flatnonzero(OV.anchors_topk(e, 2)), [2, 5])
    assert np.array_equal(np.flatnonzero(OV.anchors_topk(e, 1)), [5])
    # three anchors: the third is the first silent segment (ties go to the lower index)
    assert np.array_equal(np.flatnonzero(OV.anchors_topk(e, 3)), [0, 2, 5])


def test_random_anchors_are_the_largest_keys():
    keys = synth.random_anchor_keys(21, seed=3)
    m = OV.anchors_topk(keys, 7)
    assert m.sum() == 7
    assert keys[m == 1].min() > keys[m == 0].max()


def test_uniform_anchors_by_hand():
    idx = lambda T, k: list(np.flatnonzero(OV.anchors_uniform(T, k)))
    assert idx(21, 7) == [1, 4, 7, 10, 13, 16, 19]
    assert idx(10, 4) == [1, 3, 6, 8]
    assert idx(21, 1) == [10]
    assert idx(8, 8) == list(range(8))
    assert idx(5, 0) == []
    with pytest.raises(ValueError):
        OV.anchors_uniform(5, 6)


def test_uniform_anchors_spacing():
    for T in range(1, 40):
        for k in range(1, T + 1):
            t = np.flatnonzero(OV.anchors_uniform(T, k))
            assert len(t) == k
            gaps = np.diff(t)
            assert np.all(gaps >= math.floor(T / k)) and np.all(gaps <= math.ceil(T / k))
            # centred: the first and last anchors are equally far from the ends (to 1 segment)
            assert abs(t[0] - (T - 1 - t[-1])) <= 1


def test_select_segments_brute_force():
    rng = np.random.default_rng(1)
    for trial in range(60):
        T, N = int(rng.integers(1, 5)), int(rng.integers(1, 7))
        vals = np.array([0.0, 0.5, 1.0, 2.0, np.nan, -1.0], np.float32)
        s = rng.choice(vals, size=T * N) if trial % 2 else rng.standard_normal(T * N).astype(np.float32)
        anchors = (rng.random(T) < 0.6).astype(np.uint8)
        for k in range(N + 2):
            got = OV.select_segments(s, anchors, N, k)
            want = []
            for t in np.flatnonzero(anchors):
                want += [t * N + j for j in _brute_subset(s[t * N:(t + 1) * N], min(k, N))]
            assert list(got) == sorted(want), (s, anchors, k)
            assert len(got) == int(anchors.sum()) * min(k, N)


def test_select_segments_special_cases():
    T, N = 4, 6
    s = np.repeat(np.array([3.0, 1.0, 2.0, 0.0], np.float32), N)   # constant within a segment
    anchors = np.array([0, 1, 1, 0], np.uint8)
    # equal saliencies inside a segment: its first k tokens
    assert list(OV.select_segments(s, anchors, N, 2)) == [6, 7, 12, 13]
    # k >= N: every token of every anchor segment
    assert list(OV.select_segments(s, anchors, N, 9)) == list(range(6, 18))
    assert len(OV.select_segments(s, np.zeros(T, np.uint8), N, 3)) == 0
    assert len(OV.select_segments(s, anchors, N, 0)) == 0


def _cast_torch(a, dtype):
    if dtype == "f32":
        return np.asarray(a, np.float32)
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).float().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_naive_int8_is_residual_against_zero(dtype):
    rng = np.random.default_rng(2)
    L, D = 24, 40
    cache_n = OV.empty_codec_cache(L, D)
    cache_r = OC.empty_cache(L, D)
    zeros = np.zeros((L, D), np.float32)
    for step in range(3):
        idx = np.sort(rng.choice(L, 9, replace=False))
        y_sel = rng.standard_normal((9, D)).astype(np.float32) * (step + 1)
        x = rng.standard_normal((L, D)).astype(np.float32)
        y_n, *cache_n = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, x, idx, y_sel, *cache_n, dtype)
        y_r, *cache_r = OC.cache_update(zeros, idx, y_sel, *cache_r, dtype)
        assert np.array_equal(y_n.view(np.uint32), y_r.view(np.uint32))
        assert np.array_equal(cache_n[2], cache_r[1]) and np.array_equal(cache_n[3], cache_r[2])
        assert np.array_equal(cache_n[0][idx], x[idx])          # the saliency reference


def test_naive_int8_exact_and_bounded():
    rng = np.random.default_rng(3)
    L, D = 6, 64
    m = rng.integers(-127, 128, size=(L, D)).astype(np.float32)
    m[:, 0] = 127.0                                              # max |m| = 127 -> scale = c
    c = np.float32(2.0 ** -5)
    y_sel = m * c
    idx = np.arange(L)
    cache = OV.empty_codec_cache(L, D)
    _, *cache = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, y_sel, idx, y_sel, *cache, "f32")
    y, *_ = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, y_sel, np.zeros(0, int), np.zeros((0, D)), *cache, "f32")
    assert np.array_equal(y, y_sel)
    # general rows: |read back - y| <= scale / 2 (+ one fp32 rounding of the product)
    y_sel = rng.standard_normal((L, D)).astype(np.float32) * 3
    cache = OV.empty_codec_cache(L, D)
    _, *cache = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, y_sel, idx, y_sel, *cache, "f32")
    y, *_ = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, y_sel, np.zeros(0, int), np.zeros((0, D)), *cache, "f32")
    scale = np.abs(y_sel).max(axis=1) / 127
    assert np.all(np.abs(y - y_sel) <= scale[:, None] * (0.5 + 1e-6) + np.abs(y_sel) * 1e-7)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_full_cache_reads_the_last_write(dtype):
    rng = np.random.default_rng(4)
    L, D = 20, 24
    cache = OV.empty_codec_cache(L, D)
    last = {}
    for step in range(4):
        k = L if step == 0 and dtype == "f32" else 7
        idx = np.sort(rng.choice(L, k, replace=False))
        y_sel = rng.standard_normal((k, D)).astype(np.float32)
        x = rng.standard_normal((L, D)).astype(np.float32)
        y, *cache = OV.cache_update_codec(OV.CODEC_FULL, x, idx, y_sel, *cache, dtype)
        for l in range(L):
            if l in set(idx.tolist()):
                want = _cast_torch(y_sel[list(idx).index(l)], dtype)
            else:
                want = last.get(l, np.zeros(D, np.float32))
            assert np.array_equal(y[l], want), (step, l)
        for j, l in enumerate(idx):
            last[int(l)] = _cast_torch(y_sel[j], dtype)
        assert np.array_equal(cache[0][idx], x[idx])
        assert not cache[2].any() and not cache[3].any()        # codes and scales unused


def test_residual_beats_naive_near_the_input():
    # fresh outputs close to the input: the residual codec's step is set by
    # |y - x|, the naive one's by |y|, so the residual read-back is closer
    rng = np.random.default_rng(5)
    L, D = 16, 128
    x = rng.standard_normal((L, D)).astype(np.float32) * 4
    y_sel = (x + 0.05 * rng.standard_normal((L, D))).astype(np.float32)
    idx = np.arange(L)
    none = np.zeros(0, int)
    err = {}
    for codec in (OV.CODEC_RESIDUAL_INT8, OV.CODEC_NAIVE_INT8, OV.CODEC_FULL):
        cache = OV.empty_codec_cache(L, D)
        _, *cache = OV.cache_update_codec(codec, x, idx, y_sel, *cache, "f32")
        y, *_ = OV.cache_update_codec(codec, x, none, np.zeros((0, D)), *cache, "f32")
        err[codec] = float(np.abs(y - y_sel).max())
    assert err[OV.CODEC_FULL] == 0.0
    assert err[OV.CODEC_RESIDUAL_INT8] * 10 < err[OV.CODEC_NAIVE_INT8]


def test_schedule_presets_by_hand():
    L = 100
    st = ScheduleState()
    cfg = OV.step_only(n_full=1, refresh_delta=1.0)
    out = [schedule_next(cfg, st, d, L) for d in [5.0, 0.4, 0.4, 0.4, 0.3, 0.3, 0.5]]
    # accumulated 0.4, 0.8, 1.2 -> refresh; 0.3, 0.6, 1.1 -> refresh
    assert out == [(100, True), (0, False), (0, False), (100, True), (0, False), (0, False), (100, True)]
    st = ScheduleState()
    cfg = OV.latent_only(n_full=2, ratio=0.37)
    out = [schedule_next(cfg, st, d, L) for d in [1.0, 1.0, 0.9, 0.01, 0.5]]
    assert out == [(100, True), (100, True), (37, False), (37, False), (37, False)]


def _tiny_stack(n_blocks=2):
    w = synth.TINY
    blocks = [synth.make_block_weights(w.with_(seed=w.seed + 100 * b)) for b in range(n_blocks)]
    rng = np.random.default_rng(7)
    x = rng.standard_normal((w.L, w.D)).astype(np.float32)
    xs = []
    for t in range(5):
        xs.append(x.copy())
        x = (x + rng.standard_normal(x.shape) * (0.3 / (t + 1))).astype(np.float32)
    return w, blocks, xs


def test_two_stage_stack_all_anchors_full_ratio_is_all_full():
    w, blocks, xs = _tiny_stack()
    anchors = np.ones(w.T, np.uint8)
    fw = np.linspace(0.3, 1.0, w.T).astype(np.float32)
    got = stack_trajectory(blocks, xs, fw, w.N, w.H, Schedule(1, 1.0, 1.0, 0.0), "f32", anchors=anchors)
    want = stack_trajectory(blocks, xs, fw, w.N, w.H, Schedule(len(xs), 0.0, 0.0, 0.0), "f32")
    for (k, full, _, y), (_, _, _, wy) in zip(got, want):
        assert k == w.N or full
        assert np.array_equal(y, wy)


def test_two_stage_stack_step_by_hand():
    # the first cached step of a one-block stack, composed directly
    w, blocks, xs = _tiny_stack(n_blocks=1)
    anchors = np.array([0, 1], np.uint8)
    cfg = Schedule(1, 0.25, 0.25, 0.0)
    got = stack_trajectory(blocks, xs[:2], np.ones(w.T, np.float32), w.N, w.H, cfg, "f32",
                           anchors=anchors, codec=OV.CODEC_NAIVE_INT8)
    p = blocks[0]
    cache = OV.empty_codec_cache(w.L, w.D)
    y0, *cache = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, xs[0], np.arange(w.L),
                                       OB.block_partial(p, xs[0], np.arange(w.L), w.H).astype(np.float32),
                                       *cache, "f32")
    assert np.array_equal(got[0][3], y0)
    # cached step: delta_i against the first input; 4 tokens of segment 1
    delta = np.abs(xs[1].astype(np.float64) - xs[0]).sum(1) / (np.abs(xs[0].astype(np.float64)).sum(1) + 1e-6)
    seg = delta[w.N:].astype(np.float32)
    top = w.N + np.sort(np.argsort(-seg, kind="stable")[:4])
    y1, *_ = OV.cache_update_codec(OV.CODEC_NAIVE_INT8, xs[1], top,
                                   OB.block_partial(p, xs[1], top, w.H).astype(np.float32), *cache, "f32")
    assert got[1][:2] == (4, False)
    assert np.array_equal(got[1][3], y1)
