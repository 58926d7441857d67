"""Pins of the step-level schedule oracle (Sec. 3.1 Eq. 2, Sec. 3.3 r_t and
k_t): hand-computed sequences for the full steps, the clip, the running-max
normalization, the Eq. 2 refresh and the ceiling; the stack runner against
direct compositions of the block and cache oracles."""
import numpy as np
import pytest

import synth
from oracle import block as OB
from oracle import cache as OC
from oracle import select as OS
from oracle import step as OST
from oracle.schedule import Schedule, ScheduleState, schedule_next, stack_trajectory


def _run(cfg, deltas, L=100):
    st = ScheduleState()
    return [schedule_next(cfg, st, d, L) for d in deltas]


def test_leading_full_steps_ignore_delta():
    out = _run(Schedule(n_full=2, r_min=0.1, r_max=0.5, alpha=1.0), [9.0, 9.0, 0.3])
    assert out[0] == (100, True) and out[1] == (100, True)
    assert out[2] == (50, False)        # first cached step: normalized delta 1 -> clip(1.1) = 0.5


def test_running_max_normalization_by_hand():
    # r_min 0.1, alpha 0.4: deltas 0.5, 1.0, 0.25 -> normalized 1, 1, 0.25 -> r 0.5, 0.5, 0.2
    out = _run(Schedule(n_full=0, r_min=0.1, r_max=0.6, alpha=0.4), [0.5, 1.0, 0.25])
    assert out == [(50, False), (50, False), (20, False)]


def test_clip_bounds():
    assert _run(Schedule(0, 0.15, 0.3, 100.0), [1.0])[0] == (30, False)
    assert _run(Schedule(0, 0.15, 0.3, 0.0), [1.0])[0] == (15, False)
    # a delta of 0 after a positive one: normalized 0 -> r_min
    assert _run(Schedule(0, 0.15, 0.3, 1.0), [1.0, 0.0])[1] == (15, False)


def test_eq2_refresh():
    cfg = Schedule(n_full=1, r_min=0.2, r_max=0.2, alpha=0.0, refresh_delta=1.0)
    out = _run(cfg, [0.0, 0.4, 0.4, 0.4, 0.4, 0.4, 0.4])
    # accumulated 0.4, 0.8, 1.2 > 1 -> full and restart; 0.4, 0.8, 1.2 -> full
    assert [f for _, f in out] == [True, False, False, True, False, False, True]
    assert [k for k, _ in out] == [100, 20, 20, 100, 20, 20, 100]


def test_ceiling_of_exact_products():
    # r L exactly 25 stays 25; 25.000001 goes to 26
    assert _run(Schedule(0, 0.25, 0.25, 0.0), [1.0])[0][0] == 25
    assert _run(Schedule(0, 0.2500001, 0.3, 0.0), [1.0])[0][0] == 26


def _tiny_inputs(w, steps, seed=5):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((w.L, w.D)).astype(np.float32)
    out = []
    for t in range(steps):
        out.append(x.copy())
        x = (x + rng.standard_normal(x.shape) * (0.3 / (t + 1))).astype(np.float32)
    return out


def test_stack_all_full_is_the_block_composition():
    w = synth.TINY
    blocks = [synth.make_block_weights(w.with_(seed=s)) for s in (0, 1)]
    xs = _tiny_inputs(w, 2)
    fw = np.ones(w.T, np.float32)
    res = stack_trajectory(blocks, xs, fw, w.N, w.H, Schedule(n_full=9, r_min=0.1, r_max=0.5, alpha=1.0),
                           "f32")
    for (k, full, _, y), x in zip(res, xs):
        assert full and k == w.L
        want = x
        for p in blocks:
            want = OB.block_full(p, want, w.H).astype(np.float32)
        assert np.allclose(y, want, rtol=0, atol=1e-6)


def test_stack_of_one_block_is_the_cached_step():
    w = synth.TINY
    p = synth.make_block_weights(w)
    xs = _tiny_inputs(w, 3)
    fw = np.linspace(0.2, 1.0, w.T).astype(np.float32)
    cfg = Schedule(n_full=1, r_min=0.25, r_max=0.75, alpha=0.5)
    res = stack_trajectory([p], xs, fw, w.N, w.H, cfg, "f32")
    o = OST.init_step(p, xs[0], w.H, "f32")
    assert np.array_equal(res[0][3], o["y"])
    cache = o["cache"]
    st = ScheduleState()
    schedule_next(cfg, st, 0.0, w.L)
    for t in (1, 2):
        s, num, den = OS.saliency(xs[t], cache[0], fw, w.N)
        k, full = schedule_next(cfg, st, OS.step_delta(num, den), w.L)
        assert not full and res[t][0] == k
        c = OST.cached_step(p, xs[t], cache, fw, w.N, w.H, k, "f32")
        assert np.array_equal(res[t][3], c["y"])
        cache = c["cache"]
