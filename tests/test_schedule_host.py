"""The library's step schedule (a host function of the C ABI, no GPU needed)
against the schedule oracle: identical k and full-step decisions over random
Eq. 1 sequences, and argument validation."""
import ctypes

import numpy as np
import pytest

from oracle.schedule import Schedule, ScheduleState, schedule_next
from paper_2608_02474_amd import _lib


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def _lib_run(lib, cfg: Schedule, deltas, L):
    c = _lib.ScheduleCfg(cfg.n_full, cfg.r_min, cfg.r_max, cfg.alpha, cfg.refresh_delta)
    st = _lib.ScheduleState(0, 0.0, 0.0)
    full = ctypes.c_int32(-1)
    out = []
    for d in deltas:
        k = lib.echo_schedule_next(ctypes.byref(c), ctypes.byref(st), float(d), L, ctypes.byref(full))
        assert k >= 0
        out.append((k, bool(full.value)))
    return out


@pytest.mark.parametrize("seed", range(6))
def test_schedule_matches_oracle(lib, seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 100000))
    cfg = Schedule(n_full=int(rng.integers(0, 5)), r_min=float(rng.uniform(0, 0.4)),
                   r_max=0.0, alpha=float(rng.uniform(0, 2)),
                   refresh_delta=float(rng.choice([0.0, rng.uniform(0.1, 2.0)])))
    cfg.r_max = float(rng.uniform(cfg.r_min, 1.0))
    deltas = np.abs(rng.standard_normal(40)) * rng.uniform(0.01, 1.0)
    deltas[rng.random(40) < 0.1] = 0.0
    st = ScheduleState()
    want = [schedule_next(cfg, st, float(d), L) for d in deltas]
    assert _lib_run(lib, cfg, deltas, L) == want


def test_schedule_rejects_bad_arguments(lib):
    st = _lib.ScheduleState(0, 0.0, 0.0)
    full = ctypes.c_int32(0)
    bad = [_lib.ScheduleCfg(0, 0.5, 0.4, 1.0, 0.0),          # r_min > r_max
           _lib.ScheduleCfg(0, -0.1, 0.4, 1.0, 0.0),         # r_min < 0
           _lib.ScheduleCfg(0, 0.1, 1.5, 1.0, 0.0),          # r_max > 1
           _lib.ScheduleCfg(-1, 0.1, 0.4, 1.0, 0.0),         # n_full < 0
           _lib.ScheduleCfg(0, 0.1, 0.4, float("inf"), 0.0)]
    for c in bad:
        assert lib.echo_schedule_next(ctypes.byref(c), ctypes.byref(st), 0.5, 100,
                                      ctypes.byref(full)) == -_lib.ECHO_EINVAL
    ok = _lib.ScheduleCfg(0, 0.1, 0.4, 1.0, 0.0)
    assert lib.echo_schedule_next(ctypes.byref(ok), ctypes.byref(st), float("nan"), 100,
                                  ctypes.byref(full)) == -_lib.ECHO_EINVAL
    assert lib.echo_schedule_next(ctypes.byref(ok), ctypes.byref(st), 0.5, 0,
                                  ctypes.byref(full)) == -_lib.ECHO_EINVAL
    assert st.step == 0                                     # rejected calls leave the state alone


def test_topk_count_matches_oracle(lib):
    """echo_topk_count (the K the host passes to the top-K) against the
    oracle's count: every workload's K, the sweep ratios, random ratios."""
    import synth
    from oracle.select import topk_count
    for w in synth.ALL.values():
        assert lib.echo_topk_count(w.ratio, w.L) == w.K == topk_count(w.ratio, w.L)
    for r in synth.SWEEP_RATIOS:
        assert lib.echo_topk_count(r, 32760) == topk_count(r, 32760)
    rng = np.random.default_rng(3)
    for _ in range(2000):
        L = int(rng.integers(1, 200000))
        r = float(rng.choice([rng.random(), round(rng.random(), 2), 0.0, 1.0]))
        assert lib.echo_topk_count(r, L) == topk_count(r, L), (r, L)
    assert lib.echo_topk_count(0.01, 10) == 1                 # ceil, not round
    for bad in (-0.1, 1.01, float("nan")):
        assert lib.echo_topk_count(bad, 10) == -_lib.ECHO_EINVAL
    assert lib.echo_topk_count(0.5, 0) == -_lib.ECHO_EINVAL


def test_segments_count(lib):
    assert lib.echo_segments_count(14, 1560, 624) == 14 * 624
    assert lib.echo_segments_count(14, 1560, 5000) == 14 * 1560     # at most N per segment
    assert lib.echo_segments_count(0, 1560, 10) == 0
    assert lib.echo_segments_count(21, 1560, 0) == 0
    assert lib.echo_segments_count(-1, 10, 1) == -_lib.ECHO_EINVAL
    assert lib.echo_segments_count(1, 0, 1) == -_lib.ECHO_EINVAL
    assert lib.echo_segments_count(1, 10, -1) == -_lib.ECHO_EINVAL
    assert lib.echo_segments_count(65536, 65536, 65536) == -_lib.ECHO_EINVAL
