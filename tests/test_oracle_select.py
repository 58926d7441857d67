"""Pins for the saliency / selection oracle (Sec. 3.1 Eq. 1; Sec. 3.3):
closed forms for the relative change, brute-force ranking with pure-Python
sorting, and special cases (K = 0, K = L, ties, NaN)."""
import math

import numpy as np
import pytest

from oracle import select as S
import synth


def _brute_topk(s, K):
    # pure-Python: sort (index) by (NaN first, larger value first, smaller index)
    L = len(s)
    keyed = sorted(range(L), key=lambda i: (0 if math.isnan(s[i]) else 1,
                                            -float(s[i]) if not math.isnan(s[i]) else 0.0, i))
    return sorted(keyed[:K])


def test_relative_change_closed_forms():
    rng = np.random.default_rng(0)
    xref = rng.standard_normal((6, 40)).astype(np.float32)
    num, den, d = S.relative_change(xref, xref)
    assert (num == 0).all() and (d == 0).all()
    for c in (0.5, -0.25, 2.0):
        x = ((1 + c) * xref.astype(np.float64))
        _, den, d = S.relative_change(x, xref, xi=1e-6)
        l1 = np.abs(xref.astype(np.float64)).sum(axis=1)
        assert np.allclose(den, l1, rtol=1e-14)
        assert np.allclose(d, abs(c) * l1 / (l1 + 1e-6), rtol=1e-12)
    # zero reference row: delta = ||x||_1 / xi
    x = np.ones((1, 8))
    _, _, d = S.relative_change(x, np.zeros((1, 8)), xi=1e-6)
    assert d[0] == pytest.approx(8e6)


def test_saliency_uses_frame_of_token():
    # token i belongs to frame floor(i / N); weight 0 on a frame zeroes it
    T, N, D = 3, 4, 8
    rng = np.random.default_rng(2)
    xref = rng.standard_normal((T * N, D))
    x = 2 * xref                                  # delta = 1 (up to xi) everywhere
    w = np.array([0.0, 0.5, 1.0], np.float32)
    s, _, _ = S.saliency(x, xref, w, N)
    assert (s[:4] == 0).all()
    assert np.allclose(s[4:8], 0.5, rtol=1e-6) and np.allclose(s[8:], 1.0, rtol=1e-6)
    assert s.dtype == np.float32


@pytest.mark.parametrize("L,seed", [(1, 0), (7, 1), (64, 2), (300, 3)])
def test_topk_brute_force(L, seed):
    rng = np.random.default_rng(seed)
    # few distinct values -> many exact ties
    s = rng.integers(0, 5, size=L).astype(np.float32) / 4
    for K in sorted({0, 1, L // 3, L // 2, L - 1, L}):
        if K < 0:
            continue
        assert S.select_topk(s, K).tolist() == _brute_topk(s.tolist(), K)


def test_topk_special_cases():
    L = 50
    s = np.random.default_rng(4).random(L).astype(np.float32)
    assert S.select_topk(s, 0).tolist() == []
    assert S.select_topk(s, L).tolist() == list(range(L))
    z = np.zeros(L, np.float32)                   # all ties -> lowest indices
    assert S.select_topk(z, 7).tolist() == list(range(7))
    s2 = s.copy()
    s2[[3, 17]] = np.nan                          # NaN ranks above every number
    top2 = S.select_topk(s2, 2).tolist()
    assert top2 == [3, 17]
    with pytest.raises(ValueError):
        S.select_topk(s, L + 1)


def test_half_silence_ties_fill_in_index_order():
    # frames 0..1 silent (weight 0): once the nonzero tokens are exhausted the
    # remaining picks are the lowest-index zero-saliency tokens.
    T, N, D = 4, 5, 16
    rng = np.random.default_rng(5)
    xref = rng.standard_normal((T * N, D))
    x = xref + 0.1 * rng.standard_normal((T * N, D))
    w = np.array([0, 0, 0.7, 1.0], np.float32)
    s, _, _ = S.saliency(x, xref, w, N)
    idx = S.select_topk(s, 13)
    assert idx.tolist() == list(range(3)) + list(range(10, 20))


def test_topk_count_exact_for_workloads():
    assert S.topk_count(0.5, 32) == 16
    assert S.topk_count(0.25, 7800) == 1950
    assert S.topk_count(0.4, 32760) == 13104
    assert [S.topk_count(r, 32760) for r in synth.SWEEP_RATIOS] == [3276, 8190, 16380, 32760]
    assert S.topk_count(0.3, 75600) == 22680
    assert S.topk_count(0.0, 10) == 0 and S.topk_count(1.0, 10) == 10
    assert S.topk_count(0.01, 10) == 1                       # ceil, not round
    for w in (synth.TINY, synth.SMALL, synth.WAN14B_480P, synth.WAN14B_720P):
        assert S.topk_count(w.ratio, w.L) == w.K


def test_threshold_brute_force():
    rng = np.random.default_rng(6)
    s = rng.random(200).astype(np.float32)
    s[10] = np.nan
    th = 0.6
    got = S.select_threshold(s, th).tolist()
    want = [i for i in range(200) if math.isnan(s[i]) or float(s[i]) > float(np.float32(th))]
    assert got == want


def test_step_delta_matches_eq1_over_all_tokens():
    rng = np.random.default_rng(7)
    xref = rng.standard_normal((10, 6))
    x = xref + 0.3 * rng.standard_normal((10, 6))
    num, den, _ = S.relative_change(x, xref)
    want = np.abs(x - xref).sum() / (np.abs(xref).sum() + 1e-6)
    assert S.step_delta(num, den) == pytest.approx(want, rel=1e-14)
