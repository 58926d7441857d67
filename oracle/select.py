"""Oracle: per-token saliency and recompute selection (Sec. 3.1 Eq. 1;
Sec. 3.3 "Cross-modal Saliency Anchors" and "Energy-Guided Step-Latent Cache
Scheduling").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

Readings of what the paper leaves open:

* Eq. 1's relative change is taken per token against that token's cached
  block input xref_i (its input at its last recompute):
  delta_i = ||x_i - xref_i||_1 / (||xref_i||_1 + xi), sums in fp64, xi = 1e-6;
* the audio energy enters as a per-frame weight: token i of frame
  t(i) = floor(i / N) gets saliency s_i = fp32(w_t(i) * delta_i);
* the recompute set is one global top-K over all L = T N tokens with
  K = ceil(r L), ordered by (s descending, token index ascending); a NaN
  saliency ranks above every number; the indices are returned ascending;
* threshold mode selects {i : s_i > theta} instead;
* the step-level Eq. 1 value is the same ratio over all tokens,
  sum_i num_i / (sum_i den_i + xi).
"""
from __future__ import annotations

import math

import numpy as np


def relative_change(x: np.ndarray, xref: np.ndarray, xi: float = 1e-6):
    """Per-token L1 numerator, denominator and delta (Eq. 1 form), fp64."""
    x = np.asarray(x, dtype=np.float64)
    xref = np.asarray(xref, dtype=np.float64)
    num = np.abs(x - xref).sum(axis=1)
    den = np.abs(xref).sum(axis=1)
    return num, den, num / (den + xi)


def saliency(x, xref, frame_weight, N: int, xi: float = 1e-6):
    """s_i = fp32(w_{floor(i/N)} * delta_i); returns (s fp32 [L], num, den)."""
    num, den, delta = relative_change(x, xref, xi)
    L = len(delta)
    w = np.asarray(frame_weight, dtype=np.float32).astype(np.float64)
    frame = np.arange(L) // N
    s = (w[frame] * delta).astype(np.float32)
    return s, num, den


def step_delta(num, den, xi: float = 1e-6) -> float:
    return float(np.sum(num) / (np.sum(den) + xi))


def topk_count(ratio: float, L: int) -> int:
    """K = ceil(r L), clamped to [0, L] (k_t = ceil(N r_t) over all tokens)."""
    return min(L, max(0, math.ceil(ratio * L - 1e-9)))


def _rank_key(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, dtype=np.float32).astype(np.float64)
    return np.where(np.isnan(s), np.inf, s), np.isnan(s)


def select_topk(s: np.ndarray, K: int) -> np.ndarray:
    """Indices of the K tokens ranked first by (s desc, index asc), ascending."""
    L = len(s)
    if not 0 <= K <= L:
        raise ValueError("K out of range")
    key, isnan = _rank_key(s)
    idx = np.arange(L)
    # primary: NaN first, then larger s; secondary: smaller index
    order = np.lexsort((idx, -key, ~isnan))
    return np.sort(order[:K]).astype(np.int32)


def select_threshold(s: np.ndarray, theta: float) -> np.ndarray:
    key, isnan = _rank_key(s)
    return np.nonzero(isnan | (key > np.float64(np.float32(theta))))[0].astype(np.int32)


def mask_of(idx: np.ndarray, L: int) -> np.ndarray:
    m = np.zeros(L, dtype=np.uint8)
    m[np.asarray(idx, dtype=np.int64)] = 1
    return m
