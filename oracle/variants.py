"""Oracle: the selection and cache-codec variants of the paper's module
ablation (Sec. 3.3 "Cross-modal Saliency Anchors" and the per-segment count
k_t = ceil(N r_t); Sec. 4 ablation, Table 2: Uniform / Random anchors, FP16
and naive INT8 caches, step-only and latent-only scheduling).

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

What the paper states: before generation the k highest-energy audio segments
are chosen by a top-k over the energy vector; their latents form a
[T, N] saliency mask; in a cached step, the high-saliency segments update
k_t = ceil(N r_t) latents each.  The ablation replaces the energy-based choice
of segments by a uniform or a random one, and the residual int8 cache by a
16-bit cache of the outputs themselves or by int8 quantization of the outputs
without a reference.

Readings (the paper leaves these open):

* anchors: a 0/1 mask over the T segments.  Energy anchors are the k segments
  ranked first by (frame energy desc, segment index asc), the ranking of the
  token top-k; Random anchors are the k segments ranked first by uniform
  random keys drawn per clip (an input here); Uniform anchors are the evenly
  spaced segments t_j = floor((2j + 1) T / (2k)), j = 0..k-1;
* two-stage selection: in every anchor segment, the min(k_t, N) tokens ranked
  first by (saliency desc, index asc) within that segment; tokens of other
  segments are reused; a full step recomputes every token.  The in-segment
  ranking uses s_i = fp32(delta_i) (unit frame weights), since a positive
  per-segment weight cannot reorder a segment;
* the FP16 cache is a cache of the outputs in the activation dtype (bf16 or
  fp32 here): a selected token stores cast(y_sel), an unselected token reads
  its stored row back unchanged;
* the naive INT8 cache quantizes the fresh output itself with the per-token
  absmax code of the residual cache and reads back cast(fp32(scale * code));
* every codec records the selected tokens' current input as the saliency
  reference xref, as the residual cache does;
* step-only scheduling: whole steps are either recomputed or reused (k = 0 on
  cached steps, full steps from the leading ones and the Eq. 2 refresh);
  latent-only scheduling: a fixed ratio on every step after the leading full
  ones (no step-level adaptation).
"""
from __future__ import annotations

import numpy as np

from oracle import cache as OC
from oracle import select as OS
from oracle.schedule import Schedule

CODEC_RESIDUAL_INT8, CODEC_FULL, CODEC_NAIVE_INT8 = 0, 1, 2


# -- anchors -----------------------------------------------------------------
def anchors_topk(keys, k: int) -> np.ndarray:
    """Mask [T] of the k segments ranked first by (key desc, index asc); NaN
    keys rank first.  Energy anchors: keys = frame energies; Random anchors:
    keys = per-clip uniform random numbers."""
    keys = np.asarray(keys, np.float32)
    return OS.mask_of(OS.select_topk(keys, k), len(keys))


def anchors_uniform(T: int, k: int) -> np.ndarray:
    """Mask [T] of the evenly spaced segments floor((2j + 1) T / (2k))."""
    if not 0 <= k <= T:
        raise ValueError("k out of range")
    m = np.zeros(T, np.uint8)
    for j in range(k):
        m[((2 * j + 1) * T) // (2 * k)] = 1
    return m


# -- two-stage selection -----------------------------------------------------
def select_segments(s, anchors, N: int, k: int) -> np.ndarray:
    """Ascending token indices: min(k, N) tokens per anchor segment, ranked by
    (s desc, index asc) inside the segment."""
    s = np.asarray(s, np.float32)
    anchors = np.asarray(anchors)
    T = len(anchors)
    assert len(s) == T * N and k >= 0
    kk = min(k, N)
    out = []
    for t in range(T):
        if anchors[t]:
            out.append(t * N + OS.select_topk(s[t * N:(t + 1) * N], kk).astype(np.int64))
    return (np.concatenate(out) if out else np.zeros(0, np.int64)).astype(np.int32)


# -- cache codecs --------------------------------------------------------------
def empty_codec_cache(L: int, D: int):
    """(xref, store, codes, scale): saliency reference, 16-bit output store,
    int8 codes and scales, all zero."""
    return (np.zeros((L, D), np.float32), np.zeros((L, D), np.float32),
            np.zeros((L, D), np.int8), np.zeros(L, np.float32))


def cache_update_codec(codec: int, x, idx, y_sel, xref, store, codes, scale, dtype: str):
    """Write the fresh rows with the given codec and assemble the block output.

    Returns (y, xref', store', codes', scale') without touching the inputs;
    y and the stored rows are activation-dtype values held as fp32."""
    x = np.asarray(x, np.float32)
    idx = np.asarray(idx, np.int64)
    y_sel = np.asarray(y_sel, np.float32)
    if codec == CODEC_RESIDUAL_INT8:
        y, xref2, codes2, scale2 = OC.cache_update(x, idx, y_sel, xref, codes, scale, dtype)
        return y, xref2, np.array(store, np.float32, copy=True), codes2, scale2
    L = x.shape[0]
    xref2 = np.array(xref, np.float32, copy=True)
    store2 = np.array(store, np.float32, copy=True)
    codes2 = np.array(codes, np.int8, copy=True)
    scale2 = np.array(scale, np.float32, copy=True)
    rest = np.ones(L, bool)
    rest[idx] = False
    y = np.empty_like(x)
    if codec == CODEC_FULL:
        y[rest] = store2[rest]
        if len(idx):
            store2[idx] = OC.cast_act(y_sel, dtype)
    elif codec == CODEC_NAIVE_INT8:
        prod = (scale2[rest][:, None] * codes2[rest].astype(np.float32)).astype(np.float32)
        y[rest] = OC.cast_act(prod, dtype)
        if len(idx):
            c, sc = OC.quantize_rows(y_sel)
            codes2[idx] = c
            scale2[idx] = sc
    else:
        raise ValueError("unknown codec")
    if len(idx):
        xref2[idx] = x[idx]
        y[idx] = OC.cast_act(y_sel, dtype)
    return y, xref2, store2, codes2, scale2


# -- scheduling presets ----------------------------------------------------------
def step_only(n_full: int, refresh_delta: float) -> Schedule:
    """Whole-step caching: cached steps recompute nothing; the Eq. 2 refresh
    recomputes a whole step once the accumulated change exceeds the threshold."""
    return Schedule(n_full=n_full, r_min=0.0, r_max=0.0, alpha=0.0, refresh_delta=refresh_delta)


def latent_only(n_full: int, ratio: float) -> Schedule:
    """Token-level caching at a fixed ratio on every cached step."""
    return Schedule(n_full=n_full, r_min=ratio, r_max=ratio, alpha=0.0)
