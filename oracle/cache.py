"""Oracle: int8 residual cache, its update and the reuse of cached rows
(Sec. 3.3 mask fusion; Sec. 3.4 "Memory-efficient Cache Management").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

The paper stores a cached output as a reference r plus an int8-quantized
residual (x_l - r), reads it back as r + dequantized residual, converts the
result back to the compute precision, and fuses block output and cache with
the mask: out = m * fresh + (1 - m) * cached.  Readings:

* one reference per token: r_i = the block input of token i at its last
  recompute (the same xref the saliency compares against), kept in the
  activation dtype;
* residual of a recomputed token: res = fp32(y_sel - x) (y_sel is the fresh
  fp32 block output), quantized with one symmetric absmax scale per token:
  amax = max|res|, scale = fp32(amax / 127), inv = fp32(127 / amax),
  code = clamp(rint_half_even(fp32(res * inv)), -127, 127); a zero residual
  gives scale 0 and codes 0.  These are fp32 operations because the codes
  are integers decided in the kernel's precision;
* a recomputed token's output is its fresh y_sel cast to the activation dtype;
  a reused token's output is cast(fp32(xref + fp32(scale * code)));
* the two mask fusions of the paper (after attention and after the FFN
  residual) collapse into one fusion at the block output, because unselected
  rows' attention output is never consumed inside the block.
"""
from __future__ import annotations

import numpy as np


def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 value (ties to even), returned as fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.int64)
    keep = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + keep) >> 16) << 16
    out = (rounded & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), np.float32(np.nan), out)


def cast_act(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_bf16(a) if dtype == "bf16" else a


def quantize_rows(res: np.ndarray):
    """Per-row symmetric int8 absmax quantization in fp32.  Returns
    (codes int8 [K, D], scale fp32 [K])."""
    res = np.asarray(res, dtype=np.float32)
    amax = np.abs(res).max(axis=1) if res.shape[1] else np.zeros(res.shape[0], np.float32)
    amax = amax.astype(np.float32)
    nz = amax > 0
    safe = np.where(nz, amax, np.float32(1))
    scale = np.where(nz, safe / np.float32(127), np.float32(0)).astype(np.float32)
    inv = (np.float32(127) / safe).astype(np.float32)
    q = (res * inv[:, None]).astype(np.float32)
    codes = np.clip(np.rint(q), -127, 127)
    codes = np.where(nz[:, None], codes, 0).astype(np.int8)
    return codes, scale


def dequantize_rows(xref: np.ndarray, codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """fp32(xref + fp32(scale * code)) per element (no fused multiply-add)."""
    prod = (np.asarray(scale, np.float32)[:, None] * codes.astype(np.float32)).astype(np.float32)
    return (np.asarray(xref, np.float32) + prod).astype(np.float32)


def cache_update(x, idx, y_sel, xref, codes, scale, dtype: str):
    """Write the fresh rows into the cache and assemble the block output.

    x [L, D] current block input; idx [K] ascending selected rows; y_sel
    [K, D] fp32 fresh outputs in idx order; (xref, codes, scale) the cache.
    Returns (y [L, D] in the activation dtype (as fp32 values), xref', codes',
    scale'), leaving the inputs untouched.
    """
    x = np.asarray(x, np.float32)
    idx = np.asarray(idx, np.int64)
    y_sel = np.asarray(y_sel, np.float32)
    xref2 = np.array(xref, dtype=np.float32, copy=True)
    codes2 = np.array(codes, dtype=np.int8, copy=True)
    scale2 = np.array(scale, dtype=np.float32, copy=True)
    L = x.shape[0]
    sel = np.zeros(L, dtype=bool)
    sel[idx] = True
    y = np.empty_like(x)
    rest = ~sel
    y[rest] = cast_act(dequantize_rows(xref2[rest], codes2[rest], scale2[rest]), dtype)
    if len(idx):
        res = (y_sel - x[idx]).astype(np.float32)
        c, s = quantize_rows(res)
        codes2[idx] = c
        scale2[idx] = s
        xref2[idx] = x[idx]
        y[idx] = cast_act(y_sel, dtype)
    return y, xref2, codes2, scale2


def empty_cache(L: int, D: int):
    return (np.zeros((L, D), np.float32), np.zeros((L, D), np.int8), np.zeros(L, np.float32))
