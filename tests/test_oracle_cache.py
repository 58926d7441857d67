"""Pins for the cache oracle (Sec. 3.3 mask fusion; Sec. 3.4 reference plus
int8 residual): a hand-worked quantization, the round-trip error bound,
special cases, bf16 rounding against torch, and whole-step invariants
(ratio 1 = dense block, ratio 0 = dequantized cache)."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import block as B
from oracle import cache as C
from oracle import select as S
from oracle import step as ST
import synth


def test_int8_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "int8_residual_worked.json")))
    res = np.array([g["residual"]], dtype=np.float32)
    codes, scale = C.quantize_rows(res)
    assert codes[0].tolist() == g["codes"]
    assert scale[0] == np.float32(g["scale"])


def test_roundtrip_error_bound_and_symmetry():
    rng = np.random.default_rng(0)
    res = (rng.standard_normal((64, 300)) * rng.uniform(1e-3, 10, size=(64, 1))).astype(np.float32)
    codes, scale = C.quantize_rows(res)
    rec = scale[:, None].astype(np.float64) * codes
    err = np.abs(res - rec)
    # half a quantization step, plus fp32 rounding of scale and of res * inv
    assert (err <= scale[:, None] * (0.5 + 1e-5)).all()
    assert (np.abs(codes) <= 127).all()
    assert (np.abs(codes).max(axis=1) == 127).all()       # the absmax element hits 127
    c2, s2 = C.quantize_rows(-res)
    assert np.array_equal(c2, -codes) and np.array_equal(s2, scale)


def test_codes_within_one_of_the_exact_definition():
    """The fp32 operation order that decides the codes stays within one code
    of the plain definition rint(res * 127 / amax) evaluated in fp64, and the
    scale within an fp32 rounding of amax / 127."""
    rng = np.random.default_rng(4)
    res = (rng.standard_normal((256, 513)) * rng.uniform(1e-6, 1e3, size=(256, 1))).astype(np.float32)
    res[::7, ::3] = 0.0
    res[5] = np.float32(1.0) / np.arange(1, 514, dtype=np.float32)     # many codes near .5
    codes, scale = C.quantize_rows(res)
    r64 = res.astype(np.float64)
    amax = np.abs(r64).max(axis=1, keepdims=True)
    exact = np.clip(np.rint(r64 * 127.0 / amax), -127, 127)
    assert (np.abs(codes.astype(np.int64) - exact) <= 1).all()
    assert np.mean(codes == exact) > 0.999
    assert np.allclose(scale.astype(np.float64), amax[:, 0] / 127.0, rtol=2 ** -23, atol=0)


def test_zero_and_one_hot_rows():
    z = np.zeros((2, 10), np.float32)
    z[1, 4] = -3.5
    codes, scale = C.quantize_rows(z)
    assert (codes[0] == 0).all() and scale[0] == 0
    assert codes[1].tolist() == [0, 0, 0, 0, -127, 0, 0, 0, 0, 0]
    assert scale[1] == np.float32(3.5) / np.float32(127)


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(1)
    a = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 7,
                        np.array([0.0, -0.0, 1.00390625, 1.01171875, 3e38, -1e-40], np.float32)])
    ours = C.round_bf16(a)
    ref = torch.tensor(a).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_cache_update_semantics():
    rng = np.random.default_rng(2)
    L, D = 12, 16
    x = rng.standard_normal((L, D)).astype(np.float32)
    xref = rng.standard_normal((L, D)).astype(np.float32)
    codes = rng.integers(-127, 128, size=(L, D)).astype(np.int8)
    scale = rng.uniform(0, 0.01, size=L).astype(np.float32)
    idx = np.array([1, 5, 6, 11])
    y_sel = (x[idx] + 0.1 * rng.standard_normal((4, D))).astype(np.float32)
    y, xr2, c2, s2 = C.cache_update(x, idx, y_sel, xref, codes, scale, "f32")
    rest = np.setdiff1d(np.arange(L), idx)
    # fresh rows: output = y_sel, reference = current input, codes re-quantized
    assert np.array_equal(y[idx], y_sel)
    assert np.array_equal(xr2[idx], x[idx])
    assert np.array_equal(xr2[rest], xref[rest]) and np.array_equal(c2[rest], codes[rest])
    assert np.array_equal(s2[rest], scale[rest])
    # reused rows: reference + dequantized residual, elementwise in fp32
    want = xref[rest].astype(np.float64) + scale[rest, None].astype(np.float64) * codes[rest]
    assert np.max(np.abs(y[rest] - want)) <= 1e-6 * np.max(np.abs(want))
    # the stored residual reconstructs the fresh output within half a step
    rec = xr2[idx] + s2[idx, None] * c2[idx].astype(np.float32)
    assert (np.abs(rec - y_sel) <= s2[idx, None] * 0.5 + 1e-6).all()


def test_step_ratio_zero_returns_dequantized_cache_and_one_returns_dense():
    w = synth.TINY
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    fw = synth.random_frame_weight(w.T, 0)
    init = ST.init_step(p, xref, w.H, w.dtype)
    # init output = dense block of xref (fresh rows, fp32 activations)
    dense = B.block_full(p, xref, w.H).astype(np.float32)
    assert np.array_equal(init["y"], dense)
    # ratio 0: nothing recomputed; the output is the dequantized cache, within
    # half a quantization step of the cached dense output
    r0 = ST.cached_step(p, x, init["cache"], fw, w.N, w.H, 0, w.dtype)
    xr, cd, sc = init["cache"]
    assert len(r0["idx"]) == 0
    assert np.array_equal(r0["y"], C.dequantize_rows(xr, cd, sc))
    assert (np.abs(r0["y"] - dense) <= sc[:, None] * 0.5 + 1e-5).all()
    # ratio 1: every row recomputed on the current input = dense block of x
    r1 = ST.cached_step(p, x, init["cache"], fw, w.N, w.H, w.L, w.dtype)
    assert np.array_equal(r1["y"], B.block_full(p, x, w.H).astype(np.float32))
    # cache state is plain arrays: save / restore gives the same step
    saved = tuple(a.copy() for a in init["cache"])
    again = ST.cached_step(p, x, saved, fw, w.N, w.H, w.K, w.dtype)
    first = ST.cached_step(p, x, init["cache"], fw, w.N, w.H, w.K, w.dtype)
    assert np.array_equal(again["y"], first["y"])
    assert first["idx"].tolist() == S.select_topk(first["s"], w.K).tolist()
