"""Pins for the block oracle (Sec. 3.3, latent-level caching): the partial
block must equal the dense block when every token is selected and must be
row-independent; the dense block is checked against torch's CPU functional
ops (a third-party implementation); closed forms for single-key attention,
zero gates and a hand-worked attention example."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import block as B
import synth

TINY = synth.TINY


def _params(w=TINY, seed=0, **kw):
    return synth.make_block_weights(w, seed=seed, **kw)


def _x(w=TINY, seed=0):
    return synth.make_latents(w, seed=seed)[1]


def test_partial_with_all_rows_equals_dense_block():
    p, x = _params(), _x()
    full = B.block_full(p, x, TINY.H)
    part = B.block_partial(p, x, np.arange(TINY.L), TINY.H)
    assert np.max(np.abs(part - full)) < 1e-12


def test_row_independence():
    p, x = _params(), _x()
    full = B.block_full(p, x, TINY.H)
    rng = np.random.default_rng(3)
    for K in (1, 5, 16, 31):
        idx = np.sort(rng.choice(TINY.L, size=K, replace=False))
        part = B.block_partial(p, x, idx, TINY.H)
        assert np.max(np.abs(part - full[idx])) < 1e-12


def test_dense_block_matches_torch_functional():
    p, x = _params(gate_mean=1.0, gate_std=0.1), _x()
    t = {k: torch.tensor(v, dtype=torch.float64) for k, v in p.items()}
    X = torch.tensor(x, dtype=torch.float64)
    D, H = TINY.D, TINY.H
    sh1, sc1, g1, sh2, sc2, g2 = t["mod"]
    a = Fn.layer_norm(X, (D,), eps=1e-6) * (1 + sc1) + sh1
    q = Fn.linear(a, t["wq"], t["bq"]).view(-1, H, D // H).transpose(0, 1)
    k = Fn.linear(a, t["wk"], t["bk"]).view(-1, H, D // H).transpose(0, 1)
    v = Fn.linear(a, t["wv"], t["bv"]).view(-1, H, D // H).transpose(0, 1)
    o = Fn.scaled_dot_product_attention(q, k, v).transpose(0, 1).reshape(-1, D)
    x1 = X + g1 * Fn.linear(o, t["wo"], t["bo"])
    b = Fn.layer_norm(x1, (D,), eps=1e-6) * (1 + sc2) + sh2
    y = x1 + g2 * Fn.linear(Fn.gelu(Fn.linear(b, t["w1"], t["b1"]), approximate="tanh"),
                            t["w2"], t["b2"])
    ours = B.block_full(p, x, H)
    assert np.max(np.abs(ours - y.numpy())) < 1e-12


def test_layer_norm_and_gelu_against_torch():
    z = np.random.default_rng(1).standard_normal((9, 33)) * 3 + 1
    ln = B.layer_norm(z)
    assert np.allclose(ln.mean(axis=1), 0, atol=1e-14)
    assert np.allclose((ln ** 2).mean(axis=1), 1 / (1 + 1e-6 / z.var(axis=1)), rtol=1e-12)
    ref = Fn.layer_norm(torch.tensor(z), (33,), eps=1e-6).numpy()
    assert np.max(np.abs(ln - ref)) < 1e-12
    g = B.gelu_tanh(z)
    gref = Fn.gelu(torch.tensor(z), approximate="tanh").numpy()
    assert np.max(np.abs(g - gref)) < 1e-12
    assert B.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_single_key_attention_returns_value():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((4, 8))
    k = rng.standard_normal((1, 8))
    v = rng.standard_normal((1, 8))
    o = B.attention(q, k, v, H=2)
    assert np.allclose(o, np.repeat(v, 4, axis=0), atol=1e-15)


def test_attention_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "attention_worked.json")))
    o = B.attention(np.array(g["q"]), np.array(g["k"]), np.array(g["v"]), H=1)
    assert np.allclose(o, np.array(g["out"]), atol=1e-14)


def test_attention_chunking_is_invisible():
    rng = np.random.default_rng(5)
    q, k, v = (rng.standard_normal((37, 16)) for _ in range(3))
    a = B.attention(q, k, v, H=2, chunk=1000)
    b = B.attention(q, k, v, H=2, chunk=5)
    assert np.max(np.abs(a - b)) < 1e-14


def test_zero_gates_return_input():
    p = _params(gate_mean=0.0, gate_std=0.0)
    x = _x()
    idx = np.array([0, 3, 9, 31])
    assert np.array_equal(B.block_partial(p, x, idx, TINY.H), x[idx].astype(np.float64))


def test_precomputed_kv_path_identical():
    p, x = _params(), _x()
    kv = B.kv_projection(B._f64(p), np.asarray(x, np.float64))
    idx = np.array([1, 2, 30])
    assert np.array_equal(B.block_partial(p, x, idx, TINY.H),
                          B.block_partial(p, x, idx, TINY.H, kv=kv))


def test_fp32_timing_mode_matches_fp64():
    """The fp32 mode (used only to time the oracle's steps with
    single-precision BLAS) computes the same block within fp32 rounding."""
    import synth
    w = synth.TINY
    p = synth.make_block_weights(w)
    _, x = synth.make_latents(w)
    idx = np.array([0, 5, 17, 31])
    a = B.block_partial(p, x, idx, w.H)
    b = B.block_partial(p, x, idx, w.H, dt=np.float32)
    assert b.dtype == np.float32
    assert np.abs(a - b).max() <= 1e-5 * max(1.0, np.abs(a).max())
