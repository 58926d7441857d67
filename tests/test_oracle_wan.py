"""Pins of the Wan-style block oracle (qk RMSNorm, 3D RoPE, cross-attention
with restricted queries, a batch of two): hand-computed rotary angles, the
rotation's isometry and relative-position property, torch's rms_norm, a
one-token context, and the whole block against a dense formulation built from
torch's CPU functional ops (layer_norm, rms_norm, complex rotation,
scaled_dot_product_attention, gelu) with every token selected."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import wan_block as OW

W = synth.TINY.with_(name="wan_tiny", T=3, grid=(3, 4), D=96, H=2, F=128, dtype="f32", seed=5)


def test_rope_split():
    assert OW.rope_split(128) == (22, 21, 21)
    assert OW.rope_split(12) == (2, 2, 2)
    assert sum(OW.rope_split(64)) == 32


def test_rope_angles_by_hand():
    # dh = 12: two pairs per axis with frequencies 1 and 10000^(-1/2) = 0.01;
    # token (t, r, c) = (1, 2, 3) of a grid of 4 x 5 is row 1*20 + 2*5 + 3 = 33
    ang = OW.rope_angles([33], (4, 5), 12)[0]
    assert np.allclose(ang, [1.0, 0.01, 2.0, 0.02, 3.0, 0.03], rtol=1e-15, atol=0)
    assert np.array_equal(OW.rope_angles([0], (4, 5), 12)[0], np.zeros(6))


def test_rope_is_a_rotation_per_pair():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((40, 24))
    rows = rng.integers(0, 60, 40)
    out = OW.apply_rope(z, rows, (3, 5), H=2)
    n_in = z[:, 0::2] ** 2 + z[:, 1::2] ** 2
    n_out = out[:, 0::2] ** 2 + out[:, 1::2] ** 2
    assert np.allclose(n_in, n_out, rtol=1e-12)
    # position 0 is the identity
    assert np.allclose(OW.apply_rope(z[:1], [0], (3, 5), H=2), z[:1], rtol=0, atol=0)


def test_rope_relative_position():
    # <R(i) q, R(j) k> depends only on the position difference: shift both
    # tokens by (1, 1, 1) in (t, r, c)
    rng = np.random.default_rng(1)
    grid = (6, 7)
    q, k = rng.standard_normal((1, 36)), rng.standard_normal((1, 36))
    step = grid[0] * grid[1] + grid[1] + 1
    for i, j in ((0, 10), (8, 50), (45, 9)):
        a = float((OW.apply_rope(q, [i], grid, 3) @ OW.apply_rope(k, [j], grid, 3).T)[0, 0])
        b = float((OW.apply_rope(q, [i + step], grid, 3) @ OW.apply_rope(k, [j + step], grid, 3).T)[0, 0])
        assert a == pytest.approx(b, rel=1e-11, abs=1e-12)


def test_rms_norm_against_torch():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((7, 33)) * 3
    g = rng.standard_normal(33)
    want = F.rms_norm(torch.from_numpy(z), (33,), weight=torch.from_numpy(g), eps=1e-6).numpy()
    assert np.allclose(OW.rms_norm(z, g), want, rtol=1e-13, atol=1e-14)


def test_one_token_context_gives_its_value():
    # softmax over a single key is 1: the cross-attention output is vc for every query
    p = synth.make_wan_block_weights(W)
    x = np.random.default_rng(3).standard_normal((W.L, W.D)).astype(np.float32)
    ctx = np.random.default_rng(4).standard_normal((1, W.D)).astype(np.float32)
    from oracle.block import attention, linear
    qc = np.random.default_rng(5).standard_normal((5, W.D))
    kc = OW.rms_norm(linear(ctx, p["wkc"], p["bkc"]), p["gkc"])
    vc = linear(ctx, p["wvc"], p["bvc"])
    assert np.allclose(attention(qc, kc, vc, W.H), np.repeat(vc, 5, axis=0), rtol=1e-14)


def _torch_dense(p, x, ctx, H, grid):
    """Every token selected, written with torch's CPU functional ops in fp64."""
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    x, ctx = T(x), T(ctx)
    P = {k: T(v) for k, v in p.items()}
    L, D = x.shape
    dh = D // H
    mod = P["mod"]

    def lin(a, w, b):
        return a @ P[w].T + P[b]

    def heads(z):
        return z.reshape(z.shape[0], H, dh).transpose(0, 1)   # [H, n, dh]

    def rope(z):
        ang = torch.from_numpy(OW.rope_angles(np.arange(L), grid, dh))
        rot = torch.polar(torch.ones_like(ang), ang)           # [L, dh/2]
        zc = torch.view_as_complex(z.reshape(L, H, dh // 2, 2).contiguous())
        return torch.view_as_real(zc * rot[:, None, :]).reshape(L, D)

    def attn(q, k, v):
        o = F.scaled_dot_product_attention(heads(q)[None], heads(k)[None], heads(v)[None])[0]
        return o.transpose(0, 1).reshape(q.shape[0], D)

    a = F.layer_norm(x, (D,), eps=1e-6) * (1 + mod[1]) + mod[0]
    q = rope(F.rms_norm(lin(a, "wq", "bq"), (D,), P["gq"], 1e-6))
    k = rope(F.rms_norm(lin(a, "wk", "bk"), (D,), P["gk"], 1e-6))
    x1 = x + mod[2] * lin(attn(q, k, lin(a, "wv", "bv")), "wo", "bo")
    c = F.layer_norm(x1, (D,), weight=P["g3"], bias=P["b3"], eps=1e-6)
    qc = F.rms_norm(lin(c, "wqc", "bqc"), (D,), P["gqc"], 1e-6)
    kc = F.rms_norm(lin(ctx, "wkc", "bkc"), (D,), P["gkc"], 1e-6)
    x2 = x1 + lin(attn(qc, kc, lin(ctx, "wvc", "bvc")), "woc", "boc")
    b = F.layer_norm(x2, (D,), eps=1e-6) * (1 + mod[4]) + mod[3]
    f = lin(F.gelu(lin(b, "w1", "b1"), approximate="tanh"), "w2", "b2")
    return (x2 + mod[5] * f).numpy()


def test_block_all_selected_equals_torch_dense():
    p = synth.make_wan_block_weights(W)
    _, x = synth.make_latents(W)
    ctx = synth.make_context(W, 7)
    got = OW.block_partial(p, x, ctx, np.arange(W.L), W.H, W.grid)
    want = _torch_dense(p, x, ctx, W.H, W.grid)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-11)


def test_rows_are_independent():
    # a selected token's output does not depend on which other tokens are selected
    p = synth.make_wan_block_weights(W)
    _, x = synth.make_latents(W)
    ctx = synth.make_context(W, 5)
    full = OW.block_partial(p, x, ctx, np.arange(W.L), W.H, W.grid)
    idx = np.array([0, 3, 17, 18, W.L - 1])
    assert np.allclose(OW.block_partial(p, x, ctx, idx, W.H, W.grid), full[idx], rtol=1e-12, atol=1e-13)


def test_batch_elements_are_independent():
    # classifier-free guidance: same tokens, different contexts
    p = synth.make_wan_block_weights(W)
    _, x = synth.make_latents(W)
    c0, c1 = synth.make_context(W, 6, element=0), synth.make_context(W, 6, element=1)
    idx = np.array([1, 2, 30])
    y0, y1 = OW.batch_partial(p, [x, x], [c0, c1], [idx, idx], W.H, W.grid)
    assert np.allclose(y0, OW.block_partial(p, x, c0, idx, W.H, W.grid), rtol=0, atol=0)
    assert np.allclose(y1, OW.block_partial(p, x, c1, idx, W.H, W.grid), rtol=0, atol=0)
    assert not np.allclose(y0, y1)
