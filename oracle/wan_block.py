"""Oracle: the Wan-style block on the restricted-query path -- qk RMSNorm, 3D
rotary position embedding, a cross-attention sub-layer over a context, and a
batch of two for classifier-free guidance (the block extras of the Wan2.2-S2V
family the paper evaluates, Sec. 4; the caching of Sec. 3.3 is unchanged:
queries and the FFN for the selected tokens, keys and values from all).

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

The paper describes the block only as attention and FFN computed for the
active tokens.  Readings of the Wan-style block (everything in fp64):

* qk RMSNorm: after its projection, q (selected rows) and k (all rows) are
  normalised over all D channels, z / sqrt(mean(z^2) + eps) * g, g a learned
  [D] vector, eps = 1e-6;
* 3D RoPE, after the RMSNorm, on q (each selected token at its own position)
  and k: token i of a T x gh x gw latent grid sits at (t, r, c) =
  (i // (gh gw), (i // gw) % gh, i % gw).  The dh channels of a head form dh/2
  consecutive pairs (2j, 2j + 1); the first nt = dh/2 - 2 (dh // 6) pairs turn
  with t, the next dh // 6 with r, the last dh // 6 with c (22 / 21 / 21 for
  dh = 128); an axis with n pairs has frequencies base^(-j / n), j < n,
  base = 10000, and pair (a, b) at angle phi becomes
  (a cos phi - b sin phi, a sin phi + b cos phi);
* cross-attention, after the self-attention residual: c = LN(x1) g3 + b3
  (LN with affine parameters), qc = RMSNorm(c Wqc^T + bqc) gqc for the
  selected rows, kc = RMSNorm(ctx Wkc^T + bkc) gkc and vc = ctx Wvc^T + bvc
  for all Lc context rows, x2 = x1 + attn(qc, kc, vc) Woc^T + boc (no gate, no
  RoPE);
* the FFN runs on x2 as in the plain block (LN2 modulated by shift2 / scale2,
  gate2);
* B = 2 (classifier-free guidance): the batch elements share the weights and
  have their own tokens, context and selection; a batch is B independent
  blocks.
"""
from __future__ import annotations

import numpy as np

from oracle.block import LN_EPS, _f64, attention, gelu_tanh, layer_norm, linear

RMS_EPS = 1e-6
ROPE_BASE = 10000.0


def rms_norm(z, g, eps: float = RMS_EPS):
    z = np.asarray(z, np.float64)
    return z / np.sqrt((z * z).mean(axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def rope_split(dh: int):
    """(pairs on t, pairs on r, pairs on c)."""
    n_hw = dh // 6
    return dh // 2 - 2 * n_hw, n_hw, n_hw


def token_positions(rows, grid):
    """(t, r, c) of the token indices `rows` of a T x gh x gw grid."""
    gh, gw = grid
    rows = np.asarray(rows, np.int64)
    return rows // (gh * gw), (rows // gw) % gh, rows % gw


def rope_angles(rows, grid, dh: int, base: float = ROPE_BASE):
    """Angles [len(rows), dh/2] of the pairs of one head."""
    t, r, c = token_positions(rows, grid)
    out = []
    for pos, n in zip((t, r, c), rope_split(dh)):
        freq = base ** (-np.arange(n, dtype=np.float64) / n)
        out.append(pos[:, None].astype(np.float64) * freq[None, :])
    return np.concatenate(out, axis=1)


def apply_rope(z, rows, grid, H: int, base: float = ROPE_BASE):
    """Rotate the channel pairs of every head of z [M, D] (rows = token indices)."""
    z = np.asarray(z, np.float64)
    M, D = z.shape
    dh = D // H
    ang = rope_angles(rows, grid, dh, base)
    cs, sn = np.cos(ang), np.sin(ang)
    out = np.empty_like(z)
    for h in range(H):
        a = z[:, h * dh:(h + 1) * dh:2]
        b = z[:, h * dh + 1:(h + 1) * dh:2]
        out[:, h * dh:(h + 1) * dh:2] = a * cs - b * sn
        out[:, h * dh + 1:(h + 1) * dh:2] = a * sn + b * cs
    return out


def block_partial(params: dict, x, ctx, idx, H: int, grid, eps: float = LN_EPS) -> np.ndarray:
    """Wan-style block output for the selected rows idx of one batch element:
    y_sel [len(idx), D] fp64.  x [L, D] tokens, ctx [Lc, D] context."""
    p = _f64(params)
    x = np.asarray(x, np.float64)
    ctx = np.asarray(ctx, np.float64)
    idx = np.asarray(idx, np.int64)
    L = x.shape[0]
    mod = p["mod"]
    a = layer_norm(x, eps) * (1.0 + mod[1]) + mod[0]
    q = apply_rope(rms_norm(linear(a[idx], p["wq"], p["bq"]), p["gq"]), idx, grid, H)
    k = apply_rope(rms_norm(linear(a, p["wk"], p["bk"]), p["gk"]), np.arange(L), grid, H)
    v = linear(a, p["wv"], p["bv"])
    x1 = x[idx] + mod[2] * linear(attention(q, k, v, H), p["wo"], p["bo"])
    c = layer_norm(x1, eps) * p["g3"] + p["b3"]
    qc = rms_norm(linear(c, p["wqc"], p["bqc"]), p["gqc"])
    kc = rms_norm(linear(ctx, p["wkc"], p["bkc"]), p["gkc"])
    vc = linear(ctx, p["wvc"], p["bvc"])
    x2 = x1 + linear(attention(qc, kc, vc, H), p["woc"], p["boc"])
    b = layer_norm(x2, eps) * (1.0 + mod[4]) + mod[3]
    f = linear(gelu_tanh(linear(b, p["w1"], p["b1"])), p["w2"], p["b2"])
    return x2 + mod[5] * f


def batch_partial(params: dict, xs, ctxs, idxs, H: int, grid, eps: float = LN_EPS):
    """A batch (e.g. the conditional and unconditional halves of classifier-free
    guidance): the list of per-element outputs."""
    return [block_partial(params, x, c, i, H, grid, eps) for x, c, i in zip(xs, ctxs, idxs)]
