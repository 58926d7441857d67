"""Oracle: one DiT block computed only for the selected tokens (Sec. 3.3,
"Fine-grained latent-level caching").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

The paper extracts the active tokens before attention, computes the query
branch for them only, takes keys and values from the complete token set,
runs attention on (Q', K, V), and runs the FFN on the active tokens only.
The block itself is an adaLN-style DiT block (the paper builds on DiT video
generators); its exact form is a reading:

  a   = LN(x) * (1 + scale1) + shift1                        all L rows
  q   = a[idx] Wq^T + bq,  k = a Wk^T + bk,  v = a Wv^T + bv
  o_h = softmax(q_h k_h^T / sqrt(dh)) v_h                    per head h
  x1  = x[idx] + gate1 * (o Wo^T + bo)
  b   = LN(x1) * (1 + scale2) + shift2
  y   = x1 + gate2 * (GELU_tanh(b W1^T + b1) W2^T + b2)

LN has no affine parameters, biased variance and eps = 1e-6; the modulation
rows are (shift1, scale1, gate1, shift2, scale2, gate2), broadcast over tokens.
Everything is fp64; weights are [out, in] (nn.Linear layout).  The partial
block's functions also take `dt`, the floating type they compute in: fp64 for
every parity check, fp32 only to time the same steps with single-precision
BLAS on the host.
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-6


def layer_norm(z: np.ndarray, eps: float = LN_EPS, dt=np.float64) -> np.ndarray:
    z = np.asarray(z, dtype=dt)
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return (z - mu) / np.sqrt(var + eps)


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def linear(a: np.ndarray, w: np.ndarray, b: np.ndarray, dt=np.float64) -> np.ndarray:
    return np.asarray(a, dt) @ np.asarray(w, dt).T + np.asarray(b, dt)


def _f64(p: dict, dt=np.float64) -> dict:
    return {k: np.asarray(v, dtype=dt) for k, v in p.items()}


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, H: int,
              chunk: int = 1024, dt=np.float64) -> np.ndarray:
    """Multi-head attention of the rows of q over all rows of k, v.

    q [M, D], k and v [L, D]; head h uses columns h*dh .. (h+1)*dh.  The query
    rows are processed in chunks so that the M x L score matrix is never
    materialised at once.
    """
    M, D = q.shape
    dh = D // H
    out = np.empty((M, D), dtype=dt)
    scale = dt(1.0 / np.sqrt(dh))
    for h in range(H):
        cols = slice(h * dh, (h + 1) * dh)
        kh, vh = k[:, cols], v[:, cols]
        for c0 in range(0, M, chunk):
            s = (q[c0:c0 + chunk, cols] @ kh.T) * scale
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[c0:c0 + chunk, cols] = p @ vh
    return out


def kv_projection(p: dict, x: np.ndarray, eps: float = LN_EPS, dt=np.float64):
    """Modulated LN of all rows and the key/value projections of all rows."""
    mod = p["mod"]
    a = layer_norm(x, eps, dt) * (1.0 + mod[1]) + mod[0]
    return a, linear(a, p["wk"], p["bk"], dt), linear(a, p["wv"], p["bv"], dt)


def block_partial(params: dict, x: np.ndarray, idx: np.ndarray, H: int,
                  eps: float = LN_EPS, kv=None, dt=np.float64) -> np.ndarray:
    """Block output for the selected rows idx only: y_sel [len(idx), D], fp64.

    `kv` optionally passes a precomputed (a, k, v) from kv_projection for the
    same x, so that several row samples can share the all-row projections.
    """
    p = _f64(params, dt)
    x = np.asarray(x, dtype=dt)
    idx = np.asarray(idx, dtype=np.int64)
    mod = p["mod"]
    a, k, v = kv_projection(p, x, eps, dt) if kv is None else kv
    q = linear(a[idx], p["wq"], p["bq"], dt)
    o = attention(q, k, v, H, dt=dt)
    x1 = x[idx] + mod[2] * linear(o, p["wo"], p["bo"], dt)
    b = layer_norm(x1, eps, dt) * (1.0 + mod[4]) + mod[3]
    f = linear(gelu_tanh(linear(b, p["w1"], p["b1"], dt)), p["w2"], p["b2"], dt)
    return x1 + mod[5] * f


def block_full(params: dict, x: np.ndarray, H: int, eps: float = LN_EPS) -> np.ndarray:
    """The dense block over every row, written without any row selection: the
    reference the partial block must equal when every token is selected."""
    p = _f64(params)
    x = np.asarray(x, dtype=np.float64)
    L, D = x.shape
    dh = D // H
    sh1, sc1, g1, sh2, sc2, g2 = p["mod"]
    h_in = layer_norm(x, eps) * (1.0 + sc1) + sh1
    Q = h_in @ p["wq"].T + p["bq"]
    Kt = h_in @ p["wk"].T + p["bk"]
    V = h_in @ p["wv"].T + p["bv"]
    heads = []
    for h in range(H):
        c = slice(h * dh, (h + 1) * dh)
        logits = Q[:, c] @ Kt[:, c].T / np.sqrt(dh)
        w = np.exp(logits - logits.max(axis=1, keepdims=True))
        heads.append((w / w.sum(axis=1, keepdims=True)) @ V[:, c])
    attn = np.concatenate(heads, axis=1)
    x1 = x + g1 * (attn @ p["wo"].T + p["bo"])
    hid = layer_norm(x1, eps) * (1.0 + sc2) + sh2
    up = hid @ p["w1"].T + p["b1"]
    return x1 + g2 * (gelu_tanh(up) @ p["w2"].T + p["b2"])

