"""Seeded synthetic inputs for the cached DiT block step.

Both the CPU oracle and the GPU path consume exactly these arrays.  This module
holds no arithmetic of the method itself: it draws audio, latents, weights and
modulation vectors, and rounds inputs to the storage precision (bf16, round to
nearest even) so that both sides see identical values.

Every draw uses ``np.random.default_rng([seed, stream, ...])`` with a fixed
stream number per tensor family, so any tensor can be regenerated on its own.
Large matrices are drawn in fixed blocks of rows, each block from its own
generator ``[seed, stream, sub, block]``, so the values do not depend on how
many threads fill them.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import Workload

STREAM_WEIGHTS, STREAM_BIAS, STREAM_MOD, STREAM_XREF, STREAM_DRIFT, STREAM_AUDIO = 1, 2, 3, 4, 5, 6
STREAM_WAN, STREAM_CONTEXT = 7, 8


def _rng(seed: int, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.default_rng([seed, stream, sub])


_BLOCK_ROWS = 1024
_THREADS = min(16, os.cpu_count() or 1)


def _normal_rows(seed: int, stream: int, sub: int, shape, scale: float = 1.0,
                 dtype: str | None = None) -> np.ndarray:
    """scale * N(0, 1) of `shape` (rows x cols), optionally storage-rounded,
    drawn in blocks of _BLOCK_ROWS rows (block b from [seed, stream, sub, b])."""
    rows = shape[0]
    cols = int(np.prod(shape[1:])) if len(shape) > 1 else 1
    out = np.empty((rows, cols), dtype=np.float32)

    def fill(b):
        r0, r1 = b * _BLOCK_ROWS, min(rows, (b + 1) * _BLOCK_ROWS)
        g = np.random.default_rng([seed, stream, sub, b])
        blk = g.standard_normal((r1 - r0, cols), dtype=np.float32)
        if scale != 1.0:
            blk *= np.float32(scale)
        out[r0:r1] = storage_round(blk, dtype) if dtype else blk

    nb = -(-rows // _BLOCK_ROWS)
    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(fill, range(nb)))
    return out.reshape(shape)


# ---------------------------------------------------------------- bf16 storage

def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even.  Used only
    to put inputs into their storage precision."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    # wraps only for negative NaN patterns, which are overwritten below
    r = ((u + np.uint32(0x7FFF) + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def storage_round(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round an fp32 array to what the device stores (fp32 or bf16), returned
    as fp32 values."""
    a = np.asarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype == "bf16":
        return bf16_bits_to_f32(to_bf16_bits(a))
    raise ValueError(dtype)


# ---------------------------------------------------------------------- audio

def _raised_cos_env(n: int, edge: int) -> np.ndarray:
    env = np.ones(n)
    e = min(edge, n // 2)
    if e > 0:
        ramp = 0.5 - 0.5 * np.cos(np.pi * np.arange(e) / e)
        env[:e] = ramp
        env[n - e:] = ramp[::-1]
    return env


def _burst(rng, n, sr, speech: bool) -> np.ndarray:
    t = np.arange(n) / sr
    f0 = rng.uniform(90.0, 250.0)
    if speech:
        inst = f0 * (1.0 + 0.1 * np.sin(2 * np.pi * 0.5 * t))
        phase0 = 2 * np.pi * np.cumsum(inst) / sr
    else:
        phase0 = 2 * np.pi * f0 * t
    sig = np.zeros(n)
    for h in range(1, 7):
        sig += np.cos(h * phase0 + rng.uniform(0, 2 * np.pi)) / h
    am_rate = rng.uniform(4.0, 5.0) if speech else rng.uniform(3.0, 6.0)
    sig *= 1.0 - 0.5 * (0.5 - 0.5 * np.cos(2 * np.pi * am_rate * t))
    if speech:
        # fricative-like noise bursts of 30-80 ms at level 0.1
        n_fric = rng.integers(0, 3)
        for _ in range(int(n_fric)):
            ln = int(rng.uniform(0.03, 0.08) * sr)
            if ln >= n:
                continue
            s0 = int(rng.integers(0, n - ln))
            noise = rng.standard_normal(ln)
            noise = np.convolve(noise, np.ones(4) / 4, mode="same")
            sig[s0:s0 + ln] += 0.1 * noise * _raised_cos_env(ln, ln // 4)
    sig *= _raised_cos_env(n, int(0.02 * sr))
    peak = np.max(np.abs(sig))
    if peak > 0:
        sig *= rng.uniform(0.2, 1.0) / peak
    return sig


def make_audio(profile: str, n_samples: int, sr: int, seed: int) -> np.ndarray:
    """Synthetic mono audio in [-1, 1], fp32.

    bursts        amplitude-modulated harmonic bursts (6 harmonics, 1/h) of
                  0.15-0.5 s separated by exact-zero silences of 0.05-0.35 s
    speech        bursts with an f0 glide, syllable-rate AM, fricative noise
                  and pauses of 0.1-0.4 s
    noise         white noise N(0, 0.1^2): flat energy
    half_silence  exact zeros for the first half, speech after
    """
    rng = _rng(seed, STREAM_AUDIO)
    if profile == "noise":
        return np.clip(0.1 * rng.standard_normal(n_samples), -1, 1).astype(np.float32)
    if profile == "half_silence":
        a = make_audio("speech", n_samples, sr, seed)
        a[: n_samples // 2] = 0.0
        return a
    speech = profile == "speech"
    if profile not in ("bursts", "speech"):
        raise ValueError(profile)
    out = np.zeros(n_samples)
    pos = 0
    while pos < n_samples:
        burst = int(rng.uniform(0.15, 0.5) * sr)
        b = _burst(rng, min(burst, n_samples - pos), sr, speech)
        out[pos:pos + len(b)] = b
        pos += len(b)
        gap = rng.uniform(0.1, 0.4) if speech else rng.uniform(0.05, 0.35)
        pos += int(gap * sr)
    return np.clip(out, -1, 1).astype(np.float32)


# -------------------------------------------------------------------- latents

def make_latents(w: Workload, seed: int | None = None):
    """(xref, x): the cached block input and the current step's block input,
    [L, D] fp32 holding storage-rounded values.

    xref ~ N(0, 1); x = xref + sigma_f * N(0, 1) with one sigma_f ~ U(0.01, 0.3)
    per latent frame, so frames drift by different amounts.
    """
    seed = w.seed if seed is None else seed
    xref = _normal_rows(seed, STREAM_XREF, 0, (w.L, w.D))
    sigma = _rng(seed, STREAM_DRIFT).uniform(0.01, 0.3, size=w.T).astype(np.float32)
    x = _normal_rows(seed, STREAM_DRIFT, 1, (w.L, w.D))
    row_sigma = np.repeat(sigma, w.N)[:, None]

    def mix(b):
        r0, r1 = b * _BLOCK_ROWS, min(w.L, (b + 1) * _BLOCK_ROWS)
        x[r0:r1] = storage_round(xref[r0:r1] + row_sigma[r0:r1] * x[r0:r1], w.dtype)
        xref[r0:r1] = storage_round(xref[r0:r1], w.dtype)

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(mix, range(-(-w.L // _BLOCK_ROWS))))
    return xref, x


def make_block_weights(w: Workload, seed: int | None = None, gate_mean=None,
                       gate_std=None) -> dict:
    """DiT block parameters in nn.Linear layout ([out, in]).

    Linear weights and biases ~ N(0, 0.02); modulation rows (shift1, scale1,
    gate1, shift2, scale2, gate2): shifts and scales ~ N(0, 0.1), gates
    ~ N(gate_mean, gate_std).  Weights, biases and modulation are rounded to
    the storage dtype (modulation stays fp32 on the device but is rounded the
    same way so both sides see one value).
    """
    seed = w.seed if seed is None else seed
    gm = w.gate_mean if gate_mean is None else gate_mean
    gs = w.gate_std if gate_std is None else gate_std
    D, F = w.D, w.F
    shapes = {"wq": (D, D), "wk": (D, D), "wv": (D, D), "wo": (D, D),
              "w1": (F, D), "w2": (D, F)}
    out = {}
    for i, (k, shp) in enumerate(shapes.items()):
        out[k] = _normal_rows(seed, STREAM_WEIGHTS, i, shp, scale=0.02, dtype=w.dtype)
    bshapes = {"bq": D, "bk": D, "bv": D, "bo": D, "b1": F, "b2": D}
    for i, (k, n) in enumerate(bshapes.items()):
        r = _rng(seed, STREAM_BIAS, i)
        out[k] = storage_round(0.02 * r.standard_normal(n, dtype=np.float32), w.dtype)
    r = _rng(seed, STREAM_MOD)
    mod = np.empty((6, D), dtype=np.float32)
    for row in range(6):
        if row in (2, 5):
            mod[row] = gm + gs * r.standard_normal(D)
        else:
            mod[row] = 0.1 * r.standard_normal(D)
    out["mod"] = storage_round(mod, w.dtype)
    return out


def random_frame_weight(T: int, seed: int) -> np.ndarray:
    """Arbitrary per-frame weights in [0, 1] (for selection tests that do not
    go through the audio path)."""
    return _rng(seed, 99).uniform(0.0, 1.0, size=T).astype(np.float32)


def random_anchor_keys(T: int, seed: int) -> np.ndarray:
    """Uniform [0, 1) keys, one per segment: the random draw behind the Random
    anchor strategy (its k anchors are the k largest keys)."""
    return _rng(seed, 98).uniform(0.0, 1.0, size=T).astype(np.float32)


def make_wan_block_weights(w: Workload, seed: int | None = None) -> dict:
    """The plain block parameters plus the Wan-style extras: cross-attention
    projections wqc, wkc, wvc, woc [D, D] and biases ~ N(0, 0.02); RMSNorm
    weights gq, gk, gqc, gkc and the cross-attention LN scale g3 ~ N(1, 0.1);
    the LN shift b3 ~ N(0, 0.02).  The extras are fp32 vectors on the device
    (rounded to the storage dtype like the modulation)."""
    seed = w.seed if seed is None else seed
    out = make_block_weights(w, seed)
    D = w.D
    for i, k in enumerate(("wqc", "wkc", "wvc", "woc")):
        out[k] = _normal_rows(seed, STREAM_WAN, i, (D, D), scale=0.02, dtype=w.dtype)
    r = _rng(seed, STREAM_WAN, 10)
    for k in ("bqc", "bkc", "bvc", "boc"):
        out[k] = storage_round(0.02 * r.standard_normal(D, dtype=np.float32), w.dtype)
    for k in ("gq", "gk", "gqc", "gkc", "g3"):
        out[k] = storage_round((1.0 + 0.1 * r.standard_normal(D)).astype(np.float32), w.dtype)
    out["b3"] = storage_round((0.02 * r.standard_normal(D)).astype(np.float32), w.dtype)
    return out


def make_context(w: Workload, Lc: int, seed: int | None = None, element: int = 0) -> np.ndarray:
    """Context tokens [Lc, D] ~ N(0, 1) (text / audio embeddings after their
    input projection), storage-rounded; `element` picks the batch element."""
    seed = w.seed if seed is None else seed
    return _normal_rows(seed, STREAM_CONTEXT, element, (Lc, w.D), dtype=w.dtype)
