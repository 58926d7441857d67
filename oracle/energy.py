"""Oracle: audio energy anchor (Sec. 3.3, "Cross-modal Saliency Anchors").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

The paper splits the audio S evenly into T temporal segments, takes an STFT of
each segment and uses the L2 norm of each segment's time-frequency matrix as
that segment's energy.  Readings of what the paper leaves open:

* segment t covers samples [floor(t n / T), floor((t+1) n / T));
* STFT: periodic Hann window of n_fft samples, hop `hop`, no centring or
  padding; a segment shorter than n_fft is zero-padded to one frame;
  one-sided spectrum k = 0 .. n_fft/2;
* "L2 norm of the time-frequency matrix" = Frobenius norm of the complex
  STFT, e_t = sqrt(sum_{f,k} |X_t[f,k]|^2);
* per-band energies partition the one-sided bins into n_bands bands of equal
  width on the mel scale mel(f) = 2595 log10(1 + f / 700); bin k belongs to
  band floor(mel(k sr / n_fft) / (mel(sr/2) / n_bands)), the Nyquist bin to
  the last band.  The bands partition the bins, so sum_b E[t,b] = e_t^2;
* the per-frame weight is e_t / max_u e_u (all ones for an all-silent clip).

The DFT is evaluated directly from its definition in fp64 (no FFT), and the
outputs are rounded to fp32 once, at the end.
"""
from __future__ import annotations

import numpy as np


def segment_bounds(n_samples: int, T: int):
    """[start, end) of each of the T even segments."""
    return [((t * n_samples) // T, ((t + 1) * n_samples) // T) for t in range(T)]


def periodic_hann(n_fft: int) -> np.ndarray:
    n = np.arange(n_fft, dtype=np.float64)
    return 0.5 - 0.5 * np.cos(2.0 * np.pi * n / n_fft)


def frame_count(seg_len: int, n_fft: int, hop: int) -> int:
    if seg_len < n_fft:
        return 1
    return 1 + (seg_len - n_fft) // hop


def dft_matrix(n_fft: int) -> np.ndarray:
    """W[n, k] = exp(-2 pi i k n / n_fft) for k = 0..n_fft/2; the angle is
    reduced exactly (k n mod n_fft) before the trigonometric call."""
    n = np.arange(n_fft, dtype=np.int64)[:, None]
    k = np.arange(n_fft // 2 + 1, dtype=np.int64)[None, :]
    ang = 2.0 * np.pi * ((n * k) % n_fft).astype(np.float64) / n_fft
    return np.cos(ang) - 1j * np.sin(ang)


def stft_segment(seg: np.ndarray, n_fft: int, hop: int) -> np.ndarray:
    """One-sided STFT of one segment, [frames, n_fft/2 + 1] complex128."""
    seg = np.asarray(seg, dtype=np.float64)
    nf = frame_count(len(seg), n_fft, hop)
    if len(seg) < n_fft:
        seg = np.concatenate([seg, np.zeros(n_fft - len(seg))])
    w = periodic_hann(n_fft)
    frames = np.stack([seg[f * hop: f * hop + n_fft] * w for f in range(nf)])
    return frames @ dft_matrix(n_fft)


def mel(f):
    return 2595.0 * np.log10(1.0 + np.asarray(f, dtype=np.float64) / 700.0)


def band_of_bins(sr: int, n_fft: int, n_bands: int) -> np.ndarray:
    """Band index of each one-sided bin (mel partition described above)."""
    k = np.arange(n_fft // 2 + 1)
    width = mel(sr / 2.0) / n_bands
    b = np.floor(mel(k * sr / n_fft) / width).astype(np.int64)
    return np.minimum(b, n_bands - 1)


def energy(audio: np.ndarray, T: int, sr: int = 16000, n_fft: int = 512,
           hop: int = 160, n_bands: int = 8):
    """Per-segment audio energy.

    Returns (band_energy [T, n_bands], frame_energy [T], frame_weight [T]),
    all fp32: band_energy[t, b] = sum of |X_t|^2 over the bins of band b and
    all frames of segment t; frame_energy[t] = e_t (Frobenius norm);
    frame_weight = e / max(e).
    """
    audio = np.asarray(audio, dtype=np.float64)
    bands = band_of_bins(sr, n_fft, n_bands)
    E = np.zeros((T, n_bands), dtype=np.float64)
    for t, (a, b) in enumerate(segment_bounds(len(audio), T)):
        X = stft_segment(audio[a:b], n_fft, hop)
        power = (X.real ** 2 + X.imag ** 2).sum(axis=0)   # per bin, over frames
        for band in range(n_bands):
            E[t, band] = power[bands == band].sum()
    e = np.sqrt(E.sum(axis=1))
    m = e.max() if T > 0 else 0.0
    wgt = e / m if m > 0 else np.ones(T)
    return E.astype(np.float32), e.astype(np.float32), wgt.astype(np.float32)


def total_frames(n_samples: int, T: int, n_fft: int, hop: int) -> int:
    return sum(frame_count(b - a, n_fft, hop) for a, b in segment_bounds(n_samples, T))


