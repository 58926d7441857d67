"""Pins for the energy oracle (Sec. 3.3, saliency anchors): textbook DFT
identities, closed forms for windowed tones, invariants, and the mel band
partition derived independently by the inverse mel formula."""
import json
import os

import numpy as np
import pytest

from oracle import energy as E
import synth


def test_periodic_hann_closed_forms():
    for n in (8, 64, 512):
        w = E.periodic_hann(n)
        assert w[0] == 0.0
        assert w[n // 2] == pytest.approx(1.0, abs=1e-15)
        assert np.allclose(w[1:], w[1:][::-1], atol=1e-15)         # w[n] = w[N - n]
        assert w.sum() == pytest.approx(n / 2, rel=1e-13)           # sum w = N/2
        assert (w ** 2).sum() == pytest.approx(3 * n / 8, rel=1e-13)  # sum w^2 = 3N/8


def test_dft_matches_library_fft():
    rng = np.random.default_rng(0)
    for n in (16, 512):
        frames = rng.standard_normal((5, n))
        ours = frames @ E.dft_matrix(n)
        ref = np.fft.rfft(frames, axis=1)
        assert np.max(np.abs(ours - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_one_sided_parseval():
    rng = np.random.default_rng(1)
    n, hop = 512, 160
    seg = rng.standard_normal(2000)
    X = E.stft_segment(seg, n, hop)
    w = 0.5 - 0.5 * np.cos(2 * np.pi * np.arange(n) / n)
    for f in range(X.shape[0]):
        ws = w * seg[f * hop: f * hop + n]
        lhs = np.sum(np.abs(X[f]) ** 2)
        rhs = (n * np.sum(ws ** 2) + abs(X[f, 0]) ** 2 + abs(X[f, -1]) ** 2) / 2
        assert lhs == pytest.approx(rhs, rel=1e-12)


@pytest.mark.parametrize("k0,phi", [(5, 0.0), (37, 1.1), (100, -2.5), (254, 0.3)])
def test_bin_centred_tone(k0, phi):
    # A cos(2 pi k0 n / N + phi) under a periodic Hann window: |X[k0]| = A N / 4,
    # |X[k0 +- 1]| = A N / 8, nothing else, so the frame energy is 3 (A N)^2 / 32.
    n, A = 512, 0.7
    t = np.arange(n)
    seg = A * np.cos(2 * np.pi * k0 * t / n + phi)
    X = E.stft_segment(seg, n, 160)[0]
    assert abs(X[k0]) == pytest.approx(A * n / 4, rel=1e-12)
    assert abs(X[k0 - 1]) == pytest.approx(A * n / 8, rel=1e-12)
    assert abs(X[k0 + 1]) == pytest.approx(A * n / 8, rel=1e-12)
    assert np.sum(np.abs(X) ** 2) == pytest.approx(3 * (A * n) ** 2 / 32, rel=1e-12)


def test_tone_filling_one_segment():
    # A bin-centred tone that fills segment 1 of 3 and silence elsewhere:
    # e_1^2 = F_1 * 3 (A N)^2 / 32, e_0 = e_2 = 0, weight = [0, 1, 0], and all
    # energy lands in the band holding bins k0 - 1 .. k0 + 1.
    sr, n, hop, T = 16000, 512, 160, 3
    L = 3 * 4000
    k0, A = 60, 0.5                                  # 1875 Hz, band 4 (bins 57..85)
    audio = np.zeros(L)
    a, b = 4000, 8000
    audio[a:b] = A * np.cos(2 * np.pi * k0 * np.arange(b - a) / n)
    Eb, e, wgt = E.energy(audio, T, sr, n, hop, 8)
    nf = 1 + (4000 - 512) // 160
    assert nf == 22
    assert float(e[1]) ** 2 == pytest.approx(nf * 3 * (A * n) ** 2 / 32, rel=1e-6)
    assert e[0] == 0 and e[2] == 0
    assert list(wgt) == [0.0, 1.0, 0.0]
    assert np.argmax(Eb[1]) == 4
    assert Eb[1, 4] == pytest.approx(float(e[1]) ** 2, rel=1e-6)


def test_mel_bands_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "mel_bands_16k_512_8.json")))
    bands = E.band_of_bins(g["sample_rate"], g["n_fft"], g["n_bands"])
    counts = np.bincount(bands, minlength=g["n_bands"])
    assert counts.tolist() == g["bins_per_band"]
    assert [int(np.argmax(bands == b)) for b in range(8)] == g["first_bin_of_band"]


def test_frame_counts_and_segments():
    # 81000 samples in 21 segments: lengths 3857 or 3858, 21 frames each;
    # 8000 samples in 2 segments: 22 frames each.
    b = E.segment_bounds(81000, 21)
    assert b[0] == (0, 3857) and b[-1] == (77142, 81000)
    assert sum(hi - lo for lo, hi in b) == 81000
    assert E.total_frames(81000, 21, 512, 160) == 441
    assert E.total_frames(8000, 2, 512, 160) == 44
    assert E.total_frames(20000, 5, 512, 160) == 110
    assert E.frame_count(100, 512, 160) == 1


def test_energy_invariants():
    audio = synth.make_audio("speech", 20000, 16000, 7)
    Eb, e, w = E.energy(audio, 5)
    # bands partition the bins: sum_b E = e^2
    assert np.allclose(Eb.sum(axis=1), e.astype(np.float64) ** 2, rtol=1e-5)
    # homogeneity: e(c S) = |c| e(S)
    _, e2, w2 = E.energy(-0.5 * audio, 5)
    assert np.allclose(e2, 0.5 * e, rtol=1e-6)
    assert np.allclose(w2, w, rtol=1e-6)
    assert w.max() == 1.0 and (w >= 0).all()
    # silence -> zero energy; an all-silent clip weighs every frame 1
    Eb0, e0, w0 = E.energy(np.zeros(8000), 2)
    assert (Eb0 == 0).all() and (e0 == 0).all() and (w0 == 1).all()


def test_short_segment_zero_padded():
    # a segment shorter than n_fft is zero-padded to one frame
    seg = np.ones(100)
    X = E.stft_segment(seg, 512, 160)
    assert X.shape == (1, 257)
    w = 0.5 - 0.5 * np.cos(2 * np.pi * np.arange(100) / 512)
    assert X[0, 0].real == pytest.approx(w.sum(), rel=1e-12)
