"""Workload shapes for the cached DiT block step.

Each workload is a latent video of T frames x (h x w) spatial tokens, a DiT
block of hidden width D with H heads and FFN width F, a clip of 16 kHz audio
and a recompute ratio r.  The 14B-shaped block follows Wan2.2-S2V at 480p
(81 video frames at 16 fps -> 21 latent frames of 30x52 tokens); the 720p
variant has 45x80 tokens per frame (Sec. 4.1 gives the 5 s / 81-frame / 720P
and 480P generation settings).

Nothing here computes any part of the method: these are shapes, seeds and
names only.
"""
from __future__ import annotations

import dataclasses
import math


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int                 # latent frames (temporal segments)
    grid: tuple            # (h, w) spatial latents per frame
    D: int                 # hidden width
    H: int                 # attention heads
    F: int                 # FFN width
    n_samples: int         # audio samples at sample_rate
    ratio: float           # recompute ratio r
    dtype: str             # "f32" or "bf16" activations and weights
    audio: str             # audio profile name (see synth.inputs.make_audio)
    seed: int
    sample_rate: int = 16000
    n_fft: int = 512
    hop: int = 160
    n_bands: int = 8
    gate_mean: float = 0.25
    gate_std: float = 0.05

    @property
    def N(self) -> int:
        return self.grid[0] * self.grid[1]

    @property
    def L(self) -> int:
        return self.T * self.N

    @property
    def dh(self) -> int:
        return self.D // self.H

    @property
    def K(self) -> int:
        """Number of recomputed tokens: ceil(r * L) (Sec. 3.3, k_t = ceil(N r_t),
        applied over the whole token sequence)."""
        return min(self.L, max(0, math.ceil(self.ratio * self.L - 1e-9)))

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


TINY = Workload("tiny_fp32_32tok", T=2, grid=(4, 4), D=64, H=2, F=256,
                n_samples=8000, ratio=0.5, dtype="f32", audio="bursts", seed=0)
SMALL = Workload("small_bf16_7800tok", T=5, grid=(30, 52), D=1536, H=12, F=8960,
                 n_samples=20000, ratio=0.25, dtype="bf16", audio="bursts", seed=1)
WAN14B_480P = Workload("wan14b_480p_32760tok", T=21, grid=(30, 52), D=5120, H=40,
                       F=13824, n_samples=81000, ratio=0.4, dtype="bf16",
                       audio="speech", seed=2)
WAN14B_720P = Workload("wan14b_720p_75600tok", T=21, grid=(45, 80), D=5120, H=40,
                       F=13824, n_samples=81000, ratio=0.3, dtype="bf16",
                       audio="speech", seed=4)

SWEEP_RATIOS = (0.1, 0.25, 0.5, 1.0)
SWEEP_AUDIO = ("noise", "speech", "half_silence")


def sweep():
    """The 32760-token block over recompute ratios and audio energy profiles."""
    out = []
    for a in SWEEP_AUDIO:
        for r in SWEEP_RATIOS:
            out.append(WAN14B_480P.with_(name=f"wan14b_480p_r{r}_{a}", ratio=r,
                                         audio=a, seed=3))
    return out


ALL = {w.name: w for w in (TINY, SMALL, WAN14B_480P, WAN14B_720P)}
