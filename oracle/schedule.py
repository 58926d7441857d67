"""Oracle: step-level cache schedule and a stack of cached blocks over a
denoising trajectory (Sec. 3.1 Eq. 1 and Eq. 2; Sec. 3.3 "Energy-Guided
Step-Latent Cache Scheduling").

TEST INFRASTRUCTURE ONLY: the plain CPU definition the GPU path is checked
against.  Only tests, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path never does.

What the paper states: early denoising steps keep full computation; later
steps recompute a fraction r_t = clip(r_min + alpha * normalized Delta_t,
r_min, r_max) of the latents, Delta_t being the step-level relative change of
Eq. 1, and k_t = ceil(N r_t) latents per temporal position are updated.  The
timestep-level caching it builds on (Eq. 2) refreshes the cache once the
accumulated Delta since the last full computation exceeds a threshold delta.

Readings:

* Delta_t is the Eq. 1 value of the step computed against each token's
  cached input (the step_delta the selection returns);
* the normalization divides Delta_t by the largest Delta seen on the cached
  steps so far (this one included), so normalized Delta is in [0, 1];
* the count is the global K = ceil(r_t L - 1e-9) of the top-K selection;
* the Eq. 2 refresh is optional (delta <= 0 turns it off): a cached step
  whose accumulated Delta since the last full step (its own included)
  exceeds delta is computed in full instead, and the accumulation restarts;
* one selection per step is shared by every block of the stack: it is taken
  on the first block's input; block b's input is block b-1's output;
* in the two-stage form (anchor segments given) the count is per segment,
  k_t = ceil(N r_t - 1e-9), with the normalization and the refresh above.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass
class Schedule:
    n_full: int          # leading full steps
    r_min: float
    r_max: float
    alpha: float
    refresh_delta: float = 0.0   # Eq. 2 threshold delta; <= 0: no refresh


@dataclasses.dataclass
class ScheduleState:
    step: int = 0
    delta_max: float = 0.0
    delta_acc: float = 0.0


def schedule_next(cfg: Schedule, st: ScheduleState, delta_t: float, L: int):
    """Decide the current step: returns (k, full).  delta_t is ignored on the
    leading full steps."""
    step = st.step
    st.step += 1
    if step < cfg.n_full:
        st.delta_acc = 0.0
        return L, True
    st.delta_acc += delta_t
    if cfg.refresh_delta > 0.0 and st.delta_acc > cfg.refresh_delta:
        st.delta_acc = 0.0
        return L, True
    st.delta_max = max(st.delta_max, delta_t)
    dhat = delta_t / st.delta_max if st.delta_max > 0.0 else 0.0
    r = min(max(cfg.r_min + cfg.alpha * dhat, cfg.r_min), cfg.r_max)
    k = min(L, max(0, math.ceil(r * L - 1e-9)))
    return k, False


def stack_trajectory(blocks, inputs, fw, N, H, cfg: Schedule, dtype: str, xi: float = 1e-6,
                     anchors=None, codec: int = 0):
    """Run a stack of cached blocks over a trajectory of first-block inputs.

    blocks: list of block parameter dicts; inputs: list of [L, D] first-block
    inputs, one per denoising step; fw: [T] frame weights.  anchors: None for
    the global token top-K, else a [T] segment mask for the two-stage
    selection (k_t = ceil(N r_t) tokens per anchor segment, ranked by
    saliency with unit frame weights); codec: the cache codec of
    oracle.variants.  Returns per step (k, full, delta_t, outputs of the last
    block), k being the schedule's count (per segment in the two-stage form)."""
    from oracle import block as OB
    from oracle import select as OS
    from oracle import variants as OV

    L, D = inputs[0].shape
    caches = [OV.empty_codec_cache(L, D) for _ in blocks]
    st = ScheduleState()
    out = []
    for x0 in inputs:
        x0 = np.asarray(x0, np.float32)
        # Eq. 1 on the first block's input against its cache
        w = fw if anchors is None else np.ones(L // N, np.float32)
        s, num, den = OS.saliency(x0, caches[0][0], w, N, xi)
        delta_t = OS.step_delta(num, den, xi)
        if anchors is None:
            k, full = schedule_next(cfg, st, delta_t, L)
            idx = np.arange(L) if full else OS.select_topk(s, k)
        else:
            k, full = schedule_next(cfg, st, delta_t, N)
            idx = np.arange(L) if full else OV.select_segments(s, anchors, N, k)
        x = x0
        for i, p in enumerate(blocks):
            y_sel = (OB.block_partial(p, x, idx, H).astype(np.float32) if len(idx)
                     else np.zeros((0, D), np.float32))
            y, *caches[i] = OV.cache_update_codec(codec, x, idx, y_sel, *caches[i], dtype)
            x = y
        out.append((k, full, delta_t, x))
    return out
