"""GPU parity of the step schedule and the block stack (Sec. 3.1 Eq. 1/2,
Sec. 3.3 step-latent scheduling): the two halves of the selection against
the whole, and stacks of cached blocks over multi-step trajectories against
the oracle (schedule decisions exact, outputs within the block tolerance
times the number of stacked blocks)."""
import numpy as np
import pytest
import torch

import synth
from oracle import select as OS
from oracle.schedule import Schedule, stack_trajectory
from paper_2608_02474_amd import api

from gpu_util import (TOL_BF16_ABS, TOL_BF16_REL_L2, TOL_F32_ABS, device, down, params_to_device, say,
                      tdtype, up)

pytestmark = pytest.mark.gpu

RAGGED = synth.Workload("ragged_bf16_300tok", T=3, grid=(10, 10), D=256, H=2, F=512,
                        n_samples=4000, ratio=0.37, dtype="bf16", audio="bursts", seed=21)


@pytest.mark.parametrize("w", [synth.SMALL, synth.WAN14B_480P], ids=lambda w: w.name)
def test_saliency_then_topk_is_select(w):
    xref, x = synth.make_latents(w)
    audio = synth.make_audio(w.audio, w.n_samples, w.sample_rate, w.seed)
    dt = tdtype(w.dtype)
    X, XR = up(x, dt), up(xref, dt)
    _, _, fw = api.energy(up(audio), w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
    whole = api.select(X, XR, fw, w.N, k=w.K)
    a = {n: down(getattr(whole, n)).copy() for n in ("idx", "mask", "n_sel_dev", "saliency", "step_delta")}
    half = api.saliency(X, XR, fw, w.N)
    api.topk(half, w.N, w.D, dt, k=w.K)
    torch.cuda.synchronize()
    for n, v in a.items():
        got = down(getattr(half, n))
        if n == "idx":          # only the first K entries are written
            got, v = got[:w.K], v[:w.K]
        assert np.array_equal(got.view(np.uint8), v.view(np.uint8)), n


def _trajectory(w, steps, seed=7):
    rng = np.random.default_rng(seed)
    from oracle.cache import cast_act
    x = rng.standard_normal((w.L, w.D)).astype(np.float32)
    out = []
    for t in range(steps):
        out.append(cast_act(x, w.dtype))
        x = (x + rng.standard_normal(x.shape) * (0.3 / (t + 1))).astype(np.float32)
    return out


def _stack_case(w, n_blocks, steps, sched: Schedule):
    blocks = [synth.make_block_weights(w.with_(seed=w.seed + 100 * b)) for b in range(n_blocks)]
    xs = _trajectory(w, steps)
    fw = np.linspace(0.3, 1.0, w.T).astype(np.float32)
    want = stack_trajectory(blocks, xs, fw, w.N, w.H, sched, w.dtype)
    dt = tdtype(w.dtype)
    stack = api.BlockStack([params_to_device(p, w.dtype) for p in blocks], w.H, w.L, w.D, device(), dt,
                           api.Scheduler(sched.n_full, sched.r_min, sched.r_max, sched.alpha,
                                         sched.refresh_delta))
    FW = up(fw)
    for t, x in enumerate(xs):
        y = stack.step(up(x, dt), FW, w.N)
        torch.cuda.synchronize()
        k, full, delta = stack.history[-1]
        wk, wfull, wdelta, wy = want[t]
        say(f"stack {w.name} x{n_blocks} step {t}: k={k} full={full} delta={delta:.6g}")
        assert (k, full) == (wk, wfull)
        if t >= sched.n_full:
            assert delta == pytest.approx(wdelta, rel=1e-12)
        got = down(y).astype(np.float64)
        err = np.abs(got - wy)
        mx, rel = float(err.max()), float(np.linalg.norm(got - wy) / np.linalg.norm(wy))
        say(f"  last block output: max|err| {mx:.3e} rel-L2 {rel:.3e}")
        if w.dtype == "f32":
            assert mx <= TOL_F32_ABS * n_blocks
        else:
            assert mx <= TOL_BF16_ABS * n_blocks and rel <= TOL_BF16_REL_L2 * n_blocks
    return stack


def test_stack_f32_schedule():
    w = synth.TINY
    st = _stack_case(w, n_blocks=3, steps=6, sched=Schedule(n_full=2, r_min=0.2, r_max=0.7, alpha=0.6))
    ks = [k for k, _, _ in st.history]
    assert ks[:2] == [w.L, w.L] and all(k < w.L for k in ks[2:])


def test_stack_f32_refresh():
    w = synth.TINY.with_(name="tiny_refresh")
    st = _stack_case(w, n_blocks=2, steps=7,
                     sched=Schedule(n_full=1, r_min=0.25, r_max=0.25, alpha=0.0, refresh_delta=0.15))
    assert any(full for _, full, _ in st.history[1:]), "the Eq. 2 refresh never fired"


def test_stack_bf16():
    _stack_case(RAGGED, n_blocks=3, steps=5, sched=Schedule(n_full=1, r_min=0.2, r_max=0.6, alpha=0.5))
