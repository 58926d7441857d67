"""GPU parity of the Wan-style block (qk RMSNorm, 3D RoPE, cross-attention with
restricted queries, a batch of two for classifier-free guidance) against the
oracle, within the bf16 block tolerance: a ragged small case with unequal
selections per element, an element with every token selected, and the
32760-token shape with a 512-token context in the benchmark's configuration
(sampled rows)."""
import numpy as np
import pytest
import torch

import synth
from oracle import select as OS
from oracle import wan_block as OW
from paper_2608_02474_amd import api

from gpu_util import check_block, device, down, say, tdtype, up

pytestmark = pytest.mark.gpu

FP32_KEYS = ("mod", "gq", "gk", "gqc", "gkc", "g3", "b3")
SMALL = synth.Workload("wan_ragged_bf16_300tok", T=3, grid=(10, 10), D=256, H=2, F=512,
                       n_samples=4000, ratio=0.37, dtype="bf16", audio="bursts", seed=41)


def _params(p, dtype):
    return {k: up(v, torch.float32 if k in FP32_KEYS else tdtype(dtype)) for k, v in p.items()}


def _run(w, p, xs, ctxs, idxs, batch_invariant=False):
    dt = tdtype(w.dtype)
    X = up(np.stack(xs), dt)
    C = up(np.stack(ctxs), dt)
    gidx = np.concatenate([b * w.L + np.asarray(i) for b, i in enumerate(idxs)]).astype(np.int32)
    y = api.wan_block_partial(_params(p, w.dtype), X, C, up(gidx), [len(i) for i in idxs], w.H,
                              (w.T,) + tuple(w.grid), batch_invariant=batch_invariant)
    torch.cuda.synchronize()
    out, o = [], 0
    for i in idxs:
        out.append(down(y)[o:o + len(i)])
        o += len(i)
    return out


def test_wan_block_small_batch_of_two():
    w = SMALL
    p = synth.make_wan_block_weights(w)
    _, x0 = synth.make_latents(w)
    _, x1 = synth.make_latents(w, seed=w.seed + 1)
    ctxs = [synth.make_context(w, 77, element=0), synth.make_context(w, 77, element=1)]
    rng = np.random.default_rng(3)
    idxs = [np.sort(rng.choice(w.L, 111, replace=False)), np.sort(rng.choice(w.L, 97, replace=False))]
    say(f"wan block {w.name} B=2 n_sel=(111, 97) Lc=77 (GPU)")
    got = _run(w, p, [x0, x1], ctxs, idxs)
    want = OW.batch_partial(p, [x0, x1], ctxs, idxs, w.H, w.grid)
    for b in range(2):
        check_block(got[b], want[b], w.dtype, f"{w.name}/element {b}")


def test_wan_block_all_tokens_one_element():
    w = SMALL.with_(name="wan_all_bf16_300tok", seed=42)
    p = synth.make_wan_block_weights(w)
    _, x = synth.make_latents(w)
    ctx = synth.make_context(w, 40)
    idx = np.arange(w.L)
    say(f"wan block {w.name} B=1 all {w.L} tokens (GPU)")
    got = _run(w, p, [x], [ctx], [idx])[0]
    check_block(got, OW.block_partial(p, x, ctx, idx, w.H, w.grid), w.dtype, w.name)


def test_wan_block_full_size_sampled():
    """The 32760-token shape, B = 2 with their own contexts (512 tokens) and
    selections, in the benchmark's launch configuration; the oracle computes
    the all-row projections and then sampled rows."""
    w = synth.WAN14B_480P
    Lc = 512
    p = synth.make_wan_block_weights(w)
    xref, x0 = synth.make_latents(w)
    _, x1 = synth.make_latents(w, seed=w.seed + 7)
    fw = np.linspace(0.2, 1.0, w.T).astype(np.float32)
    s, _, _ = OS.saliency(x0, xref, fw, w.N)
    idx0 = OS.select_topk(s, w.K)
    idx1 = np.sort(np.random.default_rng(5).choice(w.L, w.K, replace=False))
    ctxs = [synth.make_context(w, Lc, element=0), synth.make_context(w, Lc, element=1)]
    say(f"wan block {w.name} B=2 K={w.K} Lc={Lc} (GPU)")
    got = _run(w, p, [x0, x1], ctxs, [idx0, idx1])
    rng = np.random.default_rng(6)
    for b, (x, idx) in enumerate(((x0, idx0), (x1, idx1))):
        rows = np.unique(np.concatenate([[0, w.K - 1], rng.choice(w.K, 14, replace=False)]))
        say(f"wan block {w.name} element {b}: oracle on {len(rows)} sampled rows")
        want = OW.block_partial(p, x, ctxs[b], idx[rows], w.H, w.grid)
        check_block(got[b][rows], want, w.dtype, f"{w.name}/element {b}")
