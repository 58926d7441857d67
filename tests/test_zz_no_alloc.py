"""The allocation-free selection entry point (echo_select_noalloc) against
echo_select through the C ABI: identical selected indices, mask, count,
saliency and step-level Eq. 1 value (bit for bit), on consecutive calls that
share the library's static scratch, the second with a smaller input."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_02474_amd import _lib, api

from gpu_util import device, say

pytestmark = pytest.mark.gpu


def _inputs(T, N, D, dtype, seed):
    g = torch.Generator(device=device())
    g.manual_seed(seed)
    xref = torch.randn((T * N, D), device=device(), generator=g)
    sigma = torch.rand((T, 1, 1), device=device(), generator=g) * 0.29 + 0.01
    x = xref + (sigma * torch.randn((T, N, D), device=device(), generator=g)).reshape(T * N, D)
    fw = torch.rand(T, device=device(), generator=g)
    fw[T // 3] = 0.0                                    # a silent frame: exact zero ties
    return x.to(dtype).contiguous(), xref.to(dtype).contiguous(), fw


def _fresh_out(L, want_saliency=True):
    dev = device()
    return api.Selection(idx=torch.full((L,), -7, dtype=torch.int32, device=dev),
                         mask=torch.full((L,), 9, dtype=torch.uint8, device=dev),
                         n_sel_dev=torch.full((1,), -1, dtype=torch.int32, device=dev), n_sel=None,
                         saliency=torch.empty(L, dtype=torch.float32, device=dev) if want_saliency else None,
                         step_delta=torch.empty(1, dtype=torch.float64, device=dev))


def _compare(ref: api.Selection, got: api.Selection, L: int):
    torch.cuda.synchronize()
    n_ref, n_got = int(ref.n_sel_dev[0].item()), int(got.n_sel_dev[0].item())
    assert n_ref == n_got
    assert torch.equal(ref.idx[:n_ref], got.idx[:n_got])
    assert torch.equal(ref.mask[:L], got.mask[:L])
    if ref.saliency is not None and got.saliency is not None:
        assert torch.equal(ref.saliency[:L].view(torch.int32), got.saliency[:L].view(torch.int32))
    assert torch.equal(ref.step_delta.view(torch.int64), got.step_delta.view(torch.int64))
    return n_ref


# (T, N, D, dtype, mode, value): the first call at the 32760-token 14B shape,
# then smaller inputs (the static scratch keeps the larger call's contents)
CASES = [(21, 1560, 5120, torch.bfloat16, "k", 13104),
         (5, 1560, 1536, torch.bfloat16, "k", 1950),
         (3, 100, 256, torch.float32, "threshold", None),
         (2, 16, 64, torch.float32, "k", 16)]


def test_select_noalloc_matches_select_on_consecutive_calls():
    for i, (T, N, D, dt, mode, val) in enumerate(CASES):
        L = T * N
        say(f"select_noalloc case {i}: T={T} N={N} D={D} {dt} {mode}")
        x, xref, fw = _inputs(T, N, D, dt, seed=40 + i)
        kw = {"k": val} if mode == "k" else {"threshold": 0.0}
        if mode == "threshold":
            s = api.select(x, xref, fw, N, k=0).saliency
            kw = {"threshold": float(s.median().item())}
        ref = api.select(x, xref, fw, N, **kw)
        got = api.select_noalloc(x, xref, fw, N, _fresh_out(L), **kw)
        n = _compare(ref, got, L)
        if mode == "k":
            assert n == val
        # without a saliency output the scratch also holds the saliency
        got2 = api.select_noalloc(x, xref, fw, N, _fresh_out(L, want_saliency=False), **kw)
        _compare(ref, got2, L)
        say(f"  ok: {n} selected")


def test_select_noalloc_rejects_above_limit():
    lib = _lib.load()
    # buffers of the full claimed size, so that even a launch would stay in bounds
    T, N = 2, _lib.ECHO_SELECT_NOALLOC_MAX_TOKENS // 2 + 1
    x, xref, fw = _inputs(T, N, 64, torch.float32, seed=3)
    out = _fresh_out(T * N)
    cfg = _lib.SelectCfg(T, N, 64, _lib.ECHO_F32, 4, 0.0, 1e-6)
    st = lib.echo_select_noalloc(ctypes.byref(cfg), x.data_ptr(), xref.data_ptr(), fw.data_ptr(),
                                 out.idx.data_ptr(), out.mask.data_ptr(), out.n_sel_dev.data_ptr(), None, None,
                                 None)
    assert st == _lib.ECHO_ELIMIT
    torch.cuda.synchronize()
    assert (out.idx == -7).all() and (out.mask == 9).all()      # nothing launched
