"""Helpers shared by the GPU parity tests: device uploads of the seeded
synthetic inputs and the comparison rules.

Tolerances (block outputs, compared on fp32 y_sel):
  fp32 path: max |gpu - oracle| <= 1e-5;
  bf16 path: max |gpu - oracle| <= 2e-2 and ||gpu - oracle||_2 / ||oracle||_2 <= 1e-2.
Selections must match exactly except tokens whose saliency lies within 1e-6
(relative) of the K-th saliency.
"""
import sys

import numpy as np
import torch

TOL_F32_ABS = 1e-5
TOL_BF16_ABS = 2e-2
TOL_BF16_REL_L2 = 1e-2
TIE_REL = 1e-6


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def device():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm device")
    return torch.device("cuda:0")


def tdtype(dtype: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def up(a: np.ndarray, dtype=None, dev=None):
    """Upload a numpy array; storage-rounded fp32 values convert exactly to bf16."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(dev or device())


def params_to_device(p: dict, dtype: str, dev=None) -> dict:
    out = {}
    for k, v in p.items():
        out[k] = up(v, torch.float32 if k == "mod" else tdtype(dtype), dev)
    return out


def down(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


def check_block(got: np.ndarray, want: np.ndarray, dtype: str, what: str = "y_sel"):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - want)
    mx = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30)) if err.size else 0.0
    say(f"  {what}: max|err| {mx:.3e}  rel-L2 {rel:.3e}  ({got.shape[0]} rows)")
    if dtype == "f32":
        assert mx <= TOL_F32_ABS, f"{what}: max abs error {mx} > {TOL_F32_ABS}"
    else:
        assert mx <= TOL_BF16_ABS, f"{what}: max abs error {mx} > {TOL_BF16_ABS}"
        assert rel <= TOL_BF16_REL_L2, f"{what}: relative L2 error {rel} > {TOL_BF16_REL_L2}"
    return mx, rel


def check_selection(got_idx: np.ndarray, want_idx: np.ndarray, s_oracle: np.ndarray, K: int):
    """Exact set match, except tokens tied with the K-th saliency within TIE_REL."""
    got = set(np.asarray(got_idx).tolist())
    want = set(np.asarray(want_idx).tolist())
    assert len(got) == len(got_idx) == K, "selected indices must be distinct and number K"
    assert list(got_idx) == sorted(got_idx), "indices must be ascending"
    diff = got ^ want
    if not diff:
        return 0
    kth = float(np.sort(s_oracle.astype(np.float64))[::-1][K - 1])
    for i in diff:
        assert abs(float(s_oracle[i]) - kth) <= TIE_REL * max(abs(kth), 1e-30), (
            f"token {i} differs (s={s_oracle[i]}, K-th={kth})")
    return len(diff)
