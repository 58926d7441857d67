"""Algorithmic work of each kernel of the cached block step, and MI355X peaks.

Algorithmic = what the method must compute or move, not what a kernel happens
to re-read: FLOPs for the contractions, HBM bytes for the streaming kernels.
Symbols: L tokens, K recomputed tokens, U = L - K, D hidden, F FFN width,
b activation bytes (2 for bf16, 4 for fp32).
"""
from __future__ import annotations

# MI355X published peaks.  bf16 dense MFMA = 256 CU x 2.4 GHz x 4096 flop/clk.
PEAK_BF16_TFLOPS = 2516.6
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def kernel_work(L: int, K: int, D: int, F: int, b: int, n_samples: int = 0):
    """{kernel name prefix: (amount per launch, "flop" | "byte")}.

    The names are the ones the library records for each launch; GEMMs are
    named after their call site (q, kv, o, ffn_up, ffn_down).
    """
    U = L - K
    return {
        # saliency: read x and xref, write s, num, den
        "saliency_rows": (2 * L * D * b + 20 * L, "byte"),
        # selection: a few passes over 4-byte keys (latency-bound); write idx, mask
        "select_rows": (4 * L + 4 * K + L, "byte"),
        "select_segments": (4 * L + 4 * K + L, "byte"),
        # LN1 over all rows: read x, write a
        "modln_in": (2 * L * D * b, "byte"),
        "gemm_q": (2 * K * D * D, "flop"),
        "gemm_kv": (4 * L * D * D, "flop"),
        "attn_fwd": (4 * K * L * D, "flop"),
        "gemm_o": (2 * K * D * D, "flop"),
        # LN2 over the recomputed rows: read x1 (fp32), write b
        "modln_x1": (K * D * (4 + b), "byte"),
        "gemm_ffn_up": (2 * K * D * F, "flop"),
        "gemm_ffn_down": (2 * K * F * D, "flop"),
        # 16-bit output cache: fresh rows read y_sel and x, write y, xref and the
        # stored row; reused rows copy their stored row to y; plus the mask
        "cache_update_full": (K * D * (4 + 4 * b) + U * D * 2 * b + L, "byte"),
        # naive int8: as the residual cache, but reused rows read no reference
        "cache_update_naive": (K * D * (4 + b + b + 1 + b) + U * D * (1 + b) + 4 * L + L, "byte"),
        # cache update: fresh rows read y_sel (fp32) and x, write xref, codes, y;
        # reused rows read xref and codes and write y; plus scale and mask
        "cache_update": (K * D * (4 + b + b + 1 + b) + U * D * (b + 1 + b) + 4 * L + L, "byte"),
        # energy: read the audio once (latency-bound, once per clip)
        "energy_frames": (4 * n_samples, "byte"),
        "energy_reduce": (0, "byte"),
    }


def work_of(name: str, table: dict):
    for prefix, v in table.items():
        if name.startswith(prefix):
            return v
    return None


def block_flops(L: int, K: int, D: int, F: int) -> int:
    return 2 * K * D * D + 4 * L * D * D + 4 * K * L * D + 2 * K * D * D + 4 * K * D * F


def wan_block_work(B: int, L: int, K: int, D: int, F: int, Lc: int, b: int):
    """Work per launch of the Wan-style block's kernels for a batch of B
    elements with K selected tokens each and Lc context rows: {name prefix:
    (amount per launch, kind)}.  The GEMMs run once over the whole batch;
    attention runs once per element; qk_norm_rope runs four times (q, k, the
    cross-attention q and k), given as the mean of the four."""
    n = B * K
    norm_bytes = (2 * n + B * L + B * Lc) * D * 2 * b // 4
    return {
        "qk_norm_rope": (norm_bytes, "byte"),
        "gemm_qc": (2 * n * D * D, "flop"),
        "gemm_kvc": (4 * B * Lc * D * D, "flop"),
        "gemm_oc": (2 * n * D * D, "flop"),
        "attn_cross": (4 * K * Lc * D, "flop"),
        "gemm_q": (2 * n * D * D, "flop"),
        "gemm_kv": (4 * B * L * D * D, "flop"),
        "attn_fwd": (4 * K * L * D, "flop"),
        "gemm_o": (2 * n * D * D, "flop"),
        "modln_in": (2 * B * L * D * b, "byte"),
        "modln_x1": (n * D * (4 + b), "byte"),
        "gemm_ffn_up": (2 * n * D * F, "flop"),
        "gemm_ffn_down": (2 * n * F * D, "flop"),
    }


def wan_block_flops(B: int, L: int, K: int, D: int, F: int, Lc: int) -> int:
    return B * (block_flops(L, K, D, F) + 4 * K * D * D + 4 * Lc * D * D + 4 * K * Lc * D)
