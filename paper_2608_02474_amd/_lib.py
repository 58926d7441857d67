"""ctypes declarations for libecho.so (the C ABI declared in include/echo.h).

Loading fails loudly if the library has not been built: there is no other
implementation of the path.
"""
from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libecho.so")
HEADER = os.path.join(HERE, "..", "include", "echo.h")

ECHO_OK, ECHO_EINVAL, ECHO_EUNSUPPORTED, ECHO_EWORKSPACE, ECHO_EDEVICE, ECHO_ELIMIT = range(6)
ECHO_SELECT_NOALLOC_MAX_TOKENS = 131072
ECHO_F32, ECHO_BF16 = 0, 1
ECHO_BLOCK_BATCH_INVARIANT = 1
ECHO_ANCHOR_TOPK, ECHO_ANCHOR_UNIFORM = 0, 1
ECHO_CODEC_RESIDUAL_INT8, ECHO_CODEC_FULL, ECHO_CODEC_NAIVE_INT8 = 0, 1, 2

c_int32, c_int64, c_size_t, c_void_p, c_float, c_double = (
    ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float,
    ctypes.c_double)


class EnergyCfg(ctypes.Structure):
    _fields_ = [("T", c_int32), ("sample_rate", c_int32), ("n_fft", c_int32), ("hop", c_int32),
                ("n_bands", c_int32)]


class SelectCfg(ctypes.Structure):
    _fields_ = [("T", c_int32), ("N", c_int32), ("D", c_int32), ("dtype", c_int32),
                ("k", c_int32), ("threshold", c_float), ("xi", c_double)]


class BlockCfg(ctypes.Structure):
    _fields_ = [("L", c_int32), ("D", c_int32), ("H", c_int32), ("F", c_int32),
                ("dtype", c_int32), ("ln_eps", c_float), ("flags", c_int32)]


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("wq", "wk", "wv", "wo", "w1", "w2",
                                        "bq", "bk", "bv", "bo", "b1", "b2", "mod")]


WAN_EXTRA = ("wqc", "wkc", "wvc", "woc", "bqc", "bkc", "bvc", "boc", "gq", "gk", "gqc", "gkc", "g3", "b3")


class WanBlockCfg(ctypes.Structure):
    _fields_ = [("B", c_int32), ("L", c_int32), ("D", c_int32), ("H", c_int32), ("F", c_int32),
                ("Lc", c_int32), ("T", c_int32), ("gh", c_int32), ("gw", c_int32), ("dtype", c_int32),
                ("ln_eps", c_float), ("rms_eps", c_float), ("rope_base", c_double), ("flags", c_int32)]


class WanBlockWeights(ctypes.Structure):
    _fields_ = [("self", BlockWeights)] + [(n, c_void_p) for n in WAN_EXTRA]


class CacheCfg(ctypes.Structure):
    _fields_ = [("L", c_int32), ("D", c_int32), ("dtype", c_int32)]


class RefCacheCfg(ctypes.Structure):
    _fields_ = [("L", c_int32), ("D", c_int32), ("dtype", c_int32), ("chain_len", c_int32),
                ("capacity", c_int32), ("tau", c_float)]


class RefCacheState(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("pool", "refcount", "free_list", "free_top", "chain_ref",
                                        "ent_slot", "ent_kind", "codes", "scale")]


class ScheduleCfg(ctypes.Structure):
    _fields_ = [("n_full", c_int32), ("r_min", c_double), ("r_max", c_double), ("alpha", c_double),
                ("refresh_delta", c_double)]


class ScheduleState(ctypes.Structure):
    _fields_ = [("step", c_int32), ("delta_max", c_double), ("delta_acc", c_double)]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("launches", c_int64), ("total_ms", c_double)]


_P = ctypes.POINTER
_SIGNATURES = {
    "echo_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "echo_last_hip_error": (ctypes.c_int, []),
    "echo_version": (ctypes.c_char_p, []),
    "echo_energy_workspace": (c_size_t, [_P(EnergyCfg), c_int64]),
    "echo_energy": (ctypes.c_int, [_P(EnergyCfg), c_void_p, c_int64, c_void_p, c_void_p,
                                   c_void_p, c_void_p, c_size_t, c_void_p]),
    "echo_select_workspace": (c_size_t, [_P(SelectCfg)]),
    "echo_select": (ctypes.c_int, [_P(SelectCfg), c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                   c_void_p]),
    "echo_select_noalloc": (ctypes.c_int, [_P(SelectCfg), c_void_p, c_void_p, c_void_p, c_void_p,
                                           c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "echo_saliency_workspace": (c_size_t, [_P(SelectCfg)]),
    "echo_saliency": (ctypes.c_int, [_P(SelectCfg), c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_size_t, c_void_p]),
    "echo_topk": (ctypes.c_int, [_P(SelectCfg), c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "echo_anchors": (ctypes.c_int, [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p]),
    "echo_topk_segments": (ctypes.c_int, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_void_p,
                                          c_void_p, c_void_p, c_void_p]),
    "echo_topk_count": (c_int32, [c_double, c_int32]),
    "echo_segments_count": (c_int32, [c_int32, c_int32, c_int32]),
    "echo_schedule_next": (c_int32, [_P(ScheduleCfg), _P(ScheduleState), c_double, c_int32,
                                     _P(c_int32)]),
    "echo_block_workspace": (c_size_t, [_P(BlockCfg), c_int32]),
    "echo_block_partial": (ctypes.c_int, [_P(BlockCfg), _P(BlockWeights), c_void_p, c_void_p,
                                          c_int32, c_void_p, c_void_p, c_size_t, c_void_p]),
    "echo_wan_block_workspace": (c_size_t, [_P(WanBlockCfg), c_int32]),
    "echo_wan_block_partial": (ctypes.c_int, [_P(WanBlockCfg), _P(WanBlockWeights), c_void_p, c_void_p,
                                              c_void_p, _P(c_int32), c_void_p, c_void_p, c_size_t,
                                              c_void_p]),
    "echo_cache_update": (ctypes.c_int, [_P(CacheCfg), c_void_p, c_void_p, c_void_p, c_int32,
                                         c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                         c_void_p]),
    "echo_cache_update_codec": (ctypes.c_int, [_P(CacheCfg), c_int32, c_void_p, c_void_p, c_void_p,
                                               c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                               c_void_p, c_void_p, c_void_p]),
    "echo_refcache_init": (ctypes.c_int, [_P(RefCacheCfg), _P(RefCacheState), c_void_p]),
    "echo_refcache_update": (ctypes.c_int, [_P(RefCacheCfg), _P(RefCacheState), c_void_p,
                                            c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                            c_void_p, c_void_p]),
    "echo_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "echo_profile_read": (ctypes.c_int, [_P(KernelTime), c_int32]),
    "echo_mfma_ceiling": (ctypes.c_int, [c_int32, c_int32, c_double, _P(c_double), c_void_p]),
}

_lib = None


class EchoError(RuntimeError):
    def __init__(self, fn: str, status: int, hip_error: int | None = None):
        msg = f"{fn} failed: status {status}"
        if _lib is not None:
            msg += f" ({_lib.echo_status_str(status).decode()})"
        if hip_error:
            msg += f", hipError {hip_error}"
        super().__init__(msg)
        self.status = status
        self.hip_error = hip_error


def load() -> ctypes.CDLL:
    """Load libecho.so (built by paper_2608_02474_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2608_02474_amd.build` "
            "(the HIP library is the only implementation of this path)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def check(fn: str, status: int) -> None:
    if status != ECHO_OK:
        hip = _lib.echo_last_hip_error() if status == ECHO_EDEVICE else None
        raise EchoError(fn, status, hip)


def header_functions() -> list:
    """Names of every function the public header declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(echo_[a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))
