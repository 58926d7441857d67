"""Python binding of libecho: the four calls of one cached DiT block step on
torch device tensors.

Argument marshalling only: torch provides device memory (outputs and
workspaces are torch tensors) and the stream (the current torch stream); every
step of the path runs in the library's HIP kernels.

  energy(audio, T)                       audio energy anchor, once per clip
  select(x, xref, frame_weight, N, k)    saliency + top-K / threshold selection
  block_partial(w, x, idx, n_sel, H)     DiT block on the selected tokens
  cache_update(x, idx, mask, n_sel, ...) int8 residual cache write + reuse
  CachedBlock                            the four calls composed, with its cache
"""
from __future__ import annotations

import ctypes
import dataclasses

import torch

from . import _lib
from ._lib import (BlockCfg, BlockWeights, CacheCfg, EnergyCfg, KernelTime, RefCacheCfg, WanBlockCfg,
                   WanBlockWeights,
                   RefCacheState, ScheduleCfg, ScheduleState, SelectCfg,
                   ECHO_BF16, ECHO_F32, check)

_DTYPES = {torch.float32: ECHO_F32, torch.bfloat16: ECHO_BF16}


def _lib_handle():
    return _lib.load()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, name: str, dtype=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t


def _echo_dtype(t: torch.Tensor) -> int:
    if t.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return _DTYPES[t.dtype]


class Workspace:
    """A growable device byte buffer reused across calls."""

    def __init__(self):
        self.buf = None

    def get(self, nbytes: int, device) -> torch.Tensor:
        nbytes = max(int(nbytes), 256)
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != device:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        return self.buf


_WS = {"energy": Workspace(), "select": Workspace(), "block": Workspace()}


# --------------------------------------------------------------------- energy

def energy_cfg(T, sample_rate=16000, n_fft=512, hop=160, n_bands=8) -> EnergyCfg:
    return EnergyCfg(T, sample_rate, n_fft, hop, n_bands)


def energy(audio: torch.Tensor, T: int, sample_rate: int = 16000, n_fft: int = 512,
           hop: int = 160, n_bands: int = 8, workspace: Workspace | None = None):
    """(band_energy [T, n_bands], frame_energy [T], frame_weight [T]), fp32."""
    lib = _lib_handle()
    _dev(audio, "audio", torch.float32)
    cfg = energy_cfg(T, sample_rate, n_fft, hop, n_bands)
    n = audio.numel()
    dev = audio.device
    band = torch.empty((T, n_bands), dtype=torch.float32, device=dev)
    fe = torch.empty(T, dtype=torch.float32, device=dev)
    fw = torch.empty(T, dtype=torch.float32, device=dev)
    need = lib.echo_energy_workspace(ctypes.byref(cfg), n)
    if need == 0:
        check("echo_energy", _lib.ECHO_EINVAL)
    ws = (workspace or _WS["energy"]).get(need, dev)
    check("echo_energy", lib.echo_energy(ctypes.byref(cfg), _ptr(audio), n, _ptr(band), _ptr(fe),
                                         _ptr(fw), _ptr(ws), ws.numel(), _stream()))
    return band, fe, fw


# --------------------------------------------------------------------- select

@dataclasses.dataclass
class Selection:
    idx: torch.Tensor          # int32 [L]; the first n_sel entries are valid, ascending
    mask: torch.Tensor         # uint8 [L]
    n_sel_dev: torch.Tensor    # int32 [1] on the device
    n_sel: int | None          # known on the host in top-k mode
    saliency: torch.Tensor | None
    step_delta: torch.Tensor | None

    def count(self) -> int:
        return self.n_sel if self.n_sel is not None else int(self.n_sel_dev.item())

    def indices(self) -> torch.Tensor:
        return self.idx[: self.count()]


def select(x: torch.Tensor, xref: torch.Tensor, frame_weight: torch.Tensor, N: int,
           k: int | None = None, threshold: float | None = None, xi: float = 1e-6,
           want_saliency: bool = True, want_step_delta: bool = True,
           out: Selection | None = None, workspace: Workspace | None = None) -> Selection:
    """Saliency and selection; pass k for top-k mode or threshold for threshold mode."""
    lib = _lib_handle()
    _dev(x, "x")
    _dev(xref, "xref", x.dtype)
    _dev(frame_weight, "frame_weight", torch.float32)
    L, D = x.shape
    if L % N:
        raise ValueError("L must be a multiple of N")
    T = L // N
    if (k is None) == (threshold is None):
        raise ValueError("pass exactly one of k and threshold")
    cfg = SelectCfg(T, N, D, _echo_dtype(x), -1 if k is None else int(k),
                    0.0 if threshold is None else float(threshold), float(xi))
    dev = x.device
    if out is None:
        out = Selection(
            idx=torch.empty(L, dtype=torch.int32, device=dev),
            mask=torch.empty(L, dtype=torch.uint8, device=dev),
            n_sel_dev=torch.empty(1, dtype=torch.int32, device=dev),
            n_sel=None,
            saliency=torch.empty(L, dtype=torch.float32, device=dev) if want_saliency else None,
            step_delta=torch.empty(1, dtype=torch.float64, device=dev) if want_step_delta else None)
    out.n_sel = None if k is None else int(k)
    need = lib.echo_select_workspace(ctypes.byref(cfg))
    if need == 0:
        check("echo_select", _lib.ECHO_EINVAL)
    ws = (workspace or _WS["select"]).get(need, dev)
    check("echo_select", lib.echo_select(ctypes.byref(cfg), _ptr(x), _ptr(xref), _ptr(frame_weight),
                                         _ptr(out.idx), _ptr(out.mask), _ptr(out.n_sel_dev),
                                         _ptr(out.saliency), _ptr(out.step_delta), _ptr(ws),
                                         ws.numel(), _stream()))
    return out


def select_noalloc(x: torch.Tensor, xref: torch.Tensor, frame_weight: torch.Tensor, N: int,
                   out: Selection, k: int | None = None, threshold: float | None = None,
                   xi: float = 1e-6) -> Selection:
    """select into caller-provided outputs (`out`, e.g. from a previous
    select) through echo_select_noalloc: the library's static scratch instead
    of a workspace, so the call allocates no device memory (at most
    ECHO_SELECT_NOALLOC_MAX_TOKENS tokens)."""
    lib = _lib_handle()
    _dev(x, "x")
    _dev(xref, "xref", x.dtype)
    _dev(frame_weight, "frame_weight", torch.float32)
    L, D = x.shape
    if L % N:
        raise ValueError("L must be a multiple of N")
    if (k is None) == (threshold is None):
        raise ValueError("pass exactly one of k and threshold")
    for t, n, dt in ((out.idx, "idx", torch.int32), (out.mask, "mask", torch.uint8),
                     (out.n_sel_dev, "n_sel", torch.int32)):
        _dev(t, n, dt)
        if t.numel() < (1 if n == "n_sel" else L):
            raise ValueError(f"out.{n} is too small")
    if out.saliency is not None and (_dev(out.saliency, "saliency", torch.float32).numel() < L):
        raise ValueError("out.saliency is too small")
    if out.step_delta is not None:
        _dev(out.step_delta, "step_delta", torch.float64)
    cfg = SelectCfg(L // N, N, D, _echo_dtype(x), -1 if k is None else int(k),
                    0.0 if threshold is None else float(threshold), float(xi))
    check("echo_select_noalloc",
          lib.echo_select_noalloc(ctypes.byref(cfg), _ptr(x), _ptr(xref), _ptr(frame_weight), _ptr(out.idx),
                                  _ptr(out.mask), _ptr(out.n_sel_dev), _ptr(out.saliency),
                                  _ptr(out.step_delta), _stream()))
    out.n_sel = None if k is None else int(k)
    return out


def saliency(x: torch.Tensor, xref: torch.Tensor, frame_weight: torch.Tensor, N: int,
             xi: float = 1e-6, out: Selection | None = None,
             workspace: Workspace | None = None) -> Selection:
    """First half of select: saliency and the step's Eq. 1 value (out.saliency,
    out.step_delta); idx/mask are left for topk."""
    lib = _lib_handle()
    _dev(x, "x")
    _dev(xref, "xref", x.dtype)
    _dev(frame_weight, "frame_weight", torch.float32)
    L, D = x.shape
    if L % N:
        raise ValueError("L must be a multiple of N")
    cfg = SelectCfg(L // N, N, D, _echo_dtype(x), 0, 0.0, float(xi))
    dev = x.device
    if out is None:
        out = Selection(idx=torch.empty(L, dtype=torch.int32, device=dev),
                        mask=torch.empty(L, dtype=torch.uint8, device=dev),
                        n_sel_dev=torch.empty(1, dtype=torch.int32, device=dev), n_sel=None,
                        saliency=torch.empty(L, dtype=torch.float32, device=dev),
                        step_delta=torch.empty(1, dtype=torch.float64, device=dev))
    need = lib.echo_saliency_workspace(ctypes.byref(cfg))
    if need == 0:
        check("echo_saliency", _lib.ECHO_EINVAL)
    ws = (workspace or _WS["select"]).get(need, dev)
    check("echo_saliency", lib.echo_saliency(ctypes.byref(cfg), _ptr(x), _ptr(xref), _ptr(frame_weight),
                                             _ptr(out.saliency), _ptr(out.step_delta), _ptr(ws),
                                             ws.numel(), _stream()))
    return out


def topk(sel: Selection, N: int, D: int, dtype, k: int | None = None,
         threshold: float | None = None) -> Selection:
    """Second half of select: top-k (or threshold) selection from sel.saliency
    into sel.idx / sel.mask / sel.n_sel_dev."""
    lib = _lib_handle()
    L = sel.saliency.numel()
    if (k is None) == (threshold is None):
        raise ValueError("pass exactly one of k and threshold")
    if dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {dtype}")
    cfg = SelectCfg(L // N, N, D, _DTYPES[dtype], -1 if k is None else int(k),
                    0.0 if threshold is None else float(threshold), 1e-6)
    check("echo_topk", lib.echo_topk(ctypes.byref(cfg), _ptr(sel.saliency), _ptr(sel.idx),
                                     _ptr(sel.mask), _ptr(sel.n_sel_dev), _stream()))
    sel.n_sel = None if k is None else int(k)
    return sel


ANCHOR_MODES = ("energy", "uniform", "random")


def anchors(T: int, k: int, mode: str = "energy", keys: torch.Tensor | None = None,
            out: torch.Tensor | None = None, device=None) -> torch.Tensor:
    """Anchor segments, uint8 [T] on the device (echo_anchors): "energy" and
    "random" take the k segments with the largest keys (the frame energies,
    or per-clip uniform random numbers the caller draws); "uniform" the
    evenly spaced ones (keys unused)."""
    lib = _lib_handle()
    if mode not in ANCHOR_MODES:
        raise ValueError(f"mode must be one of {ANCHOR_MODES}")
    if mode == "uniform":
        dev = keys.device if keys is not None else device
        kp = None
    else:
        if keys is None:
            raise ValueError(f"{mode} anchors need keys")
        _dev(keys, "keys", torch.float32)
        dev, kp = keys.device, _ptr(keys)
    if out is None:
        out = torch.empty(T, dtype=torch.uint8, device=dev)
    m = _lib.ECHO_ANCHOR_UNIFORM if mode == "uniform" else _lib.ECHO_ANCHOR_TOPK
    check("echo_anchors", lib.echo_anchors(kp, int(T), int(k), m, _ptr(out), _stream()))
    return out


def topk_segments(sel: Selection, anchor_mask: torch.Tensor, N: int, k: int) -> Selection:
    """Two-stage selection from sel.saliency: min(k, N) tokens in every anchor
    segment into sel.idx / sel.mask / sel.n_sel_dev (echo_topk_segments)."""
    lib = _lib_handle()
    L = sel.saliency.numel()
    T = anchor_mask.numel()
    if T * N != L:
        raise ValueError("anchor mask and saliency disagree on T * N")
    _dev(anchor_mask, "anchors", torch.uint8)
    check("echo_topk_segments",
          lib.echo_topk_segments(_ptr(sel.saliency), _ptr(anchor_mask), T, int(N), int(k), _ptr(sel.idx),
                                 _ptr(sel.mask), _ptr(sel.n_sel_dev), _stream()))
    sel.n_sel = None
    return sel


class Scheduler:
    """Step-level cache schedule (echo_schedule_next, a host function)."""

    @classmethod
    def step_only(cls, n_full: int, refresh_delta: float) -> "Scheduler":
        """Whole-step caching: cached steps recompute nothing; the Eq. 2
        refresh recomputes whole steps."""
        return cls(n_full, 0.0, 0.0, 0.0, refresh_delta)

    @classmethod
    def latent_only(cls, n_full: int, ratio: float) -> "Scheduler":
        """A fixed token ratio on every cached step."""
        return cls(n_full, ratio, ratio, 0.0)

    def __init__(self, n_full: int, r_min: float, r_max: float, alpha: float,
                 refresh_delta: float = 0.0):
        self.cfg = ScheduleCfg(int(n_full), float(r_min), float(r_max), float(alpha),
                               float(refresh_delta))
        self.state = ScheduleState(0, 0.0, 0.0)

    def next(self, delta_t: float, L: int):
        """(k, full) for the current step."""
        full = ctypes.c_int32(0)
        k = _lib_handle().echo_schedule_next(ctypes.byref(self.cfg), ctypes.byref(self.state),
                                             float(delta_t), int(L), ctypes.byref(full))
        if k < 0:
            check("echo_schedule_next", -k)
        return int(k), bool(full.value)


class BlockStack:
    """A stack of cached blocks over a denoising trajectory: per step one Eq. 1
    value and one selection on the first block's input (shared by all blocks),
    the scheduled K, then block_partial + the cache update block after block.

    anchor_mask (uint8 [T] on the device, from `anchors`) switches to the
    two-stage selection: k_t = ceil(N r_t) tokens per anchor segment, ranked
    by the saliency with unit frame weights; n_anchors is the number of
    anchor segments it marks (the k given to `anchors`).  codec:
    "residual_int8" (the default), "full" (the outputs in the activation
    dtype) or "naive_int8"."""

    CODECS = {"residual_int8": 0, "full": 1, "naive_int8": 2}

    def __init__(self, params: list, H: int, L: int, D: int, device, dtype, scheduler: Scheduler,
                 xi: float = 1e-6, ln_eps: float = 1e-6, anchor_mask: torch.Tensor | None = None,
                 n_anchors: int | None = None, codec: str = "residual_int8"):
        if scheduler.cfg.n_full < 1:
            raise ValueError("the first step must be a full step (n_full >= 1)")
        if (anchor_mask is None) != (n_anchors is None):
            raise ValueError("pass anchor_mask and n_anchors together")
        if codec not in self.CODECS:
            raise ValueError(f"codec must be one of {tuple(self.CODECS)}")
        self.params, self.H, self.L, self.D = params, H, L, D
        self.sched, self.xi, self.ln_eps = scheduler, xi, ln_eps
        self.anchor_mask, self.n_anchors, self.codec = anchor_mask, n_anchors, self.CODECS[codec]
        kw = dict(device=device)
        full = self.codec == self.CODECS["full"]
        self.xref = [torch.zeros((L, D), dtype=dtype, **kw) for _ in params]
        self.codes = [None if full else torch.zeros((L, D), dtype=torch.int8, **kw) for _ in params]
        self.scale = [None if full else torch.zeros(L, dtype=torch.float32, **kw) for _ in params]
        self.store = [torch.zeros((L, D), dtype=dtype, **kw) if full else None for _ in params]
        self.y = [torch.empty((L, D), dtype=dtype, **kw) for _ in params]
        self.y_sel = torch.empty((L, D), dtype=torch.float32, **kw)
        self.all_idx = torch.arange(L, dtype=torch.int32, **kw)
        self.all_mask = torch.ones(L, dtype=torch.uint8, **kw)
        self._w = [block_weights(p) for p in params]
        self.ws, self.sel_ws, self.sel = Workspace(), Workspace(), None
        self._unit = None
        self.history = []   # (k, full, delta_t) per step; k per segment in the two-stage form

    def step(self, x0: torch.Tensor, frame_weight: torch.Tensor, N: int) -> torch.Tensor:
        two_stage = self.anchor_mask is not None
        if two_stage:
            if self._unit is None or self._unit.numel() != self.L // N:
                self._unit = torch.ones(self.L // N, dtype=torch.float32, device=x0.device)
            frame_weight = self._unit
        self.sel = saliency(x0, self.xref[0], frame_weight, N, self.xi, out=self.sel,
                            workspace=self.sel_ws)
        delta_t = float(self.sel.step_delta[0].item())      # host needs it to choose K
        k, full = self.sched.next(delta_t, N if two_stage else self.L)
        if full:
            idx, mask, n = self.all_idx, self.all_mask, self.L
        elif two_stage:
            # the count is fixed by k and the anchors: no device read-back
            topk_segments(self.sel, self.anchor_mask, N, k)
            idx, mask, n = self.sel.idx, self.sel.mask, segments_count(self.n_anchors, N, k)
        else:
            topk(self.sel, N, self.D, x0.dtype, k=k)
            idx, mask, n = self.sel.idx, self.sel.mask, k
        x = x0
        for b, p in enumerate(self.params):
            ys = block_partial(p, x, idx, n, self.H, self.ln_eps, y_sel=self.y_sel,
                               workspace=self.ws, _weights=self._w[b])
            x = cache_update_codec(self.codec, x, idx, mask, n, ys, self.xref[b], self.y[b],
                                   store=self.store[b], codes=self.codes[b], scale=self.scale[b])
        self.history.append((k, full, delta_t))
        return x

    def cache_bytes(self) -> int:
        """Device bytes of the per-block cache state (saliency reference,
        codes and scales or the 16-bit store)."""
        t = [*self.xref, *self.codes, *self.scale, *self.store]
        return sum(a.numel() * a.element_size() for a in t if a is not None)


def topk_count(ratio: float, L: int) -> int:
    """K for a recompute ratio (echo_topk_count: ceil(r L), clamped to [0, L])."""
    k = _lib_handle().echo_topk_count(float(ratio), int(L))
    if k < 0:
        check("echo_topk_count", -k)
    return int(k)


def segments_count(n_anchors: int, N: int, k: int) -> int:
    """Tokens the two-stage selection recomputes (echo_segments_count)."""
    n = _lib_handle().echo_segments_count(int(n_anchors), int(N), int(k))
    if n < 0:
        check("echo_segments_count", -n)
    return int(n)


# ------------------------------------------------------------- block partial

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "w1", "w2", "bq", "bk", "bv", "bo", "b1", "b2", "mod")


def block_weights(params: dict) -> BlockWeights:
    for n in WEIGHT_NAMES:
        _dev(params[n], n)
    return BlockWeights(*[params[n].data_ptr() for n in WEIGHT_NAMES])


def block_partial(params: dict, x: torch.Tensor, idx: torch.Tensor, n_sel: int, H: int,
                  ln_eps: float = 1e-6, y_sel: torch.Tensor | None = None,
                  workspace: Workspace | None = None, _weights: BlockWeights | None = None,
                  batch_invariant: bool = False):
    """y_sel [n_sel, D] fp32 = block output of tokens idx[:n_sel].  With
    batch_invariant, each row is bit-identical for any selection containing it."""
    lib = _lib_handle()
    _dev(x, "x")
    _dev(idx, "idx", torch.int32)
    L, D = x.shape
    F = params["w1"].shape[0]
    for n in WEIGHT_NAMES[:-1]:
        if params[n].dtype != x.dtype:
            raise TypeError(f"{n} must have the activation dtype {x.dtype}")
    _dev(params["mod"], "mod", torch.float32)
    cfg = BlockCfg(L, D, H, F, _echo_dtype(x), float(ln_eps),
                   _lib.ECHO_BLOCK_BATCH_INVARIANT if batch_invariant else 0)
    w = _weights if _weights is not None else block_weights(params)
    if y_sel is None:
        y_sel = torch.empty((max(n_sel, 1), D), dtype=torch.float32, device=x.device)
    if n_sel == 0:
        return y_sel[:0]
    need = lib.echo_block_workspace(ctypes.byref(cfg), n_sel)
    if need == 0:
        check("echo_block_partial", _lib.ECHO_EINVAL)
    ws = (workspace or _WS["block"]).get(need, x.device)
    check("echo_block_partial",
          lib.echo_block_partial(ctypes.byref(cfg), ctypes.byref(w), _ptr(x), _ptr(idx), n_sel,
                                 _ptr(y_sel), _ptr(ws), ws.numel(), _stream()))
    return y_sel[:n_sel]


# ----------------------------------------------------------- Wan-style block

def wan_block_partial(params: dict, x: torch.Tensor, ctx: torch.Tensor, idx: torch.Tensor, n_sel,
                      H: int, grid, ln_eps: float = 1e-6, rms_eps: float = 1e-6, rope_base: float = 10000.0,
                      y_sel: torch.Tensor | None = None, workspace: Workspace | None = None,
                      batch_invariant: bool = False) -> torch.Tensor:
    """echo_wan_block_partial: x [B, L, D], ctx [B, Lc, D] (bf16); idx int32 global
    rows b * L + i, element by element; n_sel the B per-element counts (host
    ints); grid (T, gh, gw).  Returns y_sel [sum(n_sel), D] fp32 in idx order.
    params: the block weights plus wqc, wkc, wvc, woc, bqc, bkc, bvc, boc (in
    x's dtype) and gq, gk, gqc, gkc, g3, b3 (fp32 [D])."""
    lib = _lib_handle()
    _dev(x, "x")
    _dev(ctx, "ctx", x.dtype)
    B, L, D = x.shape
    Lc = ctx.shape[1]
    if ctx.shape[0] != B or ctx.shape[2] != D:
        raise ValueError("ctx must be [B, Lc, D]")
    counts = [int(v) for v in n_sel]
    if len(counts) != B:
        raise ValueError("n_sel needs one count per batch element")
    tot = sum(counts)
    F = params["w1"].shape[0]
    for n in WEIGHT_NAMES[:-1] + ("wqc", "wkc", "wvc", "woc", "bqc", "bkc", "bvc", "boc"):
        if params[n].dtype != x.dtype:
            raise TypeError(f"{n} must have the activation dtype {x.dtype}")
    for n in ("mod", "gq", "gk", "gqc", "gkc", "g3", "b3"):
        _dev(params[n], n, torch.float32)
    T_, gh, gw = (int(v) for v in grid)
    cfg = WanBlockCfg(B, L, D, H, F, Lc, T_, gh, gw, _echo_dtype(x), float(ln_eps), float(rms_eps),
                      float(rope_base), _lib.ECHO_BLOCK_BATCH_INVARIANT if batch_invariant else 0)
    w = WanBlockWeights(block_weights(params), *[params[n].data_ptr() for n in _lib.WAN_EXTRA])
    if y_sel is None:
        y_sel = torch.empty((max(tot, 1), D), dtype=torch.float32, device=x.device)
    if tot == 0:
        return y_sel[:0]
    _dev(idx, "idx", torch.int32)
    need = lib.echo_wan_block_workspace(ctypes.byref(cfg), tot)
    if need == 0:
        check("echo_wan_block_partial", _lib.ECHO_EINVAL)
    ws = (workspace or _WS["block"]).get(need, x.device)
    arr = (ctypes.c_int32 * B)(*counts)
    check("echo_wan_block_partial",
          lib.echo_wan_block_partial(ctypes.byref(cfg), ctypes.byref(w), _ptr(x), _ptr(ctx), _ptr(idx), arr,
                                     _ptr(y_sel), _ptr(ws), ws.numel(), _stream()))
    return y_sel[:tot]


# --------------------------------------------------------------- cache update

def cache_update(x: torch.Tensor, idx: torch.Tensor, mask: torch.Tensor, n_sel: int,
                 y_sel: torch.Tensor, xref: torch.Tensor, codes: torch.Tensor,
                 scale: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
    """Writes the fresh rows into (xref, codes, scale) in place; returns y."""
    lib = _lib_handle()
    _dev(x, "x")
    L, D = x.shape
    _dev(mask, "mask", torch.uint8)
    _dev(xref, "xref", x.dtype)
    _dev(codes, "codes", torch.int8)
    _dev(scale, "scale", torch.float32)
    if n_sel > 0:
        _dev(idx, "idx", torch.int32)
        _dev(y_sel, "y_sel", torch.float32)
    if y is None:
        y = torch.empty_like(x)
    cfg = CacheCfg(L, D, _echo_dtype(x))
    check("echo_cache_update",
          lib.echo_cache_update(ctypes.byref(cfg), _ptr(x), _ptr(idx) if n_sel else None,
                                _ptr(mask), n_sel, _ptr(y_sel) if n_sel else None, _ptr(xref),
                                _ptr(codes), _ptr(scale), _ptr(y), _stream()))
    return y


def cache_update_codec(codec: int, x: torch.Tensor, idx: torch.Tensor, mask: torch.Tensor, n_sel: int,
                       y_sel: torch.Tensor, xref: torch.Tensor, y: torch.Tensor | None = None,
                       store: torch.Tensor | None = None, codes: torch.Tensor | None = None,
                       scale: torch.Tensor | None = None) -> torch.Tensor:
    """echo_cache_update_codec: codec 0 residual int8 (codes, scale), 1 the
    output in the activation dtype (store), 2 int8 of the output itself
    (codes, scale).  Updates the cache state in place; returns y."""
    lib = _lib_handle()
    _dev(x, "x")
    L, D = x.shape
    _dev(mask, "mask", torch.uint8)
    _dev(xref, "xref", x.dtype)
    if codec == _lib.ECHO_CODEC_FULL:
        _dev(store, "store", x.dtype)
    else:
        _dev(codes, "codes", torch.int8)
        _dev(scale, "scale", torch.float32)
    if n_sel > 0:
        _dev(idx, "idx", torch.int32)
        _dev(y_sel, "y_sel", torch.float32)
    if y is None:
        y = torch.empty_like(x)
    cfg = CacheCfg(L, D, _echo_dtype(x))
    check("echo_cache_update_codec",
          lib.echo_cache_update_codec(ctypes.byref(cfg), int(codec), _ptr(x), _ptr(idx) if n_sel else None,
                                      _ptr(mask), n_sel, _ptr(y_sel) if n_sel else None, _ptr(xref),
                                      _ptr(store), _ptr(codes), _ptr(scale), _ptr(y), _stream()))
    return y


# ---------------------------------------------------- adaptive reference cache

class RefCache:
    """Device state of the adaptive reference cache (Sec. 3.4): reference pool
    with hold counts and free slots, per-token entries (kind, slot, int8
    residual codes, scale) and each chain's current reference."""

    def __init__(self, L: int, D: int, chain_len: int, tau: float, dtype, device,
                 capacity: int | None = None):
        if L % chain_len:
            raise ValueError("L must be a multiple of chain_len")
        self.L, self.D, self.chain_len, self.tau, self.dtype = L, D, chain_len, float(tau), dtype
        self.n_chains = L // chain_len
        self.capacity = capacity if capacity is not None else L + self.n_chains
        kw = dict(device=device)
        self.pool = torch.empty((self.capacity, D), dtype=dtype, **kw)
        self.refcount = torch.empty(self.capacity, dtype=torch.int32, **kw)
        self.free_list = torch.empty(self.capacity, dtype=torch.int32, **kw)
        self.free_top = torch.empty(4, dtype=torch.int32, **kw)  # [0] used; 16-byte alignment
        self.chain_ref = torch.empty(self.n_chains, dtype=torch.int32, **kw)
        self.ent_slot = torch.empty(L, dtype=torch.int32, **kw)
        self.ent_kind = torch.empty(L, dtype=torch.uint8, **kw)
        self.codes = torch.empty((L, D), dtype=torch.int8, **kw)
        self.scale = torch.empty(L, dtype=torch.float32, **kw)
        self.cfg = RefCacheCfg(L, D, _echo_dtype(self.pool), chain_len, self.capacity, self.tau)
        self.state = RefCacheState(*[_ptr(t) for t in (self.pool, self.refcount, self.free_list,
                                                        self.free_top, self.chain_ref, self.ent_slot,
                                                        self.ent_kind, self.codes, self.scale)])
        check("echo_refcache_init",
              _lib_handle().echo_refcache_init(ctypes.byref(self.cfg), ctypes.byref(self.state),
                                               _stream()))

    def update(self, x: torch.Tensor, idx: torch.Tensor, mask: torch.Tensor, n_sel: int,
               y_sel: torch.Tensor, xref: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
        """Writes the fresh rows, records their inputs in xref; returns the fused y."""
        _dev(x, "x", self.dtype)
        _dev(mask, "mask", torch.uint8)
        _dev(xref, "xref", self.dtype)
        if n_sel > 0:
            _dev(idx, "idx", torch.int32)
            _dev(y_sel, "y_sel", torch.float32)
        if y is None:
            y = torch.empty_like(x)
        check("echo_refcache_update",
              _lib_handle().echo_refcache_update(
                  ctypes.byref(self.cfg), ctypes.byref(self.state), _ptr(x),
                  _ptr(idx) if n_sel else None, _ptr(mask), n_sel,
                  _ptr(y_sel) if n_sel else None, _ptr(xref), _ptr(y), _stream()))
        return y

    def live_refs(self) -> int:
        """References currently held (synchronizes with the device)."""
        return self.capacity - int(self.free_top[0].item())

    def live_bytes(self) -> int:
        """Bytes of live cache state: held reference rows plus codes and scales."""
        return self.live_refs() * self.D * self.pool.element_size() + self.codes.numel() + 4 * self.L


# ------------------------------------------------------------- kernel timing

def profile_enable(on: bool = True) -> None:
    check("echo_profile_enable", _lib_handle().echo_profile_enable(1 if on else 0))


def profile_read(max_entries: int = 64) -> dict:
    """{kernel name: (launches, total ms)} for launches since the last read."""
    lib = _lib_handle()
    arr = (KernelTime * max_entries)()
    n = lib.echo_profile_read(arr, max_entries)
    if n < 0:
        check("echo_profile_read", -n)
    return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms)) for i in range(n)}


# ------------------------------------------------------ sustained MFMA rate

def mfma_ceiling(pattern: str = "attention", data: str = "gaussian", seconds: float = 3.0) -> float:
    """Sustained rate (TFLOP/s) of a dense bf16 MFMA stream with the attention's
    ("attention") or the GEMM's ("gemm") instruction pattern on "gaussian" or
    "constant" operands, on the current device and stream (echo_mfma_ceiling)."""
    pat = {"attention": 0, "gemm": 1}[pattern]
    dat = {"constant": 0, "gaussian": 1}[data]
    out = ctypes.c_double(0.0)
    check("echo_mfma_ceiling", _lib_handle().echo_mfma_ceiling(pat, dat, float(seconds), ctypes.byref(out), _stream()))
    return out.value


# ---------------------------------------------------------------- composition

class CachedBlock:
    """One DiT block with an EchoCache int8 residual cache on one device.

    init(x)                 recompute every token and fill the cache (first step)
    step(x, w, ratio|k)     saliency -> top-K -> partial block -> cache update
    Returns the block output y [L, D] in the activation dtype.
    """

    def __init__(self, params: dict, H: int, L: int, D: int, device, dtype,
                 ln_eps: float = 1e-6, xi: float = 1e-6):
        self.params = params
        self.H, self.L, self.D = H, L, D
        self.ln_eps, self.xi = ln_eps, xi
        self.xref = torch.zeros((L, D), dtype=dtype, device=device)
        self.codes = torch.zeros((L, D), dtype=torch.int8, device=device)
        self.scale = torch.zeros(L, dtype=torch.float32, device=device)
        self.y = torch.empty((L, D), dtype=dtype, device=device)
        self.y_sel = torch.empty((L, D), dtype=torch.float32, device=device)
        self.all_idx = torch.arange(L, dtype=torch.int32, device=device)
        self.all_mask = torch.ones(L, dtype=torch.uint8, device=device)
        self.ws = Workspace()
        self.sel_ws = Workspace()
        self.sel = None
        self._w = block_weights(params)

    def init(self, x: torch.Tensor) -> torch.Tensor:
        ys = block_partial(self.params, x, self.all_idx, self.L, self.H, self.ln_eps,
                           y_sel=self.y_sel, workspace=self.ws, _weights=self._w)
        return cache_update(x, self.all_idx, self.all_mask, self.L, ys, self.xref, self.codes,
                            self.scale, self.y)

    def step(self, x: torch.Tensor, frame_weight: torch.Tensor, N: int,
             ratio: float | None = None, k: int | None = None) -> torch.Tensor:
        if k is None:
            k = topk_count(ratio, self.L)
        self.sel = select(x, self.xref, frame_weight, N, k=k, xi=self.xi, out=self.sel,
                          workspace=self.sel_ws)
        ys = block_partial(self.params, x, self.sel.idx, k, self.H, self.ln_eps,
                           y_sel=self.y_sel, workspace=self.ws, _weights=self._w)
        return cache_update(x, self.sel.idx, self.sel.mask, k, ys, self.xref, self.codes,
                            self.scale, self.y)
