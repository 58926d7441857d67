#!/usr/bin/env python3
"""Throughput of one cached DiT block step on one MI355X.

A step is the whole hot path on one batch of synthetic input, resident in HBM:
audio energy (echo_energy), saliency + top-K selection (echo_select), the DiT
block on the selected tokens (echo_block_partial) and the int8 cache update
with reuse of every other token (echo_cache_update).  The default workload is
the Wan2.2-S2V-14B-shaped block at 480p: 21 latent frames x 30 x 52 = 32760
tokens, hidden 5120, 40 heads of 128, FFN 13824, recompute ratio 0.4 (13104
tokens), 5.06 s of 16 kHz audio.

Prints one JSON line: whole-step tokens/s (L / step time) from exactly
`--steps` uninstrumented steps, the step-time median / p10 / p90 over at least
50 further steps with the shader clock and board power sampled meanwhile, the
dense block over every token (the speedup's denominator), the roofline of the
dominant kernel and a per-kernel table from a separate run of the same steps
in which the library records HIP events around every launch on its stream, and
the CPU oracle's throughput on bounded samples (fp64, and its fp32 timing mode;
rank 0, N = 1).  Side legs, outside the timed step: the adaptive reference
cache (update time, live references and bytes), a scheduled multi-block stack
over a denoising trajectory, and the module ablation's variants (anchor
strategies, step-only / latent-only schedules, 16-bit and naive int8 caches:
kernel times, stack latency, cache bytes, distance from an all-full run),
the Wan-style block (qk RMSNorm + 3D RoPE, cross-attention, batch of two), the
streaming kernels timed alone after a read sweep that leaves the MALL clean,
the 32760-token step swept over recompute ratios 0.1 / 0.25 / 0.5 / 1.0 under
three audio energy profiles, and the 720p-shaped step (75600 tokens) with its
cache footprint.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "latent tokens/s per cached DiT block step + %MFMA / %HBM peak"
KERNEL_SOURCES = {"attn_fwd": "attn_bf16.hip", "gemm_": "gemm_bf16.hip", "saliency": "select.hip",
                  "select": "select.hip", "cache_update": "cache.hip", "modln": "block_ln.hip",
                  "energy": "energy.hip", "refcache": "refcache.hip",
                  "anchor": "select.hip"}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_sha(kernel: str) -> str | None:
    for prefix, fname in KERNEL_SOURCES.items():
        if kernel.startswith(prefix):
            path = os.path.join(ROOT, "paper_2608_02474_amd", "csrc", fname)
            return hashlib.sha256(open(path, "rb").read()).hexdigest()
    return None


def measured_traffic(kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current source of that kernel; None otherwise."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(kernel)
    if not rec or rec.get("source_sha256") != source_sha(kernel):
        return None
    return rec.get("bytes_per_launch")


def _timed(fn, *a) -> float:
    """Seconds of fn(*a) on its second run: the first run pays one-time costs
    (page faults of fresh allocations) that are not part of the work."""
    fn(*a)
    t0 = time.perf_counter()
    fn(*a)
    return time.perf_counter() - t0


def _fit_time(fn, r1: int, r2: int, full: int) -> float:
    """Time fn(r) at two sample sizes and extrapolate t = fixed + per_row * r
    to r = full, so per-call overheads are not multiplied by the row count."""
    t1 = _timed(fn, r1)
    t2 = _timed(fn, r2)
    per_row = max(t2 - t1, 0.0) / (r2 - r1)
    fixed = max(t1 - per_row * r1, 0.0)
    return fixed + per_row * full


class ClockSampler:
    """Samples the GPU's shader clock (MHz) and socket power (W) from a host
    thread while the GPU works, through amdsmi's GPU metrics (the SMU's
    current clock of every XCD and its current socket power); summary() gives
    means and ranges, or None where a reading is unavailable."""

    def __init__(self, device_index: int = 0, period_s: float = 0.02):
        import threading
        self.dev, self.period = device_index, period_s
        self.clk, self.avg_clk, self.pwr = [], [], []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    @staticmethod
    def _num(v):
        return float(v) if isinstance(v, (int, float)) and not isinstance(v, bool) else None

    def _run(self):
        try:
            import amdsmi
            import torch
            handle = torch.cuda._get_amdsmi_handler(self.dev)
        except Exception:
            return
        while not self._stop.is_set():
            try:
                m = amdsmi.amdsmi_get_gpu_metrics_info(handle)
                xcd = [self._num(c) for c in (m.get("current_gfxclks") or [])
                       if isinstance(m.get("current_gfxclks"), list)]
                xcd = [c for c in xcd if c]
                if xcd:
                    self.clk.append(sum(xcd) / len(xcd))
                elif self._num(m.get("current_gfxclk")):
                    self.clk.append(self._num(m.get("current_gfxclk")))
                if self._num(m.get("average_gfxclk_frequency")):
                    self.avg_clk.append(self._num(m.get("average_gfxclk_frequency")))
                p = self._num(m.get("current_socket_power")) or self._num(m.get("average_socket_power"))
                if p:
                    self.pwr.append(p)
            except Exception:
                pass
            self._stop.wait(self.period)

    def __enter__(self):
        self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._thread.join()

    def summary(self):
        def stats(v):
            if not v:
                return None
            v = sorted(v)
            return {"mean": round(sum(v) / len(v), 1), "min": round(v[0], 1), "max": round(v[-1], 1),
                    "samples": len(v)}
        return {"sclk_mhz": stats(self.clk), "avg_gfxclk_mhz": stats(self.avg_clk), "power_w": stats(self.pwr),
                "source": "amdsmi GPU metrics: mean of the XCDs' current gfx clocks, the SMU's average "
                          "gfx clock, current socket power"}


def _percentiles(v):
    import numpy as np
    a = np.asarray(v, np.float64)
    return {"n": int(a.size), "median": round(float(np.median(a)), 4),
            "p10": round(float(np.percentile(a, 10)), 4), "p90": round(float(np.percentile(a, 90)), 4),
            "mean": round(float(a.mean()), 4), "min": round(float(a.min()), 4), "max": round(float(a.max()), 4)}


def _per_step_times(step, steps: int):
    """Wall times of `steps` consecutive step() calls from HIP events on the
    current stream (one event at every step boundary); (total ms, [ms])."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[-1]), [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def cpu_baseline_fp32(w, p, x, xref, audio, rows: int = 1024):
    """The oracle's steps in its fp32 timing mode (single-precision,
    BLAS-threaded numpy) on the host: the all-row LN + K/V projection of the
    whole step, `rows` selected rows through Q, attention over all L keys, O
    and the FFN (extrapolated per row to K), and the saliency, top-K and
    cache update of the whole step."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import block as OB
    from oracle import cache as OC
    from oracle import energy as OE
    from oracle import select as OS

    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    L, K = w.L, w.K
    p32 = OB._f64(p, np.float32)
    x32 = np.asarray(x, np.float32)
    t = {}
    t0 = time.perf_counter()
    fw = OE.energy(audio, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)[2]
    t["energy"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    s = OS.saliency(x, xref, fw, w.N)[0]
    t["saliency"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    idx = OS.select_topk(s, K)
    t["topk"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    kv = OB.kv_projection(p32, x32, dt=np.float32)
    t["ln_kv"] = time.perf_counter() - t0
    r = min(rows, K)
    t0 = time.perf_counter()
    y_part = OB.block_partial(p32, x32, idx[:r], w.H, kv=kv, dt=np.float32)
    t["selected_rows"] = (time.perf_counter() - t0) * K / r
    del kv
    y_sel = np.resize(y_part, (K, w.D)).astype(np.float32)
    t0 = time.perf_counter()
    OC.cache_update(x, idx, y_sel, xref, np.zeros((L, w.D), np.int8), np.zeros(L, np.float32), w.dtype)
    t["cache_update"] = time.perf_counter() - t0
    total = sum(t.values())
    return {"value": L / total, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"fp32 timing mode of the oracle (single-precision BLAS-threaded numpy): the whole "
                       f"step's energy, saliency, top-K, LN + K/V projection of all {L} rows and cache "
                       f"update; {r} of the {K} selected rows through Q, attention over all {L} keys, O "
                       f"and FFN, extrapolated per row"),
            "step_seconds": total, "parts_seconds": {k_: round(v_, 3) for k_, v_ in t.items()}}


def cpu_baseline(w, p, x, xref, audio):
    """The CPU oracle, as it stands, timed on bounded samples of the workload;
    each part is extrapolated to the full step from two sample sizes."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import block as OB
    from oracle import cache as OC
    from oracle import energy as OE
    from oracle import select as OS

    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    L, D, K = w.L, w.D, w.K
    p64 = OB._f64(p)                      # weights held in fp64 once (setup, not timed)
    t = {}
    fw = OE.energy(audio, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)[2]
    t["energy"] = _timed(OE.energy, audio, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
    r_sal, r_kv, r_cache = min(L, 4096), min(L, 2048), min(L, 4096)
    t["saliency"] = _timed(OS.saliency, x[:r_sal], xref[:r_sal], fw, w.N) * L / r_sal
    s_full = np.resize(OS.saliency(x[:r_sal], xref[:r_sal], fw, w.N)[0], L)
    t["topk"] = _timed(OS.select_topk, s_full, K)
    x64 = np.asarray(x[:r_kv], np.float64)
    t["ln_kv"] = _timed(OB.kv_projection, p64, x64) * L / r_kv
    kv = OB.kv_projection(p64, x64)
    # keys/values of all L rows, tiled from the projected sample (timing only)
    reps = -(-L // r_kv)
    kv_full = tuple(np.concatenate([m] * reps)[:L] for m in kv)
    del kv, x64

    def sel_rows(r):
        OB.block_partial(p64, x[:r], np.arange(r), w.H, kv=kv_full)
    r_sel = (min(K, 64), min(K, 256))
    t["selected_rows"] = _fit_time(sel_rows, r_sel[0], r_sel[1], K)
    del kv_full
    k_c = max(1, r_cache * K // L)
    idx = np.linspace(0, r_cache - 1, k_c).astype(np.int64)
    t["cache_update"] = _timed(OC.cache_update, x[:r_cache], idx, x[idx] + np.float32(0.01),
                               xref[:r_cache], np.zeros((r_cache, D), np.int8),
                               np.zeros(r_cache, np.float32), w.dtype) * L / r_cache
    total = sum(t.values())
    return {"value": L / total, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"fp64 numpy oracle, extrapolated: full audio energy; saliency of {r_sal} rows; a full "
                       f"{L}-key top-{K}; LN + K/V projection of {r_kv} rows; {r_sel[0]} and "
                       f"{r_sel[1]} selected rows (Q, attention over all {L} keys, O, FFN); cache "
                       f"update of {r_cache} rows. Row-proportional parts are scaled by rows; the "
                       f"selected-row part is extrapolated as fixed + per-row cost"),
            "step_seconds": total, "parts_seconds": {k_: round(v_, 3) for k_, v_ in t.items()}}


def refcache_leg(w, dev, dt, steps: int = 5, tau: float = 0.9, corr: float = 0.95,
                 shared: float = 2.0):
    """The adaptive reference cache (Sec. 3.4) at the workload's shape.  Fresh
    outputs are synthetic: per latent-grid row a shared component (N(0, 1) times
    `shared`) plus an AR(1) sequence along the row (coefficient `corr`),
    standing in for the similarity of adjacent latents the cache relies on (the
    seeded latents of the main step are independent across tokens and would
    store every token as a reference).  Times echo_refcache_update on K-token
    steps after an all-token first write; reports live memory."""
    import torch

    from paper_2608_02474_amd import api

    L, D, K, w_len = w.L, w.D, w.K, w.grid[1]
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + w.seed)

    def outputs(rows: int, gen) -> torch.Tensor:
        n = torch.randn((rows // w_len, w_len, D), device=dev, generator=gen)
        y = torch.empty_like(n)
        y[:, 0] = n[:, 0]
        a, b = corr, (1.0 - corr * corr) ** 0.5
        for t in range(1, w_len):
            y[:, t] = a * y[:, t - 1] + b * n[:, t]
        y += shared * torch.randn((rows // w_len, 1, D), device=dev, generator=gen)
        return y.reshape(rows, D)

    rc = api.RefCache(L, D, w_len, tau, dt, dev)
    x = torch.randn((L, D), device=dev, generator=g).to(dt)
    xref = torch.zeros((L, D), dtype=dt, device=dev)
    y_all = outputs(L, g)
    all_idx = torch.arange(L, dtype=torch.int32, device=dev)
    rc.update(x, all_idx, torch.ones(L, dtype=torch.uint8, device=dev), L, y_all, xref)
    sels = []
    for _ in range(steps + 1):
        perm = torch.randperm(L, device=dev, generator=g)[:K]
        idx = torch.sort(perm).values.to(torch.int32)
        mask = torch.zeros(L, dtype=torch.uint8, device=dev)
        mask[idx.long()] = 1
        y_sel = (y_all[idx.long()] + 0.05 * torch.randn((K, D), device=dev, generator=g)).contiguous()
        sels.append((idx, mask, y_sel))
    y = torch.empty((L, D), dtype=dt, device=dev)
    rc.update(x, *sels[0][:2], K, sels[0][2], xref, y)           # warmup
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for idx, mask, y_sel in sels[1:]:
        rc.update(x, idx, mask, K, y_sel, xref, y)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    b = torch.tensor([], dtype=dt).element_size()
    live = rc.live_bytes()
    return {"update_ms": round(ms, 4), "tau": tau, "chain_len": w_len, "adjacent_corr": corr,
            "shared_component": shared,
            "live_refs": rc.live_refs(), "live_cache_bytes": live,
            "full_precision_cache_bytes": L * D * b,
            "per_token_residual_cache_bytes": L * D * (b + 1) + 4 * L,
            "data": "synthetic fresh outputs: shared per-row component + AR(1) along each "
                    "latent-grid row"}


def make_stack_blocks(w, dev, dt, n_blocks: int, seed: int):
    """Random-init weights of n_blocks blocks of the workload's shape,
    generated on the device (same distributions as the main step)."""
    import torch

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    D, F = w.D, w.F

    def rnd(*shape, std=0.02, mean=0.0, dtype=dt):
        return (torch.randn(shape, device=dev, generator=g) * std + mean).to(dtype)

    blocks = []
    for _ in range(n_blocks):
        mod = torch.cat([rnd(2, D, std=0.1, dtype=torch.float32), rnd(1, D, std=0.05, mean=0.25, dtype=torch.float32),
                         rnd(2, D, std=0.1, dtype=torch.float32), rnd(1, D, std=0.05, mean=0.25, dtype=torch.float32)])
        blocks.append({"wq": rnd(D, D), "wk": rnd(D, D), "wv": rnd(D, D), "wo": rnd(D, D),
                       "w1": rnd(F, D), "w2": rnd(D, F), "bq": rnd(D), "bk": rnd(D), "bv": rnd(D),
                       "bo": rnd(D), "b1": rnd(F), "b2": rnd(D), "mod": mod.contiguous()})
    return blocks


def run_trajectory(stack, w, dev, dt, fw, steps: int, seed: int, motion=None, ref=None, keep=False):
    """First-block inputs x_{t+1} = x_t + (0.3 / (t + 1)) m N(0, 1), generated on
    the device from `seed`, m = motion[frame of the token] (1 if None).
    Returns (per-step ms, outputs): every step's output if keep, else the
    relative L2 distance of every step's output from ref[t] if ref is given,
    else the last output."""
    import torch

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    x = torch.randn((w.L, w.D), device=dev, generator=g)
    m = None if motion is None else motion.repeat_interleave(w.N)[:, None]
    times, outs, y = [], [], None
    for t in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        y = stack.step(x.to(dt), fw, w.N)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
        if keep:
            outs.append(y.clone())
        elif ref is not None:
            r = ref[t].float()
            outs.append(float(torch.linalg.vector_norm(y.float() - r) / torch.linalg.vector_norm(r)))
        dx = torch.randn((w.L, w.D), device=dev, generator=g) * (0.3 / (t + 1))
        x = x + (dx if m is None else dx * m)
    return times, (outs if keep or ref is not None else y)


def stack_leg(w, dev, dt, fw, blocks, steps: int, n_full: int = 2, r_min: float = 0.2,
              r_max: float = 0.6, alpha: float = 0.4):
    """A stack of blocks of the workload's shape over a synthetic denoising
    trajectory: one Eq. 1 value and one selection per step on the first
    block's input, K from the step schedule, then every block on the shared
    selection."""
    from paper_2608_02474_amd import api

    stack = api.BlockStack(blocks, w.H, w.L, w.D, dev, dt, api.Scheduler(n_full, r_min, r_max, alpha))
    times, _ = run_trajectory(stack, w, dev, dt, fw, steps, seed=3000 + w.seed)
    ks = [k for k, _, _ in stack.history]
    full = [f for _, f, _ in stack.history]
    full_ms = [tm for tm, f in zip(times, full) if f]
    cached_ms = [tm for tm, f in zip(times, full) if not f]
    ref = sum(full_ms) / len(full_ms)
    return {"blocks": len(blocks), "steps": steps,
            "schedule": {"n_full": n_full, "r_min": r_min, "r_max": r_max, "alpha": alpha},
            "k_per_step": ks, "full_step": full,
            "delta_per_step": [None if f else round(d, 6) for _, f, d in stack.history],
            "ms_per_step": [round(tm, 2) for tm in times],
            "full_step_ms": round(ref, 2),
            "cached_step_ms_mean": round(sum(cached_ms) / max(len(cached_ms), 1), 2),
            "trajectory_ms": round(sum(times), 1),
            "speedup_vs_all_full": round(ref * steps / sum(times), 3),
            "data": "synthetic trajectory and random-init weights (device-generated)"}


def _kernel_avgs(ktimes: dict) -> dict:
    return {n: t / c for n, (c, t) in ktimes.items()}


def variants_leg(w, dev, dt, fe, fw, blocks, steps: int, n_anchor: int = 14, n_full: int = 2,
                 r_min: float = 0.2, r_max: float = 0.6, alpha: float = 0.4, refresh: float = 0.4):
    """The module ablation's variants (anchor strategies, schedules, cache
    codecs) on the workload's shape: their kernels alone, then stacks of the
    same blocks over the same trajectory, each with its latency, cache bytes
    and the relative L2 distance of its last output from an all-full run."""
    import torch

    from paper_2608_02474_amd import api, roofline

    L, D, N, T, K = w.L, w.D, w.N, w.T, w.K
    b = 2 if dt == torch.bfloat16 else 4
    g = torch.Generator(device=dev)
    g.manual_seed(4000 + w.seed)
    out = {}

    # (1) the cache codecs alone: one full write, then updates at K rows
    X = torch.randn((L, D), device=dev, generator=g).to(dt)
    perm = torch.randperm(L, device=dev, generator=g)[:K]
    idx = torch.sort(perm).values.to(torch.int32)
    mask = torch.zeros(L, dtype=torch.uint8, device=dev)
    mask[idx.long()] = 1
    all_idx = torch.arange(L, dtype=torch.int32, device=dev)
    all_mask = torch.ones(L, dtype=torch.uint8, device=dev)
    y_all = torch.randn((L, D), device=dev, generator=g)
    y_sel = y_all[:K].contiguous()
    work = roofline.kernel_work(L, K, D, w.F, b)
    codecs = {}
    for cname, codec in (("residual_int8", 0), ("full", 1), ("naive_int8", 2)):
        st = dict(store=torch.zeros((L, D), dtype=dt, device=dev)) if codec == 1 else dict(
            codes=torch.zeros((L, D), dtype=torch.int8, device=dev), scale=torch.zeros(L, device=dev))
        xref = torch.zeros((L, D), dtype=dt, device=dev)
        y = torch.empty((L, D), dtype=dt, device=dev)
        api.cache_update_codec(codec, X, all_idx, all_mask, L, y_all, xref, y, **st)
        for _ in range(3):
            api.cache_update_codec(codec, X, idx, mask, K, y_sel, xref, y, **st)
        torch.cuda.synchronize()
        api.profile_enable(True)
        api.profile_read()
        for _ in range(20):
            api.cache_update_codec(codec, X, idx, mask, K, y_sel, xref, y, **st)
        avgs = _kernel_avgs(api.profile_read())
        api.profile_enable(False)
        kname, avg = next(iter(avgs.items()))
        amount, _ = roofline.work_of(kname, work)
        gbs = amount / (avg * 1e-3) / 1e9
        state = L * D * b + sum(t.numel() * t.element_size() for t in st.values())
        codecs[cname] = {"kernel": kname, "avg_ms": round(avg, 4), "achieved_gbs": round(gbs, 1),
                         "frac": round(gbs / roofline.PEAK_HBM_GBS, 4), "per_launch": amount,
                         "cache_bytes_per_block": state}
        del st, xref, y
    out["codec_kernels"] = codecs
    del X, y_all, y_sel

    # (2) selection: anchors once per clip; two-stage vs global top-k per step
    keys = torch.rand(T, device=dev, generator=g)
    sal = torch.rand(L, device=dev, generator=g)
    sel = api.Selection(idx=torch.empty(L, dtype=torch.int32, device=dev),
                        mask=torch.empty(L, dtype=torch.uint8, device=dev),
                        n_sel_dev=torch.empty(1, dtype=torch.int32, device=dev), n_sel=None,
                        saliency=sal, step_delta=None)
    kseg = api.topk_count(w.ratio, N)
    am = api.anchors(T, n_anchor, "random", keys=keys)
    for _ in range(3):
        api.topk_segments(sel, am, N, kseg)
        api.topk(sel, N, D, dt, k=api.segments_count(n_anchor, N, kseg))
    torch.cuda.synchronize()
    api.profile_enable(True)
    api.profile_read()
    for _ in range(20):
        api.anchors(T, n_anchor, "random", keys=keys, out=am)
        api.topk_segments(sel, am, N, kseg)
        api.topk(sel, N, D, dt, k=api.segments_count(n_anchor, N, kseg))
    avgs = _kernel_avgs(api.profile_read())
    api.profile_enable(False)
    out["selection_kernels"] = {"anchors": n_anchor, "tokens_per_anchor": kseg,
                                "selected": n_anchor * kseg,
                                "anchor_select_ms": round(avgs.get("anchor_select", 0.0), 4),
                                "select_segments_ms": round(avgs.get("select_segments", 0.0), 4),
                                "select_rows_ms_same_count": round(avgs.get("select_rows", 0.0), 4)}

    # (3) stacks: the same blocks and trajectory under each variant.  The
    # trajectory's per-frame change follows the audio energy (m_t = 0.2 + 0.8
    # w_t, w = frame weight): the premise of the energy anchors.
    unit = torch.ones(T, device=dev)
    motion = 0.2 + 0.8 * fw
    anchor_masks = {"energy": api.anchors(T, n_anchor, "energy", keys=fe),
                    "uniform": api.anchors(T, n_anchor, "uniform", device=dev),
                    "random": api.anchors(T, n_anchor, "random",
                                          keys=torch.rand(T, device=dev, generator=g))}
    sched = lambda: api.Scheduler(n_full, r_min, r_max, alpha)
    configs = [
        ("all_full", dict(scheduler=api.Scheduler(steps, 1.0, 1.0, 0.0))),
        ("echocache", dict(scheduler=sched())),
        ("unit_frame_weight", dict(scheduler=sched(), fw=unit)),
        ("two_stage_energy", dict(scheduler=sched(), anchor_mask=anchor_masks["energy"],
                                     n_anchors=n_anchor)),
        ("two_stage_uniform", dict(scheduler=sched(), anchor_mask=anchor_masks["uniform"],
                                     n_anchors=n_anchor)),
        ("two_stage_random", dict(scheduler=sched(), anchor_mask=anchor_masks["random"],
                                     n_anchors=n_anchor)),
        ("step_only", dict(scheduler=api.Scheduler.step_only(n_full, refresh))),
        ("latent_only", dict(scheduler=api.Scheduler.latent_only(n_full, w.ratio))),
        ("fp16_cache", dict(scheduler=sched(), codec="full")),
        ("naive_int8_cache", dict(scheduler=sched(), codec="naive_int8")),
    ]
    runs, ref = {}, None
    for name, cfg in configs:
        log(f"  variant stack {name}")
        f = cfg.pop("fw", fw)
        stack = api.BlockStack(blocks, w.H, L, D, dev, dt, cfg.pop("scheduler"), **cfg)
        if ref is None:
            times, ref = run_trajectory(stack, w, dev, dt, f, steps, 5000 + w.seed, motion, keep=True)
            errs = [0.0] * steps
        else:
            times, errs = run_trajectory(stack, w, dev, dt, f, steps, 5000 + w.seed, motion, ref=ref)
        two = cfg.get("anchor_mask") is not None
        cached = [e for e, (_, full, _) in zip(errs, stack.history) if not full]
        runs[name] = {"trajectory_ms": round(sum(times), 1),
                      "tokens_recomputed": int(sum(L if full else (api.segments_count(n_anchor, N, k) if two else k)
                                                   for k, full, _ in stack.history)),
                      "full_steps": int(sum(full for _, full, _ in stack.history)),
                      "cache_bytes_per_block": stack.cache_bytes() // len(blocks),
                      "rel_l2_vs_all_full_mean": round(sum(errs) / steps, 5),
                      "rel_l2_vs_all_full_cached_steps_mean": round(sum(cached) / max(len(cached), 1), 5),
                      "rel_l2_vs_all_full_max": round(max(errs), 5)}
        del stack
        torch.cuda.empty_cache()
    ref = None
    base = runs["all_full"]["trajectory_ms"]
    for r in runs.values():
        r["speedup_vs_all_full"] = round(base / r["trajectory_ms"], 3)
    out["stacks"] = {"blocks": len(blocks), "steps": steps, "anchors": n_anchor,
                     "schedule": {"n_full": n_full, "r_min": r_min, "r_max": r_max, "alpha": alpha,
                                  "step_only_refresh": refresh, "latent_only_ratio": w.ratio},
                     "runs": runs,
                     "data": "synthetic trajectory whose per-frame change scales with the audio "
                             "energy (0.2 + 0.8 w_t) and random-init weights (device-generated); the "
                             "distance from the all-full outputs is a numerical proxy, not the "
                             "paper's video-quality metrics"}
    return out


def wan_leg(w, dev, dt, B: int = 2, Lc: int = 512, steps: int = 10):
    """The Wan-style block (qk RMSNorm + 3D RoPE, cross-attention over Lc
    context tokens, a batch of B for classifier-free guidance) on the
    workload's shape with K selected tokens per element: time per call, the
    per-kernel breakdown and the rooflines of its kernels."""
    import torch

    from paper_2608_02474_amd import api, roofline

    L, D, K, F = w.L, w.D, w.K, w.F
    b = 2 if dt == torch.bfloat16 else 4
    p = make_stack_blocks(w, dev, dt, 1, 6000 + w.seed)[0]
    g = torch.Generator(device=dev)
    g.manual_seed(7000 + w.seed)
    rnd = lambda *shape, std=0.02: (torch.randn(shape, device=dev, generator=g) * std).to(dt)
    for k in ("wqc", "wkc", "wvc", "woc"):
        p[k] = rnd(D, D)
    for k in ("bqc", "bkc", "bvc", "boc"):
        p[k] = rnd(D)
    for k in ("gq", "gk", "gqc", "gkc", "g3"):
        p[k] = 1.0 + 0.1 * torch.randn(D, device=dev, generator=g)
    p["b3"] = 0.02 * torch.randn(D, device=dev, generator=g)
    x = torch.randn((B, L, D), device=dev, generator=g).to(dt)
    ctx = torch.randn((B, Lc, D), device=dev, generator=g).to(dt)
    idx = torch.cat([bb * L + torch.sort(torch.randperm(L, device=dev, generator=g)[:K]).values
                     for bb in range(B)]).to(torch.int32)
    ws = api.Workspace()
    y = torch.empty((B * K, D), dtype=torch.float32, device=dev)
    grid = (w.T,) + tuple(w.grid)
    call = lambda: api.wan_block_partial(p, x, ctx, idx, [K] * B, w.H, grid, y_sel=y, workspace=ws)
    for _ in range(2):
        call()
    torch.cuda.synchronize()
    api.profile_enable(True)
    api.profile_read()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ktimes = api.profile_read()
    api.profile_enable(False)
    ms = e0.elapsed_time(e1) / steps
    work = roofline.wan_block_work(B, L, K, D, F, Lc, b)
    kernels = {}
    for name, (launches, total) in sorted(ktimes.items(), key=lambda kv: -kv[1][1]):
        avg = total / launches
        e = {"ms_per_call": round(total / steps, 4), "launches_per_call": launches // steps,
             "avg_ms": round(avg, 4)}
        wk = roofline.work_of(name, work)
        if wk is not None and wk[0] > 0:
            amount, kind = wk
            if kind == "flop":
                a = amount / (avg * 1e-3) / 1e12
                e.update(achieved=round(a, 1), unit="TFLOP/s", frac=round(a / roofline.PEAK_BF16_TFLOPS, 4))
            else:
                a = amount / (avg * 1e-3) / 1e9
                e.update(achieved=round(a, 1), unit="GB/s", frac=round(a / roofline.PEAK_HBM_GBS, 4))
        kernels[name] = e
    tf = roofline.wan_block_flops(B, L, K, D, F, Lc) / (ms * 1e-3) / 1e12
    extra = sum(kernels[n]["ms_per_call"] for n in kernels
                if n.startswith(("qk_norm_rope", "gemm_qc", "gemm_kvc", "gemm_oc", "attn_cross", "rope_table",
                                 "vec_shift")))
    return {"batch": B, "context_tokens": Lc, "selected_per_element": K, "ms_per_call": round(ms, 3),
            "tokens_per_s": round(B * L / (ms * 1e-3), 1), "tflops": round(tf, 1),
            "frac_bf16_peak": round(tf / roofline.PEAK_BF16_TFLOPS, 4),
            "extras_ms_per_call": round(extra, 3), "kernels": kernels,
            "data": "random-init weights and synthetic tokens, context and selection (device-generated)"}


def hbm_isolated_leg(blk, X, fw, w, dev, iters: int = 20):
    """The streaming kernels of the step timed alone: each launch is preceded
    by a read sweep over 1 GiB, which leaves the 256 MB MALL holding clean
    lines of other data (none of the kernel's inputs, and no dirty lines whose
    write-back the kernel would pay for).  Inside the step, the saliency pass
    follows the previous step's cache update, whose ~0.9 GB of writes are
    still partly dirty in the MALL and are written back during the saliency
    reads."""
    import torch

    from paper_2608_02474_amd import api, roofline

    # fp32, so that sum() reads it in place (an int32 sum would first widen it
    # to int64, writing 2 GiB)
    sweep = torch.ones(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
    b = 2 if X.dtype == torch.bfloat16 else 4
    work = roofline.kernel_work(w.L, w.K, w.D, w.F, b, w.n_samples)
    calls = {
        "saliency_rows": lambda: api.select(X, blk.xref, fw, w.N, k=w.K, xi=blk.xi, out=blk.sel,
                                            workspace=blk.sel_ws),
        "cache_update": lambda: api.cache_update(X, blk.sel.idx, blk.sel.mask, w.K, blk.y_sel, blk.xref,
                                                 blk.codes, blk.scale, blk.y),
    }
    out = {}
    for prefix, fn in calls.items():
        fn()
        torch.cuda.synchronize()
        api.profile_enable(True)
        api.profile_read()
        for _ in range(iters):
            sweep.sum()
            fn()
        torch.cuda.synchronize()
        kt = api.profile_read()
        api.profile_enable(False)
        name = next(n for n in kt if n.startswith(prefix))
        launches, total = kt[name]
        avg = total / launches
        amount = roofline.work_of(name, work)[0]
        ach = amount / (avg * 1e-3) / 1e9
        out[name] = {"avg_ms": round(avg, 4), "launches": launches, "achieved": round(ach, 1),
                     "unit": "GB/s", "frac": round(ach / roofline.PEAK_HBM_GBS, 4), "per_launch": amount}
    del sweep
    return {"protocol": "each launch after a 1 GiB read sweep (clean MALL, inputs not cached)",
            "kernels": out}


def _timed_steps(step, steps: int, warmup: int = 2):
    """ms per call of step() over `steps` calls (HIP events on the current
    stream), plus the library's per-kernel record of those calls."""
    import torch

    from paper_2608_02474_amd import api

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    api.profile_enable(True)
    api.profile_read()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    kt = api.profile_read()
    api.profile_enable(False)
    return start.elapsed_time(stop) / steps, kt


def _block_frac(kt, steps, L, K, D, F):
    from paper_2608_02474_amd import roofline

    block_ms = sum(v[1] for n, v in kt.items() if n.startswith(("modln", "gemm_", "attn_fwd"))) / steps
    tf = roofline.block_flops(L, K, D, F) / (block_ms * 1e-3) / 1e12
    return round(block_ms, 4), round(tf / roofline.PEAK_BF16_TFLOPS, 4)


def sweep_leg(w, blk, X, dev, steps: int = 10):
    """The 32760-token block swept over the recompute ratio (1.0 recomputes
    every token: the full block) under the three audio energy profiles of the
    sweep; the whole step (energy, selection, partial block, cache update) is
    timed, as in the main measurement."""
    import torch

    import synth
    from paper_2608_02474_amd import api

    out = {"ratios": list(synth.SWEEP_RATIOS), "profiles": {}}
    for prof in synth.SWEEP_AUDIO:
        A = torch.from_numpy(synth.make_audio(prof, w.n_samples, w.sample_rate, w.seed)).to(dev)
        res = {}
        for r in synth.SWEEP_RATIOS:
            K = api.topk_count(r, w.L)

            def step():
                _, _, fw = api.energy(A, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
                return blk.step(X, fw, w.N, k=K)
            ms, kt = _timed_steps(step, steps)
            bms, frac = _block_frac(kt, steps, w.L, K, w.D, w.F)
            res[str(r)] = {"K": K, "ms_per_step": round(ms, 4), "tokens_per_s": round(w.L / (ms * 1e-3), 1),
                           "recomputed_tokens_per_s": round(K / (ms * 1e-3), 1),
                           "block_partial_ms": bms, "block_frac_bf16_peak": frac}
        out["profiles"][prof] = res
    return out


def p720_leg(dev, dt, steps: int = 10):
    """The 720p-shaped block (21 x 45 x 80 = 75600 tokens, ratio 0.3): whole-step
    tokens/s and the cache footprint (int8 codes, fp32 scales, the bf16 reference)."""
    import torch

    import synth
    from paper_2608_02474_amd import api

    w = synth.WAN14B_720P
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    audio = synth.make_audio(w.audio, w.n_samples, w.sample_rate, w.seed)
    P = {k: torch.from_numpy(v).to(torch.float32 if k == "mod" else dt).to(dev) for k, v in p.items()}
    X = torch.from_numpy(x).to(dt).to(dev)
    XR = torch.from_numpy(xref).to(dt).to(dev)
    A = torch.from_numpy(audio).to(dev)
    del p, x, xref
    blk = api.CachedBlock(P, w.H, w.L, w.D, dev, dt)
    blk.init(XR)
    torch.cuda.synchronize()

    def step():
        _, _, fw = api.energy(A, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
        return blk.step(X, fw, w.N, k=w.K)
    ms, kt = _timed_steps(step, steps)
    bms, frac = _block_frac(kt, steps, w.L, w.K, w.D, w.F)
    b = 2 if dt == torch.bfloat16 else 4
    codes, scale, ref = w.L * w.D, 4 * w.L, w.L * w.D * b
    return {"workload": w.name, "tokens": w.L, "recomputed_tokens": w.K, "ratio": w.ratio,
            "ms_per_step": round(ms, 4), "tokens_per_s": round(w.L / (ms * 1e-3), 1),
            "recomputed_tokens_per_s": round(w.K / (ms * 1e-3), 1),
            "block_partial_ms": bms, "block_frac_bf16_peak": frac,
            "cache_bytes": {"codes_int8": codes, "scale_fp32": scale, "reference": ref,
                            "total": codes + scale + ref, "bf16_output_cache_for_comparison": w.L * w.D * 2},
            "data": "synthetic (seeded; 720p-shaped latents, random-init block weights, speech-like audio)"}


def sustained_leg(out, kernels, work, w, args):
    """The rate a dense bf16 MFMA stream sustains on this device with Gaussian
    operands (A ~ N(0, 1), B ~ N(0, 0.02)) in the attention's and the GEMM's
    instruction patterns (echo_mfma_ceiling), and the path's matrix kernels
    against it: the nominal peak assumes a clock the part holds only while the
    matrix cores switch few bits."""
    from paper_2608_02474_amd import api, roofline
    ceil = {pat: api.mfma_ceiling(pat, "gaussian", args.ceiling_secs) for pat in ("attention", "gemm")}
    res = {"attention_pattern_tflops": round(ceil["attention"], 1), "gemm_pattern_tflops": round(ceil["gemm"], 1),
           "attention_pattern_frac_of_peak": round(ceil["attention"] / roofline.PEAK_BF16_TFLOPS, 4),
           "gemm_pattern_frac_of_peak": round(ceil["gemm"] / roofline.PEAK_BF16_TFLOPS, 4),
           "seconds_each": args.ceiling_secs,
           "what": "echo_mfma_ceiling: dense bf16 MFMAs with nothing else in the loop, Gaussian operands"}
    per = {}
    for name, k in kernels.items():
        if k.get("unit") != "TFLOP/s":
            continue
        c = ceil["attention"] if name.startswith("attn_") else ceil["gemm"]
        per[name] = round(k["achieved"] / c, 4)
    res["kernels_frac_of_sustained"] = per
    # the block's matrix work at the two sustained rates against its measured time
    attn = roofline.work_of("attn_fwd_bf16", work)
    attn_flop = attn[0] if attn else 0.0
    gemm_flop = roofline.block_flops(w.L, w.K, w.D, w.F) - attn_flop
    ideal_ms = (attn_flop / ceil["attention"] + gemm_flop / ceil["gemm"]) / 1e9
    res["block_partial_frac_of_sustained"] = round(ideal_ms / out["block_partial"]["ms"], 4)
    roof = out["roofline"]
    c = ceil["attention"] if roof["kernel"].startswith("attn_") else ceil["gemm"]
    if roof.get("unit") == "TFLOP/s" and roof.get("achieved"):
        roof["sustained"] = round(c, 1)
        roof["frac_of_sustained"] = round(roof["achieved"] / c, 4)
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wan14b_480p_32760tok")
    ap.add_argument("--stack-blocks", type=int, default=40,
                    help="blocks of the stack leg (the scheduled multi-block trajectory); 0: skip")
    ap.add_argument("--stack-steps", type=int, default=10)
    ap.add_argument("--variant-blocks", type=int, default=10,
                    help="blocks of the ablation-variants leg (anchors, schedules, codecs); 0: skip")
    ap.add_argument("--variant-steps", type=int, default=10)
    ap.add_argument("--wan-batch", type=int, default=2,
                    help="batch of the Wan-style block leg (classifier-free guidance pair); 0: skip")
    ap.add_argument("--wan-context", type=int, default=512)
    ap.add_argument("--sweep-steps", type=int, default=10,
                    help="timed steps per (ratio, audio profile) of the ratio-sweep leg; 0: skip")
    ap.add_argument("--p720-steps", type=int, default=10,
                    help="timed steps of the 720p-shaped block leg; 0: skip")
    ap.add_argument("--dist-steps", type=int, default=50,
                    help="uninstrumented steps of the step-time distribution (at least --steps)")
    ap.add_argument("--dense-steps", type=int, default=None,
                    help="timed calls of the dense block over every token (default: --steps); 0 leaves "
                         "the leg out (profiler runs: its launches would share grids with the cached step's)")
    ap.add_argument("--ceiling-secs", type=float, default=3.0,
                    help="seconds of each sustained-MFMA-rate measurement (attention and GEMM "
                         "instruction patterns on Gaussian operands); 0 leaves the leg out")
    ap.add_argument("--skip-cpu-baseline", action="store_true",
                    help="leave out the CPU oracle leg (profiler runs); the timed GPU step is "
                         "unchanged")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the cached block step runs on a single MI355X "
              "(multi-GPU sharding is designed, not built). Run with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    from paper_2608_02474_amd import api, roofline

    if args.workload not in synth.ALL:
        print(f"unknown workload {args.workload}; choose from {sorted(synth.ALL)}", file=sys.stderr)
        return 2
    w = synth.ALL[args.workload]
    dev = torch.device("cuda:0")
    dt = {"bf16": torch.bfloat16, "f32": torch.float32}[w.dtype]
    b = 2 if w.dtype == "bf16" else 4

    log(f"workload {w.name}: L={w.L} K={w.K} D={w.D} H={w.H} F={w.F}; generating inputs")
    p = synth.make_block_weights(w)
    xref, x = synth.make_latents(w)
    audio = synth.make_audio(w.audio, w.n_samples, w.sample_rate, w.seed)
    P = {k: torch.from_numpy(v).to(torch.float32 if k == "mod" else dt).to(dev) for k, v in p.items()}
    X = torch.from_numpy(x).to(dt).to(dev)
    XR = torch.from_numpy(xref).to(dt).to(dev)
    A = torch.from_numpy(audio).to(dev)

    blk = api.CachedBlock(P, w.H, w.L, w.D, dev, dt)
    blk.init(XR)                              # fill the cache: every token recomputed once
    torch.cuda.synchronize()

    def step():
        _, _, fw = api.energy(A, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
        return blk.step(X, fw, w.N, k=w.K)

    _, _, fw_last = api.energy(A, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # headline: exactly `steps` steps with no library instrumentation
    log(f"timing {args.steps} steps")
    total_ms, per_step = _per_step_times(step, args.steps)
    ms = total_ms / args.steps

    # the step-time distribution over at least 50 more steps, with the shader
    # clock and board power sampled meanwhile (uninstrumented as well)
    n_dist = max(args.dist_steps, args.steps)
    log(f"step-time distribution: {n_dist} steps, clock and power sampled")
    with ClockSampler(0) as clock:
        _, dist = _per_step_times(step, n_dist)
    clock_summary = clock.summary()

    # the plain dense block over every token (no selection, no cache update):
    # the denominator of the cached step's speedup
    n_dense = args.steps if args.dense_steps is None else args.dense_steps
    dense_out = None
    if n_dense > 0:
        log(f"dense block: {n_dense} calls over all {w.L} tokens")

        def dense():
            api.block_partial(P, X, blk.all_idx, w.L, w.H, y_sel=blk.y_sel, workspace=blk.ws, _weights=blk._w)
        dense()
        dense_total, _ = _per_step_times(dense, n_dense)
        dense_ms = dense_total / n_dense
        dense_out = {"ms": round(dense_ms, 4), "tokens_per_s": round(w.L / (dense_ms * 1e-3), 1),
                     "tflops": round(roofline.block_flops(w.L, w.L, w.D, w.F) / (dense_ms * 1e-3) / 1e12, 2),
                     "speedup_of_cached_step": round(dense_ms / ms, 3),
                     "what": "echo_block_partial over all L tokens (no selection, no cache update)"}

    # per-kernel times from a separate, instrumented run of the same steps
    log(f"per-kernel timing: {args.steps} instrumented steps")
    api.profile_enable(True)
    api.profile_read()                        # drop anything recorded so far
    inst_total, _ = _per_step_times(step, args.steps)
    ktimes = api.profile_read()
    api.profile_enable(False)
    inst_ms = inst_total / args.steps

    work = roofline.kernel_work(w.L, w.K, w.D, w.F, b, w.n_samples)
    kernels = {}
    for name, (launches, total_ms) in sorted(ktimes.items(), key=lambda kv: -kv[1][1]):
        avg = total_ms / launches
        wk = roofline.work_of(name, work)
        entry = {"avg_ms": round(avg, 4), "launches": launches,
                 "share": round(total_ms / (inst_ms * args.steps), 4)}
        if wk is not None and wk[0] > 0:
            amount, kind = wk
            if kind == "flop":
                ach = amount / (avg * 1e-3) / 1e12
                entry.update(achieved=round(ach, 2), unit="TFLOP/s",
                             frac=round(ach / roofline.PEAK_BF16_TFLOPS, 4), per_launch=amount)
            else:
                ach = amount / (avg * 1e-3) / 1e9
                entry.update(achieved=round(ach, 1), unit="GB/s",
                             frac=round(ach / roofline.PEAK_HBM_GBS, 4), per_launch=amount)
        kernels[name] = entry

    dom = max(ktimes, key=lambda n: ktimes[n][1])
    d = kernels[dom]
    roof = {"kernel": dom, "bound": "mfma" if d.get("unit") == "TFLOP/s" else "hbm",
            "achieved": d.get("achieved"), "peak": (roofline.PEAK_BF16_TFLOPS if d.get("unit") ==
                                                     "TFLOP/s" else roofline.PEAK_HBM_GBS),
            "unit": d.get("unit"), "frac": d.get("frac"), "per_launch": d.get("per_launch"),
            "avg_ms": d["avg_ms"], "traffic": measured_traffic(dom)}

    block_names = [n for n in ktimes if n.startswith(("modln", "gemm_", "attn_fwd"))]
    block_ms = sum(ktimes[n][1] for n in block_names) / args.steps
    block_tf = roofline.block_flops(w.L, w.K, w.D, w.F) / (block_ms * 1e-3) / 1e12
    sal = kernels.get("saliency_rows_bf16") or kernels.get("saliency_rows_f32") or {}
    cache = kernels.get("cache_update_bf16") or kernels.get("cache_update_f32") or {}

    out = {
        "metric": METRIC, "value": round(w.L / (ms * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded; Wan2.2-S2V-shaped latents, random-init block weights, "
                "speech-like audio)",
        "config": {"workload": w.name, "tokens": w.L, "recomputed_tokens": w.K, "ratio": w.ratio,
                   "latent_frames": w.T, "grid": list(w.grid), "hidden": w.D, "heads": w.H,
                   "ffn": w.F, "audio_samples": w.n_samples},
        "recomputed_tokens_per_s": round(w.K / (ms * 1e-3), 1),
        "step_ms": {"timed_steps": _percentiles(per_step), "distribution": _percentiles(dist),
                    "instrumented_mean": round(inst_ms, 4),
                    "note": "timed_steps: the headline's steps; distribution: max(dist_steps, steps) further "
                            "uninstrumented steps; instrumented_mean: the per-kernel run with two HIP "
                            "events per launch"},
        "clock": dict(clock_summary, during="the distribution steps"),
        "dense_block": dense_out,
        "roofline": roof,
        "block_partial": {"ms": round(block_ms, 4), "tflops": round(block_tf, 2),
                          "frac_bf16_peak": round(block_tf / roofline.PEAK_BF16_TFLOPS, 4)},
        "select_hbm_frac": sal.get("frac"), "cache_hbm_frac": cache.get("frac"),
        "kernels": kernels,
    }
    if not torch.isfinite(blk.y.float()).all():
        log("non-finite block output")
        return 1

    log("streaming kernels alone (clean MALL)")
    out["hbm_isolated"] = hbm_isolated_leg(blk, X, fw_last, w, dev)
    out["select_hbm_frac_isolated"] = out["hbm_isolated"]["kernels"].get("saliency_rows_bf16", {}).get("frac")
    out["cache_hbm_frac_isolated"] = out["hbm_isolated"]["kernels"].get("cache_update_bf16", {}).get("frac")

    if args.sweep_steps > 0 and w.name == "wan14b_480p_32760tok":
        log("ratio sweep leg: ratios x audio profiles")
        out["ratio_sweep"] = sweep_leg(w, blk, X, dev, args.sweep_steps)

    log("adaptive reference cache leg")
    out["refcache"] = refcache_leg(w, dev, dt)
    if args.stack_blocks > 0 or args.variant_blocks > 0:
        blk = None                             # free the main step's block and workspace
        torch.cuda.empty_cache()
        _, fe_stack, fw_stack = api.energy(A, w.T, w.sample_rate, w.n_fft, w.hop, w.n_bands)
        blocks = make_stack_blocks(w, dev, dt, max(args.stack_blocks, args.variant_blocks), 2000 + w.seed)
        if args.stack_blocks > 0:
            log(f"stack leg: {args.stack_blocks} blocks, {args.stack_steps} steps")
            out["stack"] = stack_leg(w, dev, dt, fw_stack, blocks[:args.stack_blocks], args.stack_steps)
        if args.variant_blocks > 0:
            log(f"variants leg: {args.variant_blocks} blocks, {args.variant_steps} steps")
            out["variants"] = variants_leg(w, dev, dt, fe_stack, fw_stack, blocks[:args.variant_blocks],
                                           args.variant_steps)
        blocks = None
    if args.wan_batch > 0:
        log(f"Wan-style block leg: batch {args.wan_batch}, {args.wan_context} context tokens")
        blk = None
        torch.cuda.empty_cache()
        out["wan_block"] = wan_leg(w, dev, dt, B=args.wan_batch, Lc=args.wan_context)

    if args.p720_steps > 0 and w.name != "wan14b_720p_75600tok":
        log("720p-shaped block leg")
        blk = None
        torch.cuda.empty_cache()
        out["p720"] = p720_leg(dev, dt, args.p720_steps)
        torch.cuda.empty_cache()

    if args.ceiling_secs > 0:
        log(f"sustained MFMA rate: attention and GEMM instruction patterns, Gaussian operands, "
            f"{args.ceiling_secs:g} s each")
        blk = None
        torch.cuda.empty_cache()
        out["mfma_sustained"] = sustained_leg(out, kernels, work, w, args)

    if args.skip_cpu_baseline:
        out["cpu_baseline"] = None
    else:
        log("CPU oracle baseline on a bounded sample (fp64)")
        out["cpu_baseline"] = cpu_baseline(w, p, x, xref, audio)
        log("CPU oracle in its fp32 timing mode")
        out["cpu_baseline"]["fp32_timing_mode"] = cpu_baseline_fp32(w, p, x, xref, audio)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
