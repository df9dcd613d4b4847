#!/usr/bin/env python3
"""Benchmark of the strict-prefix linear-attention prefill on one MI355X.

Headline step: the 16-sequence varlen batch (lengths uniform in
[1,024, 8,192] rounded to 16, 77,456 tokens in all; 8 heads, dk = dv = 128,
bf16 q/k/v, fp32 gates and state, chunk 64, cache block C = 256) against a
4,096-page fp32 state pool addressed through a random permutation page
table.  Each sequence has a seeded cache state: cold (nothing cached), a
complete hit, or a partial hit.  One step is one pass of the whole path:

  1. per sequence, the strict-prefix boundary B_i inside its cached prefix
     (host: strict_prefix_boundary);
  2. one la_prefill_paged call over the 16 suffixes [B_i, n_i): each
     (sequence, head) starts from the state page of prefix B_i (the paged
     restore, folded into the scan; cold sequences start from zero), and
     every checkpoint at a multiple of C in (B_i, n_i] goes straight into its
     pool page (the paged save, folded into the scan).

A cold run of the whole batch writes every sequence's checkpoint pages once
before timing.  The step reads only pages of prefixes B_i and writes only
pages after them, so no page is read and written by one call, and what it
writes equals what the cold run wrote (a resume reproduces the recompute
bit for bit), so repeated steps see the same pool.

Timing: per-step intervals from HIP events on the launch stream.  Before
each timed step a 512 MiB buffer is written and another 512 MiB read, which
flushes the MALL (the last level cache) and leaves it clean; ``value`` and
``ms_per_step`` come from the median of those cold-cache steps, with min, mean and a back-to-back warm-cache figure beside
them.  Per-kernel durations come from events the library records inside the
call (la_trace_set_events).  Prefill tokens/s counts the tokens each call
computes (sum of n_i - B_i).

Beside the headline, each on its own timer: the same batch fully cold
(77,456 tokens), the 16-head 32K-token prefill (C = 1,024) and its resume
from 31,744, the one-TP-rank step (3,584 tokens, cold plus the resume from
3,328, as one call), paged save/restore over the full 4,096-page pool,
decode continuation, the host-memory tier and the joint KV + state restore.
The fp64 CPU oracle runs the headline step's work on the host cores.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
       python bench.py --summarize-trace DIR [--steps K]    (rocprofv3 CSV -> markdown)
       python bench.py --summarize-counters DIR... [--steps K]
"""
from __future__ import annotations

import argparse
import ctypes
import gc
import glob
import hashlib
import json
import os
import re
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0            # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0         # MI355X dense bf16 MFMA
CHUNK = 64
MALL_FLUSH_BYTES = 512 << 20

TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "prefill_varlen16_hbm_counters.md")
KERNEL_SOURCES = ["paper_2609_15030_amd/csrc/la_common.h", "paper_2609_15030_amd/csrc/gdr_prep.h",
                  "paper_2609_15030_amd/csrc/gdr_scan.h", "paper_2609_15030_amd/csrc/gdr_xprep.h",
                  "paper_2609_15030_amd/csrc/gdr_xscan.h", "paper_2609_15030_amd/csrc/linattn.hip",
                  "paper_2609_15030_amd/build.py"]


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime torch uses."""

    def __init__(self, n):
        import torch  # noqa: F401  (binds the same libamdhip64 torch loaded)
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
            self.ev.append(e.value)

    def record(self, i, stream):
        assert self.hip.hipEventRecord(self.ev[i], stream) == 0

    def ms(self, a, b):
        assert self.hip.hipEventSynchronize(self.ev[b]) == 0
        out = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(out), self.ev[a], self.ev[b]) == 0
        return float(out.value)


def flops_per_token_head(dk, dv, L=CHUNK):
    """Algorithmic flops per (token, head), triangular products counted once,
    split by the kernel that executes them.  Their sum is
    F_alg = 6 dk dv + L (3 dk + 2 dv) + L^2 / 3.

    prep: K K^T (L dk), (I + A)^-1 (L^2 / 3), and the L dk of the W = X K
          product of the WY form, which the X form here never forms (it is
          counted so that the total is the form-independent figure);
    scan: K S (2 dk dv), K^T U (2 dk dv), Q S (2 dk dv), Q K^T (L dk),
          X Z (L dv), P U (L dv).
    """
    return {"prep": 2 * L * dk + L * L / 3, "scan": 6 * dk * dv + L * (dk + 2 * dv)}


def step_bytes(tokens, heads, dk, dv, n_seqs, ckpt_pages, restored_pages, io=2):
    """Algorithmic HBM bytes of one prefill call: q, k, v read and o written
    (io bytes each), g and beta (fp32), the checkpoint pages written, the
    starting-state pages read and the final states written (fp32 dk x dv)."""
    page = 4 * dk * dv
    return (tokens * heads * (io * (2 * dk + dv) + io * dv + 8)
            + (ckpt_pages + restored_pages + n_seqs * heads) * page)


def kernel_source_hash():
    """SHA-256 of the kernel sources with their comments and blank lines
    removed (a comment edit leaves the recorded counters valid; any change to
    the code does not)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        lines = (re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()


def measured_traffic(role):
    """HBM bytes (read + write) per launch of the kernels of ``role`` from the
    committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary, or None when the
    kernel sources have changed since the counters were taken."""
    try:
        line = next(l for l in open(TRAFFIC_PROFILE) if l.startswith("traffic-record: "))
    except (OSError, StopIteration):
        return None
    rec = json.loads(line[len("traffic-record: "):])
    if rec.get("source_sha256") != kernel_source_hash():
        return None
    r = rec.get("roles", {}).get(role)
    return None if r is None else r["read_bytes"] + r["write_bytes"]


SPIN_CYCLES = 100_000_000   # ~40 ms of GPU spin ahead of each timed loop


class Timer:
    """Per-repetition HIP-event intervals on one stream.  All repetitions are
    queued behind a GPU spin before the first event is read (with Python's
    garbage collector paused), so the host's launch latency and its pauses
    stay outside the intervals."""

    def __init__(self, torch, stream_ptr):
        self.torch = torch
        self.sp = stream_ptr
        self.buf = torch.empty(MALL_FLUSH_BYTES, dtype=torch.uint8, device="cuda")
        self.clean = torch.ones(MALL_FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        self.k = 0

    def flush(self):
        """Write 512 MiB, then read another 512 MiB: the last-level cache then
        holds none of the timed work's data and no dirty lines whose
        write-back the timed work would pay for."""
        self.k = (self.k + 1) & 0xFF
        self.buf.fill_(self.k)
        self.clean.sum()

    def cold(self, run, reps):
        """Per-repetition ms, the MALL flushed before each repetition; the GPU
        time from the first repetition's start to the last one's end (flushes
        included) is kept in ``last_span_ms``."""
        ev = HipEvents(2 * reps)
        self.torch.cuda.synchronize()
        gc.disable()
        try:
            self.torch.cuda._sleep(SPIN_CYCLES)
            for r in range(reps):
                self.flush()
                ev.record(2 * r, self.sp)
                run()
                ev.record(2 * r + 1, self.sp)
        finally:
            gc.enable()
        self.last_span_ms = ev.ms(0, 2 * reps - 1)
        return [ev.ms(2 * r, 2 * r + 1) for r in range(reps)]

    def warm(self, run, reps):
        """Per-repetition ms over back-to-back repetitions (no flush)."""
        ev = HipEvents(2 * reps)
        self.torch.cuda.synchronize()
        gc.disable()
        try:
            self.torch.cuda._sleep(SPIN_CYCLES)
            run()
            for r in range(reps):
                ev.record(2 * r, self.sp)
                run()
                ev.record(2 * r + 1, self.sp)
        finally:
            gc.enable()
        return [ev.ms(2 * r, 2 * r + 1) for r in range(reps)]

    def stages(self, la, run, reps):
        """Mean per-stage ms from the library's trace events (cold cache):
        prep, maps + combine (two-level forms), scan (or replay)."""
        ev = HipEvents(4)
        acc = [0.0, 0.0, 0.0]
        for _ in range(reps):
            self.torch.cuda.synchronize()
            self.torch.cuda._sleep(2_000_000)
            self.flush()
            la.la_trace_set_events(ev.ev)
            run()
            la.la_trace_set_events([])
            for i in range(3):
                acc[i] += ev.ms(i, i + 1)
        return {"prep": acc[0] / reps, "maps_combine": acc[1] / reps, "scan": acc[2] / reps}


def summary(ms):
    return {"median_us": round(statistics.median(ms) * 1e3, 2), "min_us": round(min(ms) * 1e3, 2),
            "mean_us": round(statistics.fmean(ms) * 1e3, 2), "reps": len(ms)}


def form_kernels(la, shape, cu_host, max_segments=1):
    """Kernel names of a bf16 call (dk = dv = 128): the fused scan's widths
    are the library's choice for these lengths (a mix of 32 and 64 columns
    runs as one mixed-width kernel); the segment maps of the two-level form
    take 128 columns while their units give each of the 256 CUs two
    workgroups, else 64."""
    w, narrow = la.la_prefill_scan_columns(shape, cu_host)
    if la.la_prefill_form(shape) == la.LA_FORM_FUSED_SCAN:
        mixed = 0 < narrow < shape.n_seqs * shape.n_heads
        scan = "gdr_xscan_mixed_kernel<128, 128>" if mixed else f"gdr_xscan_kernel<128, 128, 0, {w}>"
        return {"prep": ["gdr_xprep_kernel<128>"], "maps_combine": [], "scan": [scan]}
    units = shape.n_seqs * shape.n_heads * max_segments
    return {"prep": ["gdr_xprep_kernel<128>"],
            "maps_combine": [f"gdr_xscan_kernel<128, 128, 2, {128 if units * 2 >= 512 else 64}>",
                             "gdr_xcombine_kernel<128, 128>"],
            "scan": [f"gdr_xscan_kernel<128, 128, 1, {w}>"]}


class VarlenStep:
    """The headline step's buffers: the batch on the device, the pool after
    the cold run, and the suffix call with its page tables."""

    def __init__(self, api, la, torch, wl):
        w = wl.batched_varlen()
        x, C, H = w.inputs, w.interval, w.inputs.n_heads
        self.w, self.C, self.H, self.dk, self.dv = w, C, H, x.dk, x.dv
        self.la = la
        self.lens = [int(n) for n in np.diff(x.cu_seqlens)]
        self.x = x
        self.xd = api.to_device(x)
        self.pool = torch.empty((w.pool_pages, x.dk * x.dv), dtype=torch.float32, device="cuda")
        self.cold = api.Prefill(self.xd, C, emit_ckpt=False)
        ids = np.full(self.cold.n_ckpt_rows * H, -1, np.int32)
        for i, n in enumerate(self.lens):
            for j in range(n // C):
                for h in range(H):
                    ids[(int(self.cold.ckpt_offsets[i]) + j) * H + h] = w.page_perm[wl.page_slot(i, j, h, H)]
        assert (ids >= 0).all()
        self.cold_ids = torch.from_numpy(ids).cuda()
        self.cold_pages = int(len(ids))
        self.starts = self.boundaries()
        suf = [x.seq(i).tokens(self.starts[i], n) for i, n in enumerate(self.lens)]
        cat = lambda f: np.concatenate([getattr(s, f) for s in suf])
        self.xs = wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"),
                            np.concatenate([[0], np.cumsum([n - b for n, b in zip(self.lens, self.starts)])]
                                           ).astype(np.int32), x.io_dtype)
        self.step_call = api.Prefill(api.to_device(self.xs), C, starts=self.starts, emit_ckpt=False)
        ck = np.full(self.step_call.n_ckpt_rows * H, -1, np.int32)
        st = np.full(len(self.lens) * H, -1, np.int32)
        for i, (n, b) in enumerate(zip(self.lens, self.starts)):
            for r in range(n // C - b // C):
                for h in range(H):
                    ck[(int(self.step_call.ckpt_offsets[i]) + r) * H + h] = \
                        w.page_perm[wl.page_slot(i, b // C + r, h, H)]
            if b > 0:
                for h in range(H):
                    st[i * H + h] = w.page_perm[wl.page_slot(i, b // C - 1, h, H)]
        assert (ck >= 0).all()
        self.ck_ids = torch.from_numpy(ck).cuda()
        self.st_ids = torch.from_numpy(st).cuda()
        self.step_pages = int(len(ck))
        self.restored = int((st >= 0).sum())
        self.tokens = int(self.xs.cu_seqlens[-1])

    def boundaries(self):
        return [self.la.strict_prefix_boundary(n, self.C, a) for n, a in zip(self.lens, self.w.available)]

    def run_cold(self):
        self.cold.run_paged(self.pool, ckpt_page_ids=self.cold_ids)

    def run_step(self):
        assert self.boundaries() == self.starts
        self.step_call.run_paged(self.pool, ckpt_page_ids=self.ck_ids, state_page_ids=self.st_ids)

    def check(self, torch):
        """The step's outputs and final states equal the cold run's, bit for bit."""
        self.run_cold()
        self.run_step()
        torch.cuda.synchronize()
        cu = self.x.cu_seqlens
        for i, (n, b) in enumerate(zip(self.lens, self.starts)):
            a0, a1 = int(self.xs.cu_seqlens[i]), int(self.xs.cu_seqlens[i + 1])
            c0 = int(cu[i])
            assert torch.equal(self.step_call.o[a0:a1], self.cold.o[c0 + b:c0 + n]), i
        assert torch.equal(self.step_call.final, self.cold.final)


def cpu_baseline(v, seconds):
    """The fp64 oracle on the headline step's work (each sequence's suffix
    from its boundary, every head), sequences run concurrently and heads on
    threads, repeated until about ``seconds`` of wall time.  The starting
    states of resumed sequences are seeded values: the oracle's work does not
    depend on them."""
    import concurrent.futures as cf
    import oracle
    affinity = len(os.sched_getaffinity(0))
    threads = min(affinity, int(os.environ.get("OMP_NUM_THREADS", affinity) or affinity))
    per_call = min(v.H, threads)
    workers = max(1, threads // per_call)
    xs, H, dk, dv = v.xs, v.H, v.dk, v.dv
    rng = np.random.default_rng(5)
    s_in = [None if b == 0 else rng.standard_normal((H, dk, dv)) * 0.1 for b in v.starts]
    order = sorted(range(len(v.lens)), key=lambda i: -(v.lens[i] - v.starts[i]))

    def one(i):
        a, b = int(xs.cu_seqlens[i]), int(xs.cu_seqlens[i + 1])
        oracle.gdr_prefill_seq(xs.q[a:b], xs.k[a:b], xs.v[a:b], xs.g[a:b], xs.beta[a:b], start=v.starts[i],
                               interval=v.C, state_in=s_in[i], n_threads=per_call)

    reps = 0
    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        while True:
            list(ex.map(one, order))
            reps += 1
            if time.perf_counter() - t0 >= seconds:
                break
    dt = time.perf_counter() - t0
    model = "unknown"
    try:
        model = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": round(reps * v.tokens / dt, 1), "unit": "tokens/s", "cores": workers * per_call,
            "kind": "oracle",
            "sample": f"{reps} x the headline step ({v.tokens} suffix tokens x {H} heads over {len(v.lens)} "
                      f"sequences), fp64 token loop, {workers} sequences at a time x {per_call} head threads, "
                      f"{dt:.1f} s wall; {affinity} cores in the affinity mask; CPU: {model}"}


def bench_long(api, la, torch, wl, timer, reps):
    """16-head 32K-token prefill (C = 1,024): the cold call (checkpoints to a
    dense array) and the resume of the last 1,024 tokens from the
    checkpoint at 31,744."""
    w = wl.long_prefill()
    x, C = w.inputs, w.interval
    N, H = x.total_tokens, x.n_heads
    cold = api.Prefill(api.to_device(x), C)
    B = la.strict_prefix_boundary(N, C, N)
    j = B // C - 1
    cold.run()
    torch.cuda.synchronize()
    st = cold.ckpt[j:j + 1].clone()
    res = api.Prefill(api.to_device(x.tokens(B, N)), C, starts=[B])
    res.run(st)
    torch.cuda.synchronize()
    assert torch.equal(res.o, cold.o[B:]) and torch.equal(res.final, cold.final)
    fl = flops_per_token_head(x.dk, x.dv)
    ms = timer.cold(lambda: cold.run(), reps)
    stg = timer.stages(la, lambda: cold.run(), max(3, reps // 2))
    ms_r = timer.cold(lambda: res.run(st), reps)
    med = statistics.median(ms) * 1e-3
    return {"workload": w.name, "form": la.la_prefill_form(cold.shape),
            "scan_columns": la.la_prefill_scan_columns(cold.shape, cold.x.cu_host), "tokens": N, "heads": H,
            "cold": dict(summary(ms), tokens_per_s=round(N / med, 1),
                         alg_tflops=round(sum(fl.values()) * N * H / med / 1e12, 2),
                         stage_us={k: round(v * 1e3, 2) for k, v in stg.items()}),
            "resume_from": B, "resume": dict(summary(ms_r), tokens_per_s=round((N - B) / (statistics.median(ms_r) * 1e-3), 1))}


def bench_tp_rank(api, la, torch, wl, timer, reps):
    """One TP rank's share (3,584 tokens, 8 heads, C = 256): the cold prefill
    and the resume of its 256-token suffix from the checkpoint page at 3,328,
    batched as one la_prefill_paged call over two sequences.  The pool holds
    two page regions written on alternate steps, so no page is read and
    written in one call."""
    w = wl.tp_rank_3584()
    x, C = w.inputs, w.interval
    N, H, dk, dv = x.total_tokens, x.n_heads, x.dk, x.dv
    B = la.strict_prefix_boundary(N, C, w.available[0])
    xr = x.tokens(B, N)
    cat = lambda a, b: np.ascontiguousarray(np.concatenate([a, b]))
    batch = wl.Inputs(cat(x.q, xr.q), cat(x.k, xr.k), cat(x.v, xr.v), cat(x.g, xr.g), cat(x.beta, xr.beta),
                      np.array([0, N, N + (N - B)], np.int32), x.io_dtype)
    both = api.Prefill(api.to_device(batch), C, starts=[0, B], emit_ckpt=False)
    rows = both.n_ckpt_rows
    perm = np.random.default_rng(11).permutation(2 * rows * H).astype(np.int32)
    pool = torch.zeros((2 * rows * H, dk * dv), dtype=torch.float32, device="cuda")
    region = [torch.from_numpy(perm[r * rows * H:(r + 1) * rows * H]).cuda() for r in (0, 1)]
    j = B // C - 1
    cold_start = torch.full((H,), -1, dtype=torch.int32, device="cuda")
    state_ids = [torch.cat([cold_start, region[1 - r][j * H:(j + 1) * H]]).contiguous() for r in (0, 1)]
    k = [0]

    def step():
        r = k[0] % 2
        k[0] += 1
        both.run_paged(pool, ckpt_page_ids=region[r], state_page_ids=state_ids[r])

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    assert torch.equal(both.o[N:], both.o[B:N]) and torch.equal(both.final[1], both.final[0])
    ms = timer.cold(step, reps)
    warm = statistics.median(timer.warm(step, reps))
    stg = timer.stages(la, step, max(3, reps // 2))
    T = N + (N - B)
    return {"workload": w.name, "form": la.la_prefill_form(both.shape),
            "scan_columns": la.la_prefill_scan_columns(both.shape, both.x.cu_host), "tokens_per_step": T,
            "restore_at": B, "step": dict(summary(ms), tokens_per_s=round(T / (statistics.median(ms) * 1e-3), 1)),
            "warm_us": round(warm * 1e3, 2), "stage_us": {k: round(v * 1e3, 2) for k, v in stg.items()}}


def bench_sweep(api, la, torch, wl, timer, reps):
    """The nine-length serial sweep (T = 512 i, 8 heads, d = 128, bf16,
    C = 256): per length, the cold paged prefill (every checkpoint into its
    pool page) and the resume of the suffix from the strict-prefix page, each
    timed on its own after a cache flush; the resume's output is checked
    against the cold run's suffix, bit for bit."""
    rows_out = []
    for w in wl.nine_length_sweep():
        x, C = w.inputs, w.interval
        N, H, dk, dv = x.total_tokens, x.n_heads, x.dk, x.dv
        B = la.strict_prefix_boundary(N, C, w.available[0])
        cold = api.Prefill(api.to_device(x), C, emit_ckpt=False)
        res = api.Prefill(api.to_device(x.tokens(B, N)), C, starts=[B], emit_ckpt=False)
        pool = torch.zeros((cold.n_ckpt_rows * H, dk * dv), dtype=torch.float32, device="cuda")
        ids = torch.arange(cold.n_ckpt_rows * H, dtype=torch.int32, device="cuda")
        j = B // C - 1
        st_ids = ids[j * H:(j + 1) * H].contiguous()
        ck_ids = ids[(j + 1) * H:(j + 1 + res.n_ckpt_rows) * H].contiguous()
        run_cold = lambda: cold.run_paged(pool, ckpt_page_ids=ids)
        run_res = lambda: res.run_paged(pool, ckpt_page_ids=ck_ids, state_page_ids=st_ids)
        run_cold()
        run_res()
        torch.cuda.synchronize()
        assert torch.equal(res.o, cold.o[B:]) and torch.equal(res.final, cold.final)
        mc = statistics.median(timer.cold(run_cold, reps))
        mr = statistics.median(timer.cold(run_res, reps))
        rows_out.append({"T": N, "restore_at": B, "cold_us": round(mc * 1e3, 2),
                         "cold_tokens_per_s": round(N / (mc * 1e-3), 1), "resume_us": round(mr * 1e3, 2),
                         "ckpt_pages": cold.n_ckpt_rows * H})
    return {"workload": "sweep_T512..4608_H8_d128_bf16_C256", "runs": rows_out}


def bench_decode(la, torch, stream_ptr, H, dk, dv, C, batches=(1, 64), steps=200):
    """Decode continuation: one token per (sequence, head) per call, state read
    and written in HBM (2 x 4 dk dv bytes per head-token)."""
    out = {}
    ev = HipEvents(2)
    for n in batches:
        shape = la.make_shape(n, H, dk, dv, C)
        q = torch.randn((n, H, dk), device="cuda").to(torch.bfloat16)
        k = torch.nn.functional.normalize(torch.randn((n, H, dk), device="cuda"), dim=-1).to(torch.bfloat16)
        v = torch.randn((n, H, dv), device="cuda").to(torch.bfloat16)
        g = -torch.nn.functional.softplus(torch.randn((n, H), device="cuda"))
        beta = torch.sigmoid(torch.randn((n, H), device="cuda"))
        state = torch.zeros((n, H, dk, dv), device="cuda")
        o = torch.empty((n, H, dv), dtype=torch.bfloat16, device="cuda")
        for _ in range(20):
            la.la_decode_step(shape, q, k, v, g, beta, state, o)
        ev.record(0, stream_ptr)
        for _ in range(steps):
            la.la_decode_step(shape, q, k, v, g, beta, state, o)
        ev.record(1, stream_ptr)
        us = ev.ms(0, 1) / steps * 1e3
        gbps = 2.0 * 4 * dk * dv * n * H / (us * 1e-6) / 1e9
        out[f"{n}x{H}"] = {"us_per_step": round(us, 2), "tokens_per_s": round(n / (us * 1e-6), 1),
                           "state_GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
    return out


def bench_pool(la, torch, timer, n_pages=4096, page_elems=128 * 128, reps=20):
    """Full-pool scatter and gather under a random permutation (2 x 256 MiB),
    each repetition after a MALL flush; GB/s = (read + write bytes) / time."""
    rng = np.random.default_rng(7)
    perm = torch.from_numpy(rng.permutation(n_pages).astype(np.int32)).cuda()
    states = torch.randn((n_pages, page_elems), device="cuda")
    pool = torch.empty((n_pages, page_elems), device="cuda")
    back = torch.empty_like(states)
    for _ in range(3):
        la.la_state_save_paged(states, pool, perm)
        la.la_state_restore_paged(pool, perm, back)
    torch.cuda.synchronize()
    assert torch.equal(back, states)
    ms_s = timer.cold(lambda: la.la_state_save_paged(states, pool, perm), reps)
    ms_r = timer.cold(lambda: la.la_state_restore_paged(pool, perm, back), reps)
    nbytes = 2.0 * n_pages * page_elems * 4
    out = {"pages": n_pages, "page_bytes": page_elems * 4, "bytes_per_call": nbytes}
    for name, ms in (("save", ms_s), ("restore", ms_r)):
        med = statistics.median(ms) * 1e-3
        out[name] = dict(summary(ms), GBps=round(nbytes / med / 1e9, 1),
                         frac_hbm=round(nbytes / med / 1e9 / HBM_PEAK_GBPS, 4),
                         best_frac_hbm=round(nbytes / (min(ms) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4))
    return out


def bench_host_tier(la, torch, timer, sizes=(112, 4096), page_elems=128 * 128, reps=10):
    """Pages between device states and a pinned host pool (the host tier):
    payload bytes per second over the host link, each direction."""
    out = {}
    for n in sizes:
        perm = torch.from_numpy(np.random.default_rng(8).permutation(n).astype(np.int32)).cuda()
        states = torch.randn((n, page_elems), device="cuda")
        pool = torch.empty((n, page_elems), dtype=torch.float32, pin_memory=True)
        back = torch.empty_like(states)
        la.la_state_save_host(states, pool, perm)
        la.la_state_restore_host(pool, perm, back)
        torch.cuda.synchronize()
        assert torch.equal(back, states)
        ms_s = timer.cold(lambda: la.la_state_save_host(states, pool, perm), reps)
        ms_r = timer.cold(lambda: la.la_state_restore_host(pool, perm, back), reps)
        nbytes = n * page_elems * 4
        out[f"{n}_pages"] = {"bytes": nbytes,
                             "d2h_GBps": round(nbytes / (statistics.median(ms_s) * 1e-3) / 1e9, 1),
                             "h2d_GBps": round(nbytes / (statistics.median(ms_r) * 1e-3) / 1e9, 1),
                             "d2h_us": round(statistics.median(ms_s) * 1e3, 1),
                             "h2d_us": round(statistics.median(ms_r) * 1e3, 1)}
    return out


KV_TOKEN_BYTES = 8268    # attention entries per token per rank, fixed by the paper's reload byte counts
KV_BLOCK_TOKENS = 16


def bench_hybrid(la, torch, timer, n_tokens=3584, interval=256, n_heads=8, page_elems=128 * 128, reps=20):
    """Joint restore at the one-TP-rank reload: the attention KV blocks of the
    prefix [0, B) (opaque bytes, 8,268 per token) and the 8 state pages of the
    checkpoint at B, in one launch, from a device pool and from a pinned
    host pool.  Payload GB/s; the device-pool figure also as HBM traffic
    (read + write) against the HBM peak."""
    B, nb = la.la_hybrid_boundary(n_tokens, interval, KV_BLOCK_TOKENS, n_tokens, n_tokens)
    block = KV_TOKEN_BYTES * KV_BLOCK_TOKENS
    rng = np.random.default_rng(9)
    n_blocks = n_tokens // KV_BLOCK_TOKENS
    kv_dev = torch.randint(0, 256, (n_blocks, block), dtype=torch.uint8, device="cuda")
    kv_host = torch.empty((n_blocks, block), dtype=torch.uint8, pin_memory=True)
    kv_host.copy_(kv_dev)
    n_pages = 14 * n_heads
    st_dev = torch.randn((n_pages, page_elems), device="cuda")
    st_host = torch.empty((n_pages, page_elems), dtype=torch.float32, pin_memory=True)
    st_host.copy_(st_dev)
    cache = torch.empty((nb + 16, block), dtype=torch.uint8, device="cuda")
    src = torch.from_numpy(rng.permutation(n_blocks)[:nb].astype(np.int32)[None]).cuda()
    dst = torch.from_numpy(rng.permutation(nb + 16)[:nb].astype(np.int32)[None]).cuda()
    sid = torch.from_numpy(rng.permutation(n_pages)[:n_heads].astype(np.int32)).cuda()
    states = torch.empty((n_heads, page_elems), device="cuda")
    bdev = torch.tensor([B], dtype=torch.int64, device="cuda")
    payload = nb * block + n_heads * page_elems * 4
    out = {"boundary": B, "kv_blocks": nb, "kv_block_bytes": block, "payload_bytes": payload}
    for name, kvp, stp in (("device_pool", kv_dev, st_dev), ("host_pool", kv_host, st_host)):
        kv = la.make_kv_blocks(kvp, cache, src, dst, KV_BLOCK_TOKENS)
        for _ in range(3):
            la.la_hybrid_restore(kv, bdev, [B], stp, sid, states, n_heads)
        torch.cuda.synchronize()
        ms = timer.cold(lambda: la.la_hybrid_restore(kv, bdev, [B], stp, sid, states, n_heads), reps)
        us = statistics.median(ms) * 1e3
        gbps = payload / (us * 1e-6) / 1e9
        out[name] = {"us": round(us, 2), "payload_GBps": round(gbps, 1)}
        if name == "device_pool":
            out[name]["hbm_frac"] = round(2 * gbps / HBM_PEAK_GBPS, 4)
    got = cache[dst[0].long()].cpu()
    assert torch.equal(got, kv_dev[src[0].long()].cpu()) and torch.equal(states, st_dev[sid.long()])
    return out


def headline(args, torch, api, la, wl, timer, sp):
    v = VarlenStep(api, la, torch, wl)
    v.run_cold()                                  # every checkpoint page, once
    for _ in range(max(args.warmup, 1)):
        v.run_step()
    v.check(torch)
    # the timed region: K steps, each after a MALL flush
    torch.cuda.synchronize()
    ms = timer.cold(v.run_step, args.steps)
    torch.cuda.synchronize()
    res = {"v": v, "ms": ms, "span": timer.last_span_ms}
    if args.only_headline:
        n = 4096
        perm = torch.from_numpy(np.random.default_rng(7).permutation(n).astype(np.int32)).cuda()
        src = torch.randn((n, 128 * 128), device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            la.la_state_save_paged(src, dst, perm)
        torch.cuda.synchronize()
        return res
    res["warm"] = timer.warm(v.run_step, args.steps)
    res["stages"] = timer.stages(la, v.run_step, max(10, args.steps // 2))
    res["cold_ms"] = timer.cold(v.run_cold, max(5, args.steps // 2))
    res["cold_stages"] = timer.stages(la, v.run_cold, max(5, args.steps // 4))
    return res


def roofline_of(v, la, stages, dk, dv, tokens):
    """The dominant stage of the call and its fraction of the bf16 MFMA peak
    (algorithmic flops) and of the HBM peak (algorithmic bytes)."""
    fl = flops_per_token_head(dk, dv)
    scan_ms = stages["maps_combine"] + stages["scan"]
    dom = "prep" if stages["prep"] > scan_ms else "scan"
    dur = stages["prep"] if dom == "prep" else scan_ms
    flops = fl[dom] * tokens * v.H
    achieved = flops / (dur * 1e-3) / 1e12
    fk = form_kernels(la, v.step_call.shape, v.xs.cu_seqlens)
    kernels = fk[dom] if dom == "prep" else fk["maps_combine"] + fk["scan"]
    return {"bound": "mfma", "kernel": " + ".join(kernels), "achieved": round(achieved, 3),
            "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 5),
            "traffic": measured_traffic("step " + dom),
            "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated on a copy)",
            "flops_per_launch": flops, "avg_launch_us": round(dur * 1e3, 2)}


# ---------------------------------------------------------------------------
# rocprofv3 CSV summaries (runs of ``bench.py --only-headline``).  In such a
# run each prefill kernel's last K dispatches are the K timed steps; the
# earlier ones are the cold run, the warmup and the check.  The run ends
# with three full-pool paged saves (256 MiB read + 256 MiB written each),
# the copy that calibrates the byte counters.

def _csv_rows(dirs, suffix):
    import csv
    rows = []
    for d in dirs:
        for f in sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)):
            with open(f, newline="") as fh:
                rows.extend(csv.DictReader(fh))
    return rows


def _short(name):
    name = name.replace("void ", "").replace("la::", "")
    depth, out = 0, []
    for ch in name:          # drop the argument list, keep template arguments
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip()


def _role(kernel, index, count, steps):
    if kernel.startswith("page_save_kernel"):
        return "calibration copy"
    if kernel.startswith(("gdr_xprep_", "gdr_xscan_", "gdr_xcombine_")):
        return "step" if index >= count - steps else "cold run, warmup, check"
    return "other"


def trace_markdown(d, steps):
    rows = _csv_rows([d], "kernel_trace.csv")
    by = {}
    for r in sorted(rows, key=lambda r: int(r["Dispatch_Id"])):
        by.setdefault(_short(r["Kernel_Name"]), []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    lines = ["| kernel | role | calls | avg us | min us | max us |", "|---|---|---|---|---|---|"]
    for k, ds in sorted(by.items()):
        roles = {}
        for i, t in enumerate(ds):
            roles.setdefault(_role(k, i, len(ds), steps), []).append(t)
        for role, ts in roles.items():
            if role == "other":
                continue
            lines.append(f"| {k} | {role} | {len(ts)} | {statistics.fmean(ts):.2f} | {min(ts):.2f} | {max(ts):.2f} |")
    return "\n".join(lines)


def counters_markdown(dirs, steps):
    rows = _csv_rows(dirs, "counter_collection.csv")
    trace = _csv_rows(dirs, "kernel_trace.csv")
    per = {}                                   # (counter, kernel) -> values in dispatch order
    for r in sorted(rows, key=lambda r: int(r["Dispatch_Id"])):
        per.setdefault((r["Counter_Name"], _short(r["Kernel_Name"])), []).append(float(r["Counter_Value"]))
    dur = {}
    for r in sorted(trace, key=lambda r: int(r["Dispatch_Id"])):
        dur.setdefault(_short(r["Kernel_Name"]), []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    cal = 4096 * 128 * 128 * 4
    factor = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        v = [x for (cn, k), xs in per.items() if cn == c and k.startswith("page_save_kernel") for x in xs]
        if v:
            factor[c] = cal / (statistics.fmean(v) * 1024)
    out = [f"Copy calibration (full-pool paged save, {cal:,} B each way): " +
           ", ".join(f"{c}: 1 KiB reads as {f:.4f} KiB" for c, f in factor.items()), "",
           "| kernel | role | counter | dispatches | mean per dispatch |", "|---|---|---|---|---|"]
    step_vals = {}
    for (c, k), xs in sorted(per.items()):
        if not k.startswith(("gdr_xprep_", "gdr_xscan_", "gdr_xcombine_")):
            continue
        sel = xs[len(xs) - steps:] if len(xs) >= steps else xs
        m = statistics.fmean(sel)
        step_vals[(c, k)] = m
        out.append(f"| {k} | step | {c} | {len(sel)} | {m:,.1f} |")
    rec = {"source_sha256": kernel_source_hash(), "roles": {}}
    stage_of = {"gdr_xprep_kernel": "prep"}
    roles = {}
    for (c, k), m in step_vals.items():
        if c not in factor or not k.startswith(("gdr_xprep_", "gdr_xscan_", "gdr_xcombine_")):
            continue
        stage = stage_of.get(k.split("<")[0], "scan")
        key = "read_bytes" if c == "FETCH_SIZE" else "write_bytes"
        roles.setdefault("step " + stage, {"read_bytes": 0, "write_bytes": 0})[key] += int(m * 1024 * factor[c])
    rec["roles"] = roles
    if roles:
        out += ["", "| stage | HBM read MB | HBM write MB |", "|---|---|---|"]
        for s_, r in sorted(roles.items()):
            out.append(f"| {s_} | {r['read_bytes'] / 1e6:.2f} | {r['write_bytes'] / 1e6:.2f} |")
    busy = {k: m for (c, k), m in step_vals.items() if c == "SQ_VALU_MFMA_BUSY_CYCLES"}
    mops = {k: m for (c, k), m in step_vals.items() if c == "SQ_INSTS_VALU_MFMA_MOPS_BF16"}
    gui = {k: m for (c, k), m in step_vals.items() if c == "GRBM_GUI_ACTIVE"}
    if mops:
        out += ["", "GRBM_GUI_ACTIVE sums the 8 XCDs (it reads 8x the kernel's cycles at 2.4 GHz), so the MFMA "
                "busy fraction is SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1,024 SIMDs).", "",
                "| kernel | trace avg us (step) | executed bf16 MFMA flops (MOPS x 512) | executed TFLOP/s | "
                "% of 2,500 | MFMA busy fraction |", "|---|---|---|---|---|---|"]
        for k, m in sorted(mops.items()):
            if not k.startswith(("gdr_xprep_", "gdr_xscan_", "gdr_xcombine_")):
                continue
            ds = dur.get(k, [])
            t = statistics.fmean(ds[len(ds) - steps:]) if ds else float("nan")
            fl = m * 512
            util = busy.get(k, float("nan")) / (gui.get(k, float("nan")) / 8 * 1024) if k in gui else float("nan")
            out.append(f"| {k} | {t * 1e6:.2f} | {fl:,.0f} | {fl / t / 1e12:.1f} | "
                       f"{100 * fl / t / 1e12 / BF16_PEAK_TFLOPS:.2f} | {util:.4f} |")
    out += ["", "traffic-record: " + json.dumps(rec)]
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="headline step, its stages and the cold batch only")
    ap.add_argument("--only-headline", action="store_true",
                    help="the cold run, the warmup and the K timed steps only (for counter runs)")
    ap.add_argument("--summarize-trace", metavar="DIR")
    ap.add_argument("--summarize-counters", metavar="DIR", nargs="+")
    args = ap.parse_args()
    if args.summarize_trace:
        print(trace_markdown(args.summarize_trace, args.steps))
        return
    if args.summarize_counters:
        print(counters_markdown(args.summarize_counters, args.steps))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path holds one tensor-parallel rank's heads and needs no "
              "collectives, and only one GPU is used; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_15030_amd import api
    from paper_2609_15030_amd import linattn as la
    from paper_2609_15030_amd import workloads as wl

    torch.cuda.set_device(0)
    sp = torch.cuda.current_stream().cuda_stream
    timer = Timer(torch, sp)
    h = headline(args, torch, api, la, wl, timer, sp)
    v, ms = h["v"], h["ms"]
    T, H, dk, dv = v.tokens, v.H, v.dk, v.dv
    med = statistics.median(ms) * 1e-3
    out = {
        "metric": "linear-attn prefill tokens/s per rank + % MFMA peak; state save/restore GB/s",
        "value": round(T / med, 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(med * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": v.w.name, "n_seqs": len(v.lens), "heads": H, "dk": dk, "dv": dv,
                   "batch_tokens": int(sum(v.lens)), "tokens_per_step": T, "chunk": CHUNK,
                   "ckpt_interval": v.C, "pool_pages": v.w.pool_pages,
                   "modes": {m: v.w.modes.count(m) for m in ("cold", "complete", "partial")}},
        "timing": {"value_from": "median of the K per-step HIP-event intervals, MALL flushed before each",
                   **summary(ms), "gpu_ms_per_step_incl_flush": round(h["span"] / args.steps, 4)},
    }
    if args.only_headline:
        print(json.dumps(out), flush=True)
        return
    st = h["stages"]
    fl = flops_per_token_head(dk, dv)
    out["timing"]["warm"] = summary(h["warm"])
    out["step_call"] = {"form": la.la_prefill_form(v.step_call.shape),
                        "scan_columns": la.la_prefill_scan_columns(v.step_call.shape, v.xs.cu_seqlens),
                        "stage_us": {k: round(x * 1e3, 2) for k, x in st.items()},
                        "alg_tflops": round(sum(fl.values()) * T * H / med / 1e12, 3),
                        "frac_bf16_peak": round(sum(fl.values()) * T * H / med / 1e12 / BF16_PEAK_TFLOPS, 5),
                        "ckpt_pages_written": v.step_pages, "state_pages_read": v.restored}
    alg_b = step_bytes(T, H, dk, dv, len(v.lens), v.step_pages, v.restored)
    out["step_call"]["alg_bytes"] = alg_b
    out["step_call"]["alg_GBps"] = round(alg_b / med / 1e9, 1)
    out["step_call"]["frac_hbm_alg"] = round(alg_b / med / 1e9 / HBM_PEAK_GBPS, 4)
    out["roofline"] = roofline_of(v, la, st, dk, dv, T)
    cm = h["cold_ms"]
    TC = int(sum(v.lens))
    out["cold_batch"] = dict(summary(cm), tokens=TC,
                             tokens_per_s=round(TC / (statistics.median(cm) * 1e-3), 1),
                             alg_tflops=round(sum(fl.values()) * TC * H / (statistics.median(cm) * 1e-3) / 1e12, 2),
                             stage_us={k: round(x * 1e3, 2) for k, x in h["cold_stages"].items()},
                             ckpt_pages_written=v.cold_pages,
                             scan_columns=la.la_prefill_scan_columns(v.cold.shape, v.x.cu_seqlens))
    if not args.no_extras:
        reps = max(10, args.steps // 2)
        out["long_prefill"] = bench_long(api, la, torch, wl, timer, reps)
        out["tp_rank"] = bench_tp_rank(api, la, torch, wl, timer, reps)
        out["sweep"] = bench_sweep(api, la, torch, wl, timer, max(5, reps // 2))
        out["save_restore"] = bench_pool(la, torch, timer)
        out["decode"] = bench_decode(la, torch, sp, H, dk, dv, v.C)
        out["host_tier"] = bench_host_tier(la, torch, timer)
        out["hybrid_restore"] = bench_hybrid(la, torch, timer)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(v, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
