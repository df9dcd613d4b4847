#!/usr/bin/env python3
"""Benchmark of the strict-prefix linear-attention prefill on one MI355X.

One step is one pass of the whole path over the one-TP-rank workload
(8 heads, dk = dv = 128, T = 3,584 bf16 tokens, fp32 state, chunk 64,
checkpoint interval C = 256):

  1. strict-prefix boundary on the host: B = 3,328 for N = 3,584;
  2. cold prefill of all 3,584 tokens, its 14 x 8 fp32 checkpoint pages
     written straight into a pool through a random-permutation page table
     (the paged save folded into the scan);
  3. resume over the 256-token suffix [B, N), its starting state read
     straight from the 8 pages of the checkpoint at B (the paged restore
     folded into the scan) and its checkpoint at N written to a page.

Steps 2 and 3 are two requests that a serving step batches: they go to the
library as one la_prefill_paged call over two sequences (start 0 and start
B).  The resume starts from the checkpoint page of prefix B that the
previous step's cold run wrote: the pool holds two page regions written on
alternate steps, so no page is read and written in the same call (the
call's contract).  The same step issued as two calls, the resume reading
the page its step's cold run has just written, is timed as well
("serial_calls").

Beside the step it reports, each on its own timer: paged save/restore
bandwidth on the full 4,096-page pool, decode continuation (one token per
sequence and head per call, state in HBM) at 1 and 64 sequences, the
host-memory tier (pages to and from a pinned host pool) for the 112
checkpoint pages of a step and for 4,096 pages, and the joint restore of a
hybrid cache at the reload's boundary (the attention KV blocks of [0, B),
8,268 B per token per rank, with the state pages at B) from a device and
from a pinned host pool.

Inputs are resident in HBM before timing starts.  The JSON line reports
whole-step prefill tokens/s (3,584 + 256 tokens per step), the dominant
kernel's roofline (per-kernel durations from HIP events recorded inside the
library on the launch stream), paged save/restore bandwidth on the full
4,096-page pool, and the fp64 CPU oracle's rate on the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0            # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0         # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3          # MI355X dense fp32 MFMA
CHUNK = 64


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
    """Algorithmic flops per (token, head), triangular products counted once.

    prep:  K K^T (L dk), W = X (..K) (L dk), U~ = X (..V) (L dv), inverse (L^2 / 3),
           Q K^T (L dk)
    scan:  W S (2 dk dv), K~^T U (2 dk dv)
    out:   Q S (2 dk dv), P U (L dv)
    """
    return {"prep": 3 * L * dk + L * dv + L * L / 3,
            "scan": 4 * dk * dv,
            "out": 2 * dk * dv + L * dv}


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "prefill_tp_rank_T3584_hbm_counters.md")
SCAN_SOURCES = ["paper_2609_15030_amd/csrc/la_common.h", "paper_2609_15030_amd/csrc/gdr_scan.h",
                "paper_2609_15030_amd/csrc/gdr_out.h",
                "paper_2609_15030_amd/csrc/linattn.hip", "paper_2609_15030_amd/build.py"]


def scan_kernel_name(io_bf16, dk):
    """The scan form the library launches for the benchmark's single-level
    interval (its default choice, or LA_SCAN_WAVES / LA_SCAN_OUTPUT)."""
    forced = os.environ.get("LA_SCAN_WAVES", "")
    waves = int(forced) if forced in ("1", "4") else (4 if (not io_bf16 and dk == 128) else 1)
    if waves != 1:
        return "gdr_scan_kernel"
    return "gdr_scan1_kernel" if os.environ.get("LA_SCAN_OUTPUT", "") == "0" else "gdr_scan1o_kernel"


def measured_traffic(kernel):
    """HBM bytes per cold launch of ``kernel`` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None when the scan sources have changed
    since the counters were taken (or no record exists)."""
    import hashlib
    try:
        line = next(l for l in open(TRAFFIC_PROFILE) if l.startswith("traffic-record: "))
    except (OSError, StopIteration):
        return None
    rec = json.loads(line[len("traffic-record: "):])
    h = hashlib.sha256()
    for f in SCAN_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if rec.get("source_sha256") != h.hexdigest():
        return None
    for r in rec["records"]:
        if r["kernel"] == kernel and r["role"] == "step":
            return r["read_bytes"] + r["write_bytes"]
    return None


def cpu_baseline(w, B, seconds):
    """The fp64 oracle on the same workload (cold prefill + resume), repeated
    until about ``seconds`` of CPU time; threads over heads."""
    import oracle
    x, C, N = w.inputs, w.interval, w.inputs.total_tokens
    threads = min(x.n_heads, len(os.sched_getaffinity(0)))
    t0 = time.perf_counter()
    reps = 0
    used = threads
    while True:
        _, _, ck, used = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=C,
                                                n_threads=threads, return_threads=True)
        xs = x.tokens(B, N)
        oracle.gdr_prefill_seq(xs.q, xs.k, xs.v, xs.g, xs.beta, start=B, interval=C,
                               state_in=ck[B // C - 1], n_threads=threads)
        reps += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    tokens = reps * (N + (N - B))
    return {"value": tokens / dt, "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": f"{reps} x (cold prefill {N} tok + resume {N - B} tok) x {x.n_heads} heads, "
                      f"fp64 token loop, {dt:.1f} s wall"}


def bench_decode(la, torch, stream_ptr, events, H, dk, dv, C, batches=(1, 64), steps=200):
    """Decode continuation: one token per (sequence, head) per call, state read
    and written in HBM (2 x 4 dk dv bytes per head-token)."""
    out = {}
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
        events.record(4, stream_ptr)
        for _ in range(steps):
            la.la_decode_step(shape, q, k, v, g, beta, state, o)
        events.record(5, stream_ptr)
        us = events.ms(4, 5) / steps * 1e3
        gbps = 2.0 * 4 * dk * dv * n * H / (us * 1e-6) / 1e9
        out[f"{n}x{H}"] = {"us_per_step": round(us, 2), "tokens_per_s": round(n / (us * 1e-6), 1),
                           "state_GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
    return out


def bench_host_tier(la, torch, stream_ptr, events, sizes=(112, 4096), page_elems=128 * 128, reps=10):
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
        # every repetition queued before the first event is read (see bench_pool)
        ev = HipEvents(2 * reps + 1)
        la.la_state_restore_host(pool, perm, back)
        ev.record(0, stream_ptr)
        for r in range(reps):
            la.la_state_save_host(states, pool, perm)
            ev.record(2 * r + 1, stream_ptr)
            la.la_state_restore_host(pool, perm, back)
            ev.record(2 * r + 2, stream_ptr)
        ms_s = sum(ev.ms(2 * r, 2 * r + 1) for r in range(reps))
        ms_r = sum(ev.ms(2 * r + 1, 2 * r + 2) for r in range(reps))
        nbytes = n * page_elems * 4
        out[f"{n}_pages"] = {"bytes": nbytes, "d2h_GBps": round(nbytes / (ms_s / reps * 1e-3) / 1e9, 1),
                             "h2d_GBps": round(nbytes / (ms_r / reps * 1e-3) / 1e9, 1),
                             "d2h_us": round(ms_s / reps * 1e3, 1), "h2d_us": round(ms_r / reps * 1e3, 1)}
    return out


def bench_serial_step(api, la, torch, x, B, C, N, H, dk, dv, steps):
    """The step as two calls: the cold prefill (checkpoints into the pool),
    then the resume, its starting state read from the page of prefix B the
    cold run has just written.  Whole-step tokens/s over back-to-back steps."""
    cold = api.Prefill(api.to_device(x), C, emit_ckpt=False)
    resume = api.Prefill(api.to_device(x.tokens(B, N)), C, starts=[B], emit_ckpt=False)
    n_ck = cold.n_ckpt_rows
    pool = torch.empty((n_ck * H, dk * dv), dtype=torch.float32, device="cuda")
    save_ids = torch.from_numpy(np.random.default_rng(12).permutation(n_ck * H).astype(np.int32)).cuda()
    j = B // C - 1
    restore_ids = save_ids[j * H:(j + 1) * H].contiguous()
    resume_ck_ids = save_ids[(j + 1) * H:(j + 1 + resume.n_ckpt_rows) * H].contiguous()

    def step():
        cold.run_paged(pool, ckpt_page_ids=save_ids)
        resume.run_paged(pool, ckpt_page_ids=resume_ck_ids, state_page_ids=restore_ids)

    for _ in range(5):
        step()
    torch.cuda.synchronize()
    assert torch.equal(resume.o, cold.o[B:]) and torch.equal(resume.final, cold.final)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    return {"ms_per_step": round(dt * 1e3, 4), "tokens_per_s": round((N + N - B) / dt, 1)}


def bench_workloads(api, torch, stream_ptr, events, reps=10):
    """Cold prefill (checkpoints to a dense array) of the larger workloads,
    where many chains run side by side: the 16-head 32K-token prefill and
    the 16-sequence varlen batch.  Tokens/s counts every token of the call;
    TFLOP/s uses the algorithmic flops per token-head."""
    from paper_2609_15030_amd import workloads as wl
    out = {}
    for w in (wl.long_prefill(), wl.batched_varlen()):
        x = w.inputs
        xd = api.to_device(x)
        pf = api.Prefill(xd, w.interval)
        for _ in range(2):
            pf.run()
        torch.cuda.synchronize()
        pf.run()   # busy queue at the start event
        events.record(4, stream_ptr)
        for _ in range(reps):
            pf.run()
        events.record(5, stream_ptr)
        us = events.ms(4, 5) / reps * 1e3
        T = x.total_tokens
        fl = sum(flops_per_token_head(x.dk, x.dv).values()) * T * x.n_heads
        out[w.name] = {"tokens": T, "heads": x.n_heads, "ckpt_interval": w.interval, "us": round(us, 1),
                       "tokens_per_s": round(T / (us * 1e-6), 1),
                       "alg_tflops": round(fl / (us * 1e-6) / 1e12, 2),
                       "frac_bf16_peak": round(fl / (us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)}
        del pf, xd
    return out


KV_TOKEN_BYTES = 8268    # attention entries per token per rank, fixed by the paper's reload byte counts
KV_BLOCK_TOKENS = 16


def bench_hybrid(la, torch, stream_ptr, events, n_tokens, interval, n_heads, page_elems=128 * 128, reps=20):
    """Joint restore at the one-TP-rank reload: the attention KV blocks of the
    prefix [0, B) (opaque bytes, 8,268 per token) and the 8 state pages of the
    checkpoint at B, in one launch, from a device pool and from a pinned
    host pool.  Payload GB/s over back-to-back launches; the device-pool
    figure also as HBM traffic (read + write) against the HBM peak."""
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
        # One event pair per launch, all queued behind a GPU spin: the entry
        # point's host-side checks of the pools (pointer-attribute queries)
        # take from a few to ~60 us, longer than a device-pool restore, so an
        # idle GPU would wait for each launch inside its own interval.
        torch.cuda._sleep(20_000_000)
        ev = HipEvents(2 * reps)
        for r in range(reps):
            ev.record(2 * r, stream_ptr)
            la.la_hybrid_restore(kv, bdev, [B], stp, sid, states, n_heads)
            ev.record(2 * r + 1, stream_ptr)
        us = sum(ev.ms(2 * r, 2 * r + 1) for r in range(reps)) / reps * 1e3
        gbps = payload / (us * 1e-6) / 1e9
        out[name] = {"us": round(us, 2), "payload_GBps": round(gbps, 1)}
        if name == "device_pool":
            out[name]["hbm_frac"] = round(2 * gbps / HBM_PEAK_GBPS, 4)
    got = cache[dst[0].long()].cpu()
    assert torch.equal(got, kv_dev[src[0].long()].cpu()) and torch.equal(states, st_dev[sid.long()])
    return out


def bench_pool(la, torch, stream_ptr, events, n_pages=4096, page_elems=128 * 128, reps=20):
    """Full-pool scatter and gather under a random permutation (2 x 256 MiB)."""
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
    # All repetitions are queued before the first event is read: waiting on
    # each repetition would leave the GPU idle at every save's start event,
    # and the save's interval would then hold the host's launch latency.
    ev = HipEvents(2 * reps + 1)
    la.la_state_restore_paged(pool, perm, back)   # the queue is busy when the first event is recorded
    ev.record(0, stream_ptr)
    for r in range(reps):
        la.la_state_save_paged(states, pool, perm)
        ev.record(2 * r + 1, stream_ptr)
        la.la_state_restore_paged(pool, perm, back)
        ev.record(2 * r + 2, stream_ptr)
    ms_save = sum(ev.ms(2 * r, 2 * r + 1) for r in range(reps))
    ms_restore = sum(ev.ms(2 * r + 1, 2 * r + 2) for r in range(reps))
    nbytes = 2.0 * n_pages * page_elems * 4           # read + write
    save = nbytes / (ms_save / reps * 1e-3) / 1e9
    restore = nbytes / (ms_restore / reps * 1e-3) / 1e9
    return {"pages": n_pages, "page_bytes": page_elems * 4, "bytes_per_call": nbytes,
            "save_GBps": round(save, 1), "restore_GBps": round(restore, 1),
            "save_frac_hbm": round(save / HBM_PEAK_GBPS, 4),
            "restore_frac_hbm": round(restore / HBM_PEAK_GBPS, 4),
            "save_us": round(ms_save / reps * 1e3, 2), "restore_us": round(ms_restore / reps * 1e3, 2)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-pool", action="store_true")
    ap.add_argument("--no-workloads", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this path holds one tensor-parallel rank's heads and "
              "needs no collectives; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_15030_amd import api
    from paper_2609_15030_amd import linattn as la
    from paper_2609_15030_amd import workloads as wl

    torch.cuda.set_device(0)
    w = wl.tp_rank_3584()
    x, C = w.inputs, w.interval
    N, H, dk, dv = x.total_tokens, x.n_heads, x.dk, x.dv
    B = la.strict_prefix_boundary(N, C, w.available[0])
    from paper_2609_15030_amd.workloads import Inputs
    xr = x.tokens(B, N)
    cat = lambda a, b: np.ascontiguousarray(np.concatenate([a, b]))
    batch = Inputs(cat(x.q, xr.q), cat(x.k, xr.k), cat(x.v, xr.v), cat(x.g, xr.g), cat(x.beta, xr.beta),
                   np.array([0, N, N + (N - B)], np.int32), x.io_dtype)
    both = api.Prefill(api.to_device(batch), C, starts=[0, B], emit_ckpt=False)
    rows = both.n_ckpt_rows                  # 14 of the cold run, 1 of the resume
    rng = np.random.default_rng(11)
    pool = torch.zeros((2 * rows * H, dk * dv), dtype=torch.float32, device="cuda")
    perm = rng.permutation(2 * rows * H).astype(np.int32)
    region = [torch.from_numpy(perm[r * rows * H:(r + 1) * rows * H]).cuda() for r in (0, 1)]
    j = B // C - 1                            # the cold run's checkpoint row of prefix B
    cold_start = torch.full((H,), -1, dtype=torch.int32, device="cuda")
    # the resume (sequence 1) starts from the page the other region's cold run wrote
    state_ids = [torch.cat([cold_start, region[1 - r][j * H:(j + 1) * H]]).contiguous() for r in (0, 1)]
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    ev = HipEvents(10)
    stage_ev = [ev.ev[0], ev.ev[1], ev.ev[2], ev.ev[3]]
    k_step = [0]

    def step(trace):
        b = la.strict_prefix_boundary(N, C, w.available[0])
        assert b == B
        r = k_step[0] % 2
        k_step[0] += 1
        if trace:
            la.la_trace_set_events(stage_ev)
        # checkpoints straight into region r's pages (the save); the resume's
        # starting state straight from the other region's page of prefix B (the restore)
        both.run_paged(pool, ckpt_page_ids=region[r], state_page_ids=state_ids[r])
        if trace:
            la.la_trace_set_events([])

    for _ in range(max(args.warmup, 2)):      # two steps fill both regions
        step(False)
    torch.cuda.synchronize()
    # parity guard on the benchmarked buffers: the resume equals the cold run's tail
    assert torch.equal(both.o[N:], both.o[B:N]) and torch.equal(both.final[1], both.final[0])

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev.record(8, sp)
    for _ in range(args.steps):
        step(False)
    ev.record(9, sp)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev.ms(8, 9)
    ms_per_step = wall * 1e3 / args.steps
    tokens_per_step = N + (N - B)
    serial = bench_serial_step(api, la, torch, x, B, C, N, H, dk, dv, args.steps)

    # per-kernel durations of the step's call, from events inside the library
    stage = {"prep": 0.0, "scan": 0.0, "out": 0.0}
    n_trace = max(10, args.steps // 2)
    for _ in range(n_trace):
        step(True)
        stage["prep"] += ev.ms(0, 1)
        stage["scan"] += ev.ms(1, 2)
        stage["out"] += ev.ms(2, 3)
    stage_us = {k: v / n_trace * 1e3 for k, v in stage.items()}
    fl = flops_per_token_head(dk, dv)
    scan_name = scan_kernel_name(True, dk)
    fused = scan_name == "gdr_scan1o_kernel"
    # with the scan's output wave the output product runs inside the scan
    # kernel (no output launch: the "out" interval is the gap between two
    # events with no kernel between them)
    kfl = dict(fl, scan=fl["scan"] + fl["out"], out=0.0) if fused else fl
    dom = max(("prep", "scan", "out"), key=stage_us.get)
    achieved = kfl[dom] * tokens_per_step * H / (stage_us[dom] * 1e-6) / 1e12
    prefill_us = sum(stage_us.values())
    kname = {"prep": "gdr_prep_kernel", "scan": scan_name, "out": "gdr_out_kernel"}[dom]
    roofline = {"bound": "mfma", "kernel": kname,
                "achieved": round(achieved, 3), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 5), "traffic": measured_traffic(kname),
                "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)",
                "flops_per_launch": kfl[dom] * tokens_per_step * H, "avg_launch_us": round(stage_us[dom], 2)}

    out = {
        "metric": "linear-attn prefill tokens/s per rank + % MFMA peak; state save/restore GB/s",
        "value": round(tokens_per_step * args.steps / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "n_seqs": 1, "heads": H, "dk": dk, "dv": dv, "T": N,
                   "chunk": CHUNK, "ckpt_interval": C, "restore_at": B,
                   "tokens_per_step": tokens_per_step},
        "gpu_ms_per_step": round(gpu_ms / args.steps, 4),
        "step_call": {"us": round(prefill_us, 2), "tokens_per_s": round(tokens_per_step / (prefill_us * 1e-6), 1),
                      "stage_us": {k: round(v, 2) for k, v in stage_us.items()},
                      "scan_kernel": scan_name, "output_in_scan": fused,
                      "alg_tflops": round(sum(fl.values()) * tokens_per_step * H / (prefill_us * 1e-6) / 1e12, 3)},
        "serial_calls": serial,
        "roofline": roofline,
    }
    if not args.no_pool:
        out["save_restore"] = bench_pool(la, torch, sp, ev)
    out["decode"] = bench_decode(la, torch, sp, ev, H, dk, dv, C)
    if not args.no_pool:
        out["host_tier"] = bench_host_tier(la, torch, sp, ev)
        out["hybrid_restore"] = bench_hybrid(la, torch, sp, ev, N, C, H)
    if not args.no_workloads:
        out["workloads"] = bench_workloads(api, torch, sp, ev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, B, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
