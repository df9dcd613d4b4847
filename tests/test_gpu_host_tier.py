"""GPU tests of the host-memory tier: state pages saved to and restored from a
pinned host pool, through the C ABI.

* round trip of the one-TP-rank checkpoints under a permuted page table into
  a poisoned host pool: saved bytes, untouched pages, -1 and out-of-range ids;
* completion events: a save on a side stream, the device states overwritten
  only after waiting on the save's event, the host pool holds the values from
  before the overwrite; a restore ordered behind the event sees them;
* the whole reload path through host memory: cold prefill, checkpoints to the
  host tier, restore of the page at the strict-prefix boundary, resume, equal
  to the cold run's tail bit for bit;
* pageable host memory is refused before any launch (the call carries only
  -1 ids, so not even a wrong acceptance could touch the pool).
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

pytestmark = pytest.mark.gpu
POISON = np.uint32(0xFFC0DEAD)


class _Events:
    """Raw hipEvent_t handles from the HIP runtime torch uses."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipStreamWaitEvent.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint]

    def create(self):
        e = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def wait_host(self, e):
        assert self.hip.hipEventSynchronize(e) == 0

    def wait_stream(self, stream, e):
        assert self.hip.hipStreamWaitEvent(stream.cuda_stream, e, 0) == 0

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def _pinned_pool(n_pages, page_elems):
    pool = torch.empty((n_pages, page_elems), dtype=torch.float32, pin_memory=True)
    pool.view(torch.int32).fill_(int(POISON.view(np.int32)))
    return pool


def _is_poison(a):
    return np.all(a.view(np.uint32) == POISON)


def test_round_trip_permuted_poisoned_pool():
    w = wl.tp_rank_3584()
    res = api.prefill(api.to_device(w.inputs), w.interval)
    H = w.inputs.n_heads
    states = res.ckpt.reshape(-1, 128 * 128)                 # 112 pages
    n = states.shape[0]
    n_pages = 4 * n
    rng = np.random.default_rng(50)
    ids = rng.permutation(n_pages)[:n].astype(np.int32)
    pool = _pinned_pool(n_pages, 128 * 128)
    ev = _Events()
    done = ev.create()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    la.la_state_save_host(states, pool, torch.from_numpy(ids).cuda(), err, done_event=done)
    ev.wait_host(done)
    host = pool.numpy()
    ref = states.cpu().numpy()
    assert np.array_equal(host[ids].view(np.uint32), ref.view(np.uint32))
    untouched = np.setdiff1d(np.arange(n_pages), ids)
    assert _is_poison(host[untouched])
    # restore through the same table, plus a cold (-1) and an out-of-range item
    rids = np.concatenate([ids, [-1, n_pages + 3]]).astype(np.int32)
    back = torch.full((n + 2, 128 * 128), 7.0, device="cuda")
    la.la_state_restore_host(pool, torch.from_numpy(rids).cuda(), back, err, done_event=done)
    ev.wait_host(done)
    assert torch.equal(back[:n], states)
    assert torch.count_nonzero(back[n]) == 0                 # -1: zero state
    assert torch.all(back[n + 1] == 7.0)                     # out of range: untouched
    assert int(err.item()) == 1
    ev.destroy(done)
    print(f"[host tier] {n} pages round trip through a {n_pages}-page pinned pool, H={H}", flush=True)


def test_completion_event_orders_save_before_overwrite_and_restore():
    n, e = 64, 128 * 128
    states = torch.randn((n, e), device="cuda")
    before = states.cpu().numpy().copy()
    pool = _pinned_pool(n, e)
    ids = torch.arange(n, dtype=torch.int32, device="cuda")
    ev = _Events()
    saved = ev.create()
    side = torch.cuda.Stream()
    torch.cuda.current_stream().synchronize()
    with torch.cuda.stream(side):
        la.la_state_save_host(states, pool, ids, stream=side, done_event=saved)
    # overwrite the source only after the save's event, on another stream
    main = torch.cuda.current_stream()
    ev.wait_stream(main, saved)
    states.zero_()
    back = torch.empty_like(states)
    la.la_state_restore_host(pool, ids, back, stream=main)
    torch.cuda.synchronize()
    assert np.array_equal(pool.numpy().view(np.uint32), before.view(np.uint32))
    assert np.array_equal(back.cpu().numpy().view(np.uint32), before.view(np.uint32))
    assert torch.count_nonzero(states) == 0
    ev.destroy(saved)


def test_resume_through_host_tier_equals_recompute():
    w = wl.tp_rank_3584()
    x, C, N, H = w.inputs, w.interval, w.inputs.total_tokens, w.inputs.n_heads
    cold = api.prefill(api.to_device(x), C)
    n_ck = cold.n_ckpt_rows
    pool = _pinned_pool(n_ck * H, 128 * 128)
    perm = np.random.default_rng(51).permutation(n_ck * H).astype(np.int32)
    la.la_state_save_host(cold.ckpt, pool, torch.from_numpy(perm).cuda())
    B = la.strict_prefix_boundary(N, C, N)
    j = B // C - 1
    state = torch.full((1, H, 128, 128), float("nan"), device="cuda")
    la.la_state_restore_host(pool, torch.from_numpy(perm[j * H:(j + 1) * H].copy()).cuda(), state)
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], state, C)
    torch.cuda.synchronize()
    assert torch.equal(state, cold.ckpt[j:j + 1])
    assert torch.equal(r2.o, cold.o[B:]) and torch.equal(r2.final_state, cold.final_state)


def test_pageable_host_memory_is_refused():
    states = torch.zeros((4, 1024), device="cuda")
    pageable = torch.zeros((4, 1024), dtype=torch.float32)       # not pinned
    ids = torch.full((4,), -1, dtype=torch.int32, device="cuda")  # never touches the pool
    assert la.la_state_save_host(states, pageable, ids, check=False) == la.LA_ERR_INVALID_ARG
    assert la.la_state_restore_host(pageable, ids, states, check=False) == la.LA_ERR_INVALID_ARG
    torch.cuda.synchronize()
