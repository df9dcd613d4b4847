"""The save-before-reuse contract (section 3.1: a restore must wait for the
save it depends on) under a delayed save, through the C ABI, for the device
pool and for the pinned host tier.

Stream A spins on the GPU before it saves 256 state pages into a poisoned
pool through a permuted page table, so the save lands tens of milliseconds
after it was issued; stream B waits on A's completion event and restores
the pages into a poisoned buffer.  The restored pages equal the saved states
bit for bit (a restore that ran early would read poison), and every page the
table does not name still holds the poison.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_15030_amd import linattn as la

pytestmark = pytest.mark.gpu
POISON = np.uint32(0xFFC0DEAD)
SPIN_CYCLES = 50_000_000


class _Events:
    """Raw hipEvent_t handles from the HIP runtime torch uses."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipStreamWaitEvent.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint]

    def create(self):
        e = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def record(self, e, stream):
        assert self.hip.hipEventRecord(e, stream.cuda_stream) == 0

    def wait_stream(self, stream, e):
        assert self.hip.hipStreamWaitEvent(stream.cuda_stream, e, 0) == 0

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def _poison(t):
    t.view(torch.int32).fill_(int(POISON.view(np.int32)))
    return t


@pytest.mark.parametrize("tier", ["device", "host"])
def test_restore_waits_for_a_delayed_save(tier):
    n, n_pages, e = 256, 640, 128 * 128
    g = torch.Generator(device="cuda").manual_seed(70)
    states = torch.randn((n, e), device="cuda", generator=g)
    ref = states.cpu().numpy().view(np.uint32).copy()
    if tier == "device":
        pool = _poison(torch.empty((n_pages, e), dtype=torch.float32, device="cuda"))
    else:
        pool = _poison(torch.empty((n_pages, e), dtype=torch.float32, pin_memory=True))
    ids_np = np.random.default_rng(71).permutation(n_pages)[:n].astype(np.int32)
    ids = torch.from_numpy(ids_np).cuda()
    back = _poison(torch.empty((n, e), dtype=torch.float32, device="cuda"))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ev = _Events()
    saved = ev.create()
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    print(f"[delayed save] tier={tier}: {n} pages, spin {SPIN_CYCLES} cycles on stream A", flush=True)
    with torch.cuda.stream(a):
        torch.cuda._sleep(SPIN_CYCLES)
        if tier == "device":
            la.la_state_save_paged(states, pool, ids, err, stream=a)
            ev.record(saved, a)
        else:
            la.la_state_save_host(states, pool, ids, err, stream=a, done_event=saved)
    ev.wait_stream(b, saved)
    with torch.cuda.stream(b):
        if tier == "device":
            la.la_state_restore_paged(pool, ids, back, err, stream=b)
        else:
            la.la_state_restore_host(pool, ids, back, err, stream=b)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert np.array_equal(back.cpu().numpy().view(np.uint32), ref)
    host_pool = pool.cpu().numpy().view(np.uint32)
    assert np.array_equal(host_pool[ids_np], ref)
    untouched = np.setdiff1d(np.arange(n_pages), ids_np)
    assert np.all(host_pool[untouched] == POISON)
    ev.destroy(saved)
