"""GPU tests of the joint attention-KV / recurrent-state restore, through the C ABI.

* la_hybrid_restore against the oracle's plain-loop hybrid_restore, bit for
  bit, on a ragged batch (cold, block-aligned partial and long boundaries)
  with -1 and out-of-range ids on both kinds of entries and poisoned
  destinations;
* the reload path of the one-TP-rank workload: a cold prefill writes its
  checkpoint pages into a state pool while the attention layers' KV bytes
  (opaque, 8,268 B per token per rank, the figure the paper's transfer
  counts fix) sit in a block pool; la_hybrid_boundary picks B, one
  la_hybrid_restore brings back the KV blocks of [0, B) and the states at B,
  and the resume reproduces the cold run's tail bit for bit; both when every
  prefix is cached and when the KV cache is shorter than the checkpoints;
* the same restore from pinned host-memory pools (the CPU tier);
* a pageable pool is refused before any launch.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

pytestmark = pytest.mark.gpu
KV_TOKEN_BYTES = 8268          # attention entries per token per rank (section 5.2 counts)
BT = 16                        # KV block tokens
BLOCK = KV_TOKEN_BYTES * BT    # 132,288 bytes
POISON8 = 0xA5


def _rand_bytes(rng, n, nbytes):
    return torch.from_numpy(rng.integers(0, 256, size=(n, nbytes), dtype=np.uint8))


def _ids(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def _setup(rng, bounds, n_pool, n_cache, H, page_elems, n_state_pages):
    max_blocks = max(1, max(b // BT for b in bounds))
    kv_pool = _rand_bytes(rng, n_pool, BLOCK)
    src = np.full((len(bounds), max_blocks), -1, np.int32)
    dst = np.full((len(bounds), max_blocks), -1, np.int32)
    free = rng.permutation(n_cache)
    k = 0
    for i, b in enumerate(bounds):
        nb = b // BT
        src[i, :nb] = rng.integers(0, n_pool, nb)
        dst[i, :nb] = free[k:k + nb]
        k += nb
    state_pool = torch.from_numpy(rng.standard_normal((n_state_pages, page_elems)).astype(np.float32))
    state_ids = rng.integers(0, n_state_pages, len(bounds) * H).astype(np.int32)
    return kv_pool, src, dst, max_blocks, state_pool, state_ids


def test_hybrid_restore_matches_oracle():
    rng = np.random.default_rng(70)
    H, page_elems = 4, 128 * 128
    bounds = [0, 256, 3328, 592, 1024]
    kv_pool, src, dst, max_blocks, state_pool, state_ids = _setup(rng, bounds, 300, 400, H, page_elems, 9)
    # -1 and out-of-range ids on both kinds of entries
    src[1, 3], dst[2, 10], src[2, 11], dst[4, 0] = -1, -1, 300, 400 + 5
    state_ids[[2, 7, 13]] = [-1, 9, -4]
    cache = torch.full((400, BLOCK), POISON8, dtype=torch.uint8)
    states = torch.full((len(bounds) * H, page_elems), 3.5, dtype=torch.float32)
    ref_cache, ref_states, ref_err = oracle.hybrid_restore(kv_pool.numpy(), cache.numpy(), src, dst, bounds, BT,
                                                           state_pool.numpy(), state_ids, states.numpy())
    d_cache, d_states = cache.cuda(), states.cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = la.make_kv_blocks(kv_pool.cuda(), d_cache, _ids(src), _ids(dst), BT)
    bh = np.asarray(bounds, np.int64)
    d_pool = state_pool.cuda()
    la.la_hybrid_restore(kv, torch.from_numpy(bh).cuda(), bh, d_pool, _ids(state_ids), d_states, H, err)
    torch.cuda.synchronize()
    assert int(err.item()) == ref_err == 4
    assert np.array_equal(d_cache.cpu().numpy(), ref_cache)
    assert np.array_equal(d_states.cpu().numpy().view(np.uint32), ref_states.view(np.uint32))
    print(f"[hybrid] {sum(b // BT for b in bounds)} KV blocks of {BLOCK} B + {len(bounds) * H} state pages "
          f"equal the oracle; {ref_err} bad ids counted", flush=True)


def _reload(kv_cached, host_pools=False):
    """Cold prefill of the one-TP-rank workload (checkpoints to a state pool;
    the attention KV of every block of the prompt in a block pool), then the
    joint boundary, one joint restore, and the resume."""
    w = wl.tp_rank_3584()
    x, C, N, H = w.inputs, w.interval, w.inputs.total_tokens, w.inputs.n_heads
    rng = np.random.default_rng(71)
    xd = api.to_device(x)
    cold = api.Prefill(xd, C, emit_ckpt=False)
    n_items = cold.n_ckpt_rows * H
    ck_ids = rng.permutation(n_items + 5)[:n_items].astype(np.int32)
    st_pool = torch.full((n_items + 5, 128 * 128), float("nan"), dtype=torch.float32, device="cuda")
    res = cold.run_paged(st_pool, ckpt_page_ids=_ids(ck_ids))
    cold_o, cold_final = res.o.clone(), res.final_state.clone()
    n_blocks = N // BT
    kv_pool = _rand_bytes(rng, n_blocks + 7, BLOCK)
    kv_ids = rng.permutation(n_blocks + 7)[:n_blocks].astype(np.int32)    # pool block of prompt block j
    B, nb = la.la_hybrid_boundary(N, C, BT, kv_cached, N)
    assert (B, nb) == oracle.hybrid_boundary(N, C, BT, kv_cached, N)
    n_cache = nb + 11
    dst = rng.permutation(n_cache)[:max(nb, 1)].astype(np.int32)
    src = kv_ids[:max(nb, 1)].copy()
    if nb == 0:
        src[:], dst[:] = -1, -1
    cache = torch.full((n_cache, BLOCK), POISON8, dtype=torch.uint8, device="cuda")
    states = torch.full((H, 128 * 128), float("nan"), dtype=torch.float32, device="cuda")
    row = B // C - 1
    state_ids = ck_ids[row * H:(row + 1) * H] if B else np.full(H, -1, np.int32)
    if host_pools:
        kv_src = kv_pool.pin_memory()
        st_src = torch.empty(st_pool.shape, dtype=torch.float32, pin_memory=True)
        st_src.copy_(st_pool)
    else:
        kv_src, st_src = kv_pool.cuda(), st_pool
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = la.make_kv_blocks(kv_src, cache, _ids(src[None]), _ids(dst[None]), BT)
    la.la_hybrid_restore(kv, torch.tensor([B], dtype=torch.int64, device="cuda"), [B], st_src, _ids(state_ids),
                         states, H, err)
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], states.reshape(1, H, 128, 128), C)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    # the cache holds exactly the prompt's blocks [0, B); every other cache block keeps its poison
    c = cache.cpu().numpy()
    for j in range(nb):
        assert np.array_equal(c[dst[j]], kv_pool[kv_ids[j]].numpy())
    assert np.all(c[np.setdiff1d(np.arange(n_cache), dst[:nb])] == POISON8)
    # and the recurrent state is the cold run's checkpoint at the same B: the resume equals the cold tail
    assert torch.equal(r2.o, cold_o[B:]) and torch.equal(r2.final_state, cold_final)
    return B, nb


def test_joint_reload_of_the_tp_rank_prompt():
    assert _reload(3584) == (3328, 208)             # everything cached: the strict prefix
    assert _reload(1000) == (768, 48)               # the KV cache is the shorter prefix


def test_joint_reload_from_pinned_host_pools():
    assert _reload(3584, host_pools=True) == (3328, 208)


def test_pageable_pool_is_refused():
    kv_pool = torch.zeros((4, BLOCK), dtype=torch.uint8)                 # pageable host memory
    cache = torch.zeros((4, BLOCK), dtype=torch.uint8, device="cuda")
    kv = la.make_kv_blocks(kv_pool, cache, _ids([[0]]), _ids([[0]]), BT)
    st = la.la_hybrid_restore(kv, torch.tensor([BT], dtype=torch.int64, device="cuda"), [BT], None, None, None, 0,
                              check=False)
    assert st == la.LA_ERR_INVALID_ARG
    torch.cuda.synchronize()
