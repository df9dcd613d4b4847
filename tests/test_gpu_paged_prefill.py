"""GPU tests of la_prefill_paged: checkpoints written straight into pool
pages, resume states read straight from pool pages, through the C ABI.

The reference for every case is the dense path the paged one replaces: a
prefill with ckpt_out followed by la_state_save_paged, and
la_state_restore_paged followed by la_prefill_resume.  Results must match
bit for bit (the scan's arithmetic is the same; only where states are read
and written changes), pages no id names must keep their poison, and ids
outside [-1, n_pages) must be skipped and counted once each.  Covered: the
one-TP-rank shape, a ragged varlen batch resumed from mixed boundaries
(cold included), the two-level scan (C = 1,024), fp32 with mid-chunk
checkpoints (C = 16), and fp32 at dk = 128 (the dk-split scan).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, host, out_err, state_err

pytestmark = pytest.mark.gpu
POISON = -7.25e30


def _pool(n_pages, e):
    return torch.full((n_pages, e), POISON, dtype=torch.float32, device="cuda")


def _ids(a):
    return torch.from_numpy(np.asarray(a, np.int32)).cuda()


def _dense_cold(xd, C):
    res = api.prefill(xd, C)
    torch.cuda.synchronize()
    return res


@pytest.mark.parametrize("lens,C,H,dk,dv,io", [
    ([3584], 256, 8, 128, 128, wl.BF16),                 # one TP rank
    ([1000, 3584, 257, 64, 1], 256, 4, 128, 128, wl.BF16),
    ([4096, 2500], 1024, 2, 128, 128, wl.BF16),          # two-level scan
    ([1000, 300], 16, 2, 64, 64, wl.F32),                # mid-chunk checkpoints
    ([700, 513], 128, 2, 128, 128, wl.F32),              # dk-split scan
])
def test_cold_checkpoints_to_pages_equal_dense_save(lens, C, H, dk, dv, io):
    x = wl.random_inputs(200 + C + dk, lens, H, dk, dv, io_dtype=io, gate_scale=0.01)
    xd = api.to_device(x)
    ref = _dense_cold(xd, C)
    n_rows = ref.n_ckpt_rows
    n_items = n_rows * H
    n_pages = 3 * n_items + 5
    perm = np.random.default_rng(7).permutation(n_pages)[:n_items].astype(np.int32)
    pool = _pool(n_pages, dk * dv)
    p = api.Prefill(xd, C, emit_ckpt=False)
    res = p.run_paged(pool, ckpt_page_ids=_ids(perm))
    torch.cuda.synchronize()
    assert torch.equal(res.o, ref.o) and torch.equal(res.final_state, ref.final_state)
    if n_items:
        assert torch.equal(pool[torch.from_numpy(perm).long().cuda()], ref.ckpt.reshape(n_items, -1))
    untouched = np.setdiff1d(np.arange(n_pages), perm)
    assert torch.all(pool[torch.from_numpy(untouched).long().cuda()] == POISON)
    print(f"[paged] cold lens={lens} C={C} io={io}: {n_items} checkpoint pages equal the dense save", flush=True)


@pytest.mark.parametrize("lens,C,H", [([3584], 256, 8), ([1000, 3584, 257, 4196, 64, 1], 256, 4),
                                      ([4096, 2500], 1024, 2)])
def test_resume_from_pages_equals_restore_then_resume(lens, C, H):
    x = wl.random_inputs(300 + C, lens, H, 128, 128, gate_scale=0.005)
    xd = api.to_device(x)
    cold = _dense_cold(xd, C)
    n_items = cold.n_ckpt_rows * H
    # every sequence from its strict-prefix checkpoint (0 = cold: page -1)
    starts = [la.strict_prefix_boundary(n, C, n) for n in lens]
    suf = [x.seq(i).tokens(starts[i], lens[i]) for i in range(len(lens))]
    cat = lambda f: np.concatenate([getattr(s, f) for s in suf])
    cu = np.concatenate([[0], np.cumsum([n - b for n, b in zip(lens, starts)])]).astype(np.int32)
    xs = api.to_device(wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"), cu, x.io_dtype))
    p = api.Prefill(xs, C, starts=starts, emit_ckpt=False)
    n_new = p.n_ckpt_rows * H
    # one pool: the cold run's pages, disjoint pages for the resume's checkpoints, spare poisoned pages
    n_pages = n_items + n_new + 7
    perm = np.random.default_rng(8).permutation(n_pages).astype(np.int32)
    save_ids, new_ids = perm[:n_items], perm[n_items:n_items + n_new]
    pool = _pool(n_pages, 128 * 128)
    la.la_state_save_paged(cold.ckpt.reshape(n_items, -1), pool, _ids(save_ids))
    state_ids = np.full((len(lens), H), -1, np.int32)
    for i, B in enumerate(starts):
        if B:
            row = int(cold.ckpt_offsets[i]) + B // C - 1
            state_ids[i] = save_ids[row * H:(row + 1) * H]
    # dense reference: restore the same pages (-1: zero state), then resume
    restored = torch.empty((len(lens), H, 128, 128), dtype=torch.float32, device="cuda")
    la.la_state_restore_paged(pool, _ids(state_ids.reshape(-1)), restored.reshape(len(lens) * H, -1))
    ref = api.prefill_resume(xs, starts, restored, C)
    res = p.run_paged(pool, ckpt_page_ids=_ids(new_ids), state_page_ids=_ids(state_ids.reshape(-1)))
    torch.cuda.synchronize()
    assert torch.equal(res.o, ref.o) and torch.equal(res.final_state, ref.final_state)
    if n_new:
        assert torch.equal(pool[torch.from_numpy(new_ids).long().cuda()], ref.ckpt.reshape(n_new, -1))
    assert torch.all(pool[torch.from_numpy(perm[n_items + n_new:]).long().cuda()] == POISON)
    # and the first sequence's resume agrees with the oracle's full recompute
    s0 = x.seq(0)
    o_ref, fin_ref, _ = oracle.gdr_prefill_seq(s0.q, s0.k, s0.v, s0.g, s0.beta, interval=C)
    B0 = starts[0]
    assert out_err(host(res.o[:cu[1]]), o_ref[B0:], [0, lens[0] - B0]) <= TOL[la.LA_BF16]
    assert state_err(host(res.final_state[:1]), fin_ref[None]) <= TOL[la.LA_BF16]
    print(f"[paged] resume lens={lens} C={C} from pages at {starts}: equal to restore + resume", flush=True)


def test_bad_page_ids_are_skipped_and_counted_once():
    lens, C, H = [1024, 600], 256, 4
    x = wl.random_inputs(400, lens, H, 128, 128, gate_scale=0.01)
    xd = api.to_device(x)
    ref = _dense_cold(xd, C)
    n_items = ref.n_ckpt_rows * H                       # (4 + 2) rows x 4 heads
    n_pages = n_items + 4
    ids = np.arange(n_items, dtype=np.int32)
    bad = {1: -1, 5: n_pages, 9: -3, 14: 1 << 30}       # -1 skips silently; the others are errors
    for i, v in bad.items():
        ids[i] = v
    pool = _pool(n_pages, 128 * 128)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    p = api.Prefill(xd, C, emit_ckpt=False)
    p.run_paged(pool, ckpt_page_ids=_ids(ids), err_count=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 3
    good = [i for i in range(n_items) if i not in bad]
    assert torch.equal(pool[good], ref.ckpt.reshape(n_items, -1)[good])
    assert torch.all(pool[[i for i in range(n_pages) if i not in good]] == POISON)
    # a resume whose starting page ids include -1 (zero state) and a bad id (zero state, counted)
    starts = [256, 512]
    sid = np.array([[0, 2, -1, 3], [n_pages + 7, 4, 6, 7]], np.int32)   # written pages only
    suf = [x.seq(i).tokens(starts[i], lens[i]) for i in range(2)]
    cat = lambda f: np.concatenate([getattr(s, f) for s in suf])
    cu = np.concatenate([[0], np.cumsum([n - b for n, b in zip(lens, starts)])]).astype(np.int32)
    xs = api.to_device(wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"), cu, x.io_dtype))
    err.zero_()
    r = api.Prefill(xs, C, starts=starts, emit_ckpt=False).run_paged(pool, state_page_ids=_ids(sid.reshape(-1)),
                                                                     err_count=err)
    st = torch.zeros((2, H, 128, 128), dtype=torch.float32, device="cuda")
    for i in range(2):
        for h in range(H):
            if 0 <= sid[i, h] < n_pages:
                st[i, h] = pool[sid[i, h]].reshape(128, 128)
    ref2 = api.prefill_resume(xs, starts, st, C)
    torch.cuda.synchronize()
    assert int(err.item()) == 1
    assert torch.equal(r.o, ref2.o) and torch.equal(r.final_state, ref2.final_state)
