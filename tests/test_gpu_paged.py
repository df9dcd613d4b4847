"""GPU paged state save/restore against the NumPy paging oracle: bit-exact,
with poisoned destinations (a restore must overwrite exactly the addressed
pages, and a save must leave untouched pool pages as they were), -1 ids,
out-of-range ids counted on the device, and addressing checked against the
oracle's checkpoint at that position (byte equality alone does not prove
the right state was addressed)."""
import numpy as np
import pytest
import torch

from oracle.paging import paged_restore, paged_save
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, host, oracle_run, state_err

pytestmark = pytest.mark.gpu

POISON = np.uint32(0xFFC0DEAD)    # a NaN bit pattern


def _poisoned(shape):
    return np.full(shape, POISON, np.uint32).view(np.float32)


def _bits(t):
    return t.detach().cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("page_elems", [64 * 64, 128 * 128, 4, 12])
def test_save_restore_bit_exact_under_permutation(page_elems):
    rng = np.random.default_rng(page_elems)
    n_items, n_pages = 37, 64
    states = rng.standard_normal((n_items, page_elems)).astype(np.float32)
    ids = rng.permutation(n_pages)[:n_items].astype(np.int32)
    ids[3] = -1
    pool0 = _poisoned((n_pages, page_elems))
    pool_ref, e_ref = paged_save(states, pool0, ids)
    pool = torch.from_numpy(pool0.copy()).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    la.la_state_save_paged(torch.from_numpy(states).cuda(), pool, torch.from_numpy(ids).cuda(), err)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(pool), pool_ref.view(np.uint32)) and int(err) == e_ref == 0
    dest0 = _poisoned((n_items, page_elems))
    dest_ref, e2 = paged_restore(pool_ref, ids, dest0)
    dest = torch.from_numpy(dest0.copy()).cuda()
    la.la_state_restore_paged(pool, torch.from_numpy(ids).cuda(), dest, err)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(dest), dest_ref.view(np.uint32)) and int(err) == e2 == 0
    assert np.all(_bits(dest)[3] == 0)                          # -1 restores the zero state


def test_out_of_range_ids_are_counted_and_skipped():
    n_pages, pe = 8, 128
    states = np.arange(4 * pe, dtype=np.float32).reshape(4, pe)
    ids = np.array([1, 8, -2, 5], np.int32)
    pool0 = _poisoned((n_pages, pe))
    pool = torch.from_numpy(pool0.copy()).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    la.la_state_save_paged(torch.from_numpy(states).cuda(), pool, torch.from_numpy(ids).cuda(), err)
    torch.cuda.synchronize()
    ref, e = paged_save(states, pool0, ids)
    assert int(err) == e == 2 and np.array_equal(_bits(pool), ref.view(np.uint32))
    dest0 = _poisoned((4, pe))
    dest = torch.from_numpy(dest0.copy()).cuda()
    err.zero_()
    la.la_state_restore_paged(pool, torch.from_numpy(ids).cuda(), dest, err)
    torch.cuda.synchronize()
    dref, e = paged_restore(ref, ids, dest0)
    assert int(err) == e == 2 and np.array_equal(_bits(dest), dref.view(np.uint32))
    assert np.all(_bits(dest)[1] == POISON)                    # untouched destination


def test_checkpoint_pages_address_the_right_prefix():
    """Save every checkpoint of a run into a permuted pool, restore the one the
    strict-prefix rule selects, and compare it with the oracle's state for
    exactly that prefix; then resume from it."""
    x = wl.random_inputs(601, [1100], 4, 128, 128, wl.BF16)
    C, N, H = 256, 1100, 4
    xd = api.to_device(x)
    res = api.prefill(xd, C)
    n_ck = res.n_ckpt_rows                                    # 4 checkpoints: 256..1024
    pool = torch.from_numpy(_poisoned((64, 128 * 128))).cuda()
    perm = np.random.default_rng(3).permutation(64)[:n_ck * H].astype(np.int32)
    la.la_state_save_paged(res.ckpt, pool, torch.from_numpy(perm).cuda())
    B = la.strict_prefix_boundary(N, C, N)
    j = B // C - 1
    ids = perm[j * H:(j + 1) * H].copy()
    restored = torch.from_numpy(_poisoned((1, H, 128, 128))).cuda()
    la.la_state_restore_paged(pool, torch.from_numpy(ids).cuda(), restored)
    torch.cuda.synchronize()
    assert torch.equal(restored[0], res.ckpt[j])
    _, _, ck_ref = oracle_run(x.tokens(0, B), interval=C)
    assert state_err(host(restored), ck_ref[j:j + 1]) <= TOL[la.LA_BF16]
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], restored, C)
    torch.cuda.synchronize()
    assert torch.equal(r2.o, res.o[B:])
