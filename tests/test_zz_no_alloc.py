"""The no-alloc prefill entry point (la_prefill_paged_noalloc, whose
workspace is the library's static device array) against la_prefill_paged
with a caller workspace, on the same inputs: two calls in a row, the
second with a smaller input, each compared bit for bit (outputs, final
states and every pool page).  A call too large for the static array is
refused before any launch."""
import numpy as np
import pytest
import torch

from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _both(x, C, starts, n_pages, seed):
    """The same paged call through both entry points, each on its own copy of
    a seeded pool; returns (regular, no-alloc) as (o, final, pool)."""
    H, dk, dv = x.n_heads, x.dk, x.dv
    rng = np.random.default_rng(seed)
    pool0 = torch.from_numpy(rng.standard_normal((n_pages, dk * dv)).astype(np.float32) * 0.05).cuda()
    perm = rng.permutation(n_pages).astype(np.int32)
    n = len(starts)
    st_ids = np.full(n * H, -1, np.int32)
    for i, b in enumerate(starts):
        if b > 0:
            st_ids[i * H:(i + 1) * H] = perm[i * H:(i + 1) * H]
    out = []
    for noalloc in (False, True):
        pf = api.Prefill(api.to_device(x), C, starts=starts, emit_ckpt=False)
        ck_ids = perm[n * H:n * H + pf.n_ckpt_rows * H]
        assert len(ck_ids) == pf.n_ckpt_rows * H, "pool too small for the checkpoints"
        pool = pool0.clone()
        ck = torch.from_numpy(np.ascontiguousarray(ck_ids)).cuda()
        st = torch.from_numpy(st_ids).cuda()
        pages = la.make_pages(pool, ck, st)
        xd = pf.x
        args = (pf.shape, pages, xd.q, xd.k, xd.v, xd.g, xd.beta, xd.cu_dev, xd.cu_host, pf.start_dev, pf.starts,
                pf.o, pf.final, pf.ckpt_off_dev, pf.ckpt_offsets)
        if noalloc:
            la.la_prefill_paged_noalloc(*args)
        else:
            la.la_prefill_paged(*args, pf.workspace)
        torch.cuda.synchronize()
        out.append((pf.o.clone(), pf.final.clone(), pool))
    return out


def test_noalloc_matches_workspace_call_twice():
    C = 256
    # first call: three sequences (cold, resumed at 512, cold), 8 heads
    x1 = wl.random_inputs(900, [700, 1300 - 512, 256], 8, 128, 128, wl.BF16)
    print("[no-alloc] call 1: 3 seqs x 8 heads, d=128", flush=True)
    (o_a, f_a, p_a), (o_b, f_b, p_b) = _both(x1, C, [0, 512, 0], 96, 901)
    assert torch.equal(o_a, o_b) and torch.equal(f_a, f_b) and torch.equal(p_a, p_b)
    # second call, smaller: one sequence resumed at 256, 4 heads
    x2 = wl.random_inputs(902, [300], 4, 128, 128, wl.BF16)
    print("[no-alloc] call 2: 1 seq x 4 heads, d=128", flush=True)
    (o_a, f_a, p_a), (o_b, f_b, p_b) = _both(x2, C, [256], 16, 903)
    assert torch.equal(o_a, o_b) and torch.equal(f_a, f_b) and torch.equal(p_a, p_b)


def test_noalloc_refuses_a_call_beyond_the_static_workspace():
    # 2M tokens x 8 heads needs far more than 64 MiB of workspace; refused on
    # the host before any pointer is touched
    shape = la.make_shape(1, 8, 128, 128, 256)
    cu = np.array([0, 2_000_000], np.int32)
    pool = torch.empty((1, 128 * 128), device="cuda")
    pages = la.make_pages(pool)
    st = la.la_prefill_paged_noalloc(shape, pages, None, None, None, None, None, None, cu, None, None, None, None,
                                     None, None, check=False)
    assert st == la.LA_ERR_WORKSPACE, la.status_string(st)
    assert "static scratch" in la.last_error_message()
