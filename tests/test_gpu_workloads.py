"""GPU parity at full workload sizes, through the C ABI, in the launch
configuration the benchmark uses.

* Nine-length sweep (T = 512 .. 4608, 8 heads): cold prefill, save every
  checkpoint to a paged fp32 pool, restore at the strict-prefix boundary,
  resume over the suffix; every output, checkpoint and final state checked
  against the oracle.
* Long prefill (T = 32,768, 16 heads, C = 1,024, the two-level fused
  scan): every head's outputs, 32 checkpoints and final state against the
  oracle, and the resume from 31,744.
* Batched varlen (16 sequences, 8 heads, 4,096-page pool with a random
  permutation page table, cold / complete-hit / partial-hit restores):
  every head of every sequence, for the cold call (outputs, checkpoints,
  final states) and for the resume (restored pages, outputs, checkpoints,
  final states).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.boundary import strict_prefix_boundary as brute_boundary
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, host, out_err, slice_err, state_err

pytestmark = pytest.mark.gpu
TB = TOL[la.LA_BF16]


def _poisoned(shape):
    return torch.from_numpy(np.full(shape, 0xFFC0DEAD, np.uint32).view(np.float32)).cuda()


@pytest.mark.parametrize("i", range(9))
def test_nine_length_sweep(i):
    w = wl.nine_length_sweep()[i]
    x, C, N, H = w.inputs, w.interval, w.inputs.total_tokens, w.inputs.n_heads
    xd = api.to_device(x)
    res = api.prefill(xd, C)
    n_ck = res.n_ckpt_rows
    assert n_ck == N // C
    pool = _poisoned((w.pool_pages, 128 * 128))
    ids = torch.arange(n_ck * H, dtype=torch.int32, device="cuda")
    la.la_state_save_paged(res.ckpt, pool, ids)
    B = la.strict_prefix_boundary(N, C, N)
    assert B == brute_boundary(N, C, N) == N - 256
    j = B // C - 1
    state = _poisoned((1, H, 128, 128))
    la.la_state_restore_paged(pool, ids[j * H:(j + 1) * H].contiguous(), state)
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], state, C)
    torch.cuda.synchronize()
    o_ref, s_ref, ck_ref = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=C)
    e = {"o": out_err(host(res.o), o_ref, [0, N]), "final": state_err(host(res.final_state), s_ref[None]),
         "ckpt": state_err(host(res.ckpt), ck_ref),
         "resume_o": out_err(host(r2.o), o_ref[B:], [0, N - B]),
         "resume_final": state_err(host(r2.final_state), s_ref[None])}
    print(f"[parity] sweep T={N}: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
    assert all(v <= TB for v in e.values()), e
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_long_prefill_all_heads():
    w = wl.long_prefill()
    x, C, N, H = w.inputs, w.interval, w.inputs.total_tokens, w.inputs.n_heads
    assert la.la_prefill_form(la.make_shape(1, H, 128, 128, C)) == la.LA_FORM_FUSED_TWO_LEVEL
    xd = api.to_device(x)
    res = api.prefill(xd, C)
    B = la.strict_prefix_boundary(N, C, N)
    assert B == 31744
    j = B // C - 1
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], res.ckpt[j:j + 1].clone(), C)
    torch.cuda.synchronize()
    o_ref, s_ref, ck_ref = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=C)
    e = {"o": out_err(host(res.o), o_ref, [0, N]),
         "final": state_err(host(res.final_state), s_ref[None]),
         "ckpt": state_err(host(res.ckpt), ck_ref),
         "resume_o": out_err(host(r2.o), o_ref[B:], [0, N - B]),
         "resume_final": state_err(host(r2.final_state), s_ref[None])}
    print(f"[parity] long T={N} all {H} heads: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
    assert all(v <= TB for v in e.values()), e
    assert res.ckpt.shape[0] == N // C
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_batched_varlen_paged_restore_all_heads():
    w = wl.batched_varlen()
    x, C, H = w.inputs, w.interval, w.inputs.n_heads
    cu = x.cu_seqlens
    lens = np.diff(cu).tolist()
    assert la.la_prefill_form(la.make_shape(len(lens), H, 128, 128, C)) == la.LA_FORM_FUSED_SCAN
    xd = api.to_device(x)
    cold = api.prefill(xd, C)
    # the cold call, every head of every sequence
    o_ref, fin_ref, cks_ref = oracle.gdr_prefill(x, interval=C)
    cks = [c for c in cks_ref if c is not None]
    e_cold = {"o": out_err(host(cold.o), o_ref, cu), "final": state_err(host(cold.final_state), fin_ref),
              "ckpt": state_err(host(cold.ckpt), np.concatenate(cks, axis=0))}
    print("[parity] varlen cold, all heads: " + " ".join(f"{k} {v:.2e}" for k, v in e_cold.items()), flush=True)
    assert all(v <= TB for v in e_cold.values()), e_cold
    # save every checkpoint of every sequence into the permuted pool
    pool = _poisoned((w.pool_pages, 128 * 128))
    save_ids = np.full(cold.n_ckpt_rows * H, -1, np.int32)
    for i, n in enumerate(lens):
        for jj in range(n // C):
            for hh in range(H):
                save_ids[(int(cold.ckpt_offsets[i]) + jj) * H + hh] = w.page_perm[wl.page_slot(i, jj, hh, H)]
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    la.la_state_save_paged(cold.ckpt, pool, torch.from_numpy(save_ids).cuda(), err)
    # lookup: strict prefix within the available (cached) prefix of each sequence
    starts, restore_ids = [], []
    for i, (n, avail) in enumerate(zip(lens, w.available)):
        B = la.strict_prefix_boundary(n, C, avail)
        assert B == brute_boundary(n, C, avail)
        starts.append(B)
        for hh in range(H):
            restore_ids.append(-1 if B == 0 else int(w.page_perm[wl.page_slot(i, B // C - 1, hh, H)]))
    assert any(m == "partial" for m in w.modes) or any(m == "cold" for m in w.modes)
    states = _poisoned((len(lens), H, 128, 128))
    la.la_state_restore_paged(pool, torch.from_numpy(np.asarray(restore_ids, np.int32)).cuda(), states, err)
    # the suffixes, packed
    suf = [x.seq(i).tokens(starts[i], lens[i]) for i in range(len(lens))]
    cat = lambda f: np.concatenate([getattr(s, f) for s in suf])
    xs = wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"),
                   np.concatenate([[0], np.cumsum([n - b for n, b in zip(lens, starts)])]).astype(np.int32),
                   x.io_dtype)
    res = api.prefill_resume(api.to_device(xs), starts, states, C)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    worst = {"o": 0.0, "final": 0.0, "ckpt": 0.0, "restored": 0.0}
    for i, n in enumerate(lens):
        B = starts[i]
        a, b = int(xs.cu_seqlens[i]), int(xs.cu_seqlens[i + 1])
        c0 = int(cu[i])
        worst["o"] = max(worst["o"], out_err(host(res.o[a:b]), o_ref[c0 + B:c0 + n], [0, n - B]))
        worst["final"] = max(worst["final"], state_err(host(res.final_state[i:i + 1]), fin_ref[i:i + 1]))
        ck_i = cks_ref[i]
        if B > 0:   # the restored page is the oracle's state for exactly [0, B)
            worst["restored"] = max(worst["restored"], state_err(host(states[i:i + 1]), ck_i[B // C - 1][None]))
        else:
            assert torch.count_nonzero(states[i]) == 0
        off = int(res.ckpt_offsets[i])
        nck = (n // C) - (B // C)
        if nck:
            worst["ckpt"] = max(worst["ckpt"], state_err(host(res.ckpt[off:off + nck]), ck_i[B // C:]))
        # resume equals recompute, bit for bit
        assert torch.equal(res.o[a:b], cold.o[c0 + B:c0 + n]), i
        assert torch.equal(res.final_state[i], cold.final_state[i]), i
    print(f"[parity] varlen 16 seqs resume, all heads, modes {w.modes}: "
          + " ".join(f"{k} {v:.2e}" for k, v in worst.items()), flush=True)
    assert all(v <= TB for v in worst.values()), worst
