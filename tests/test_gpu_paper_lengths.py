"""GPU parity over the paper's nine-length matrix (section 5.1; the lookups of
Table 4): N in {3583, 3584, 3585, 3587, 3588, 3589, 5375, 5376, 5377} at the
checkpoint interval C = 1,792, with 1 and 8 heads of dk = dv = 128 in bf16.

For each length: the cold prefill (checkpoints at every multiple of 1,792
up to N, the two-level fused scan), the strict-prefix boundary
B = C floor((N - 1) / C) (1,792 or 3,584 or 5,376), and the resume over the
suffix [B, N) from the cold run's own checkpoint: suffixes of 1,791 to 1,793
tokens, and of 1, 3, 4 and 5 tokens just past a checkpoint (3585, 3587,
3588, 3589, 5377).  Every output, checkpoint and final state is compared with
the oracle on every head, and the resume must reproduce the cold run's tail
and final state bit for bit (the paper's acceptance criterion of identical
continuations after a reload).
"""
import pytest
import torch

import oracle
from oracle.boundary import strict_prefix_boundary as brute_boundary
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, host, out_err, state_err

pytestmark = pytest.mark.gpu
TB = TOL[la.LA_BF16]
PAPER_LENGTHS = [3583, 3584, 3585, 3587, 3588, 3589, 5375, 5376, 5377]
C = 1792


@pytest.mark.parametrize("H", [1, 8])
@pytest.mark.parametrize("N", PAPER_LENGTHS)
def test_paper_length_cold_and_strict_prefix_resume(N, H):
    x = wl.random_inputs(1000 + N + H, [N], H, 128, 128, wl.BF16)
    assert la.la_prefill_form(la.make_shape(1, H, 128, 128, C)) == la.LA_FORM_FUSED_TWO_LEVEL
    res = api.prefill(api.to_device(x), C)
    B = la.strict_prefix_boundary(N, C, N)
    assert B == brute_boundary(N, C, N) == C * ((N - 1) // C)
    assert res.n_ckpt_rows == N // C
    j = B // C - 1
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], res.ckpt[j:j + 1].clone(), C)
    torch.cuda.synchronize()
    o_ref, s_ref, ck_ref = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=C)
    e = {"o": out_err(host(res.o), o_ref, [0, N]), "final": state_err(host(res.final_state), s_ref[None]),
         "ckpt": state_err(host(res.ckpt), ck_ref),
         "resume_o": out_err(host(r2.o), o_ref[B:], [0, N - B]),
         "resume_final": state_err(host(r2.final_state), s_ref[None])}
    if r2.n_ckpt_rows:   # the checkpoint at N when C divides it (5376)
        e["resume_ckpt"] = state_err(host(r2.ckpt), ck_ref[B // C:])
    print(f"[parity] paper length N={N} H={H} B={B} suffix {N - B}: "
          + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
    assert all(v <= TB for v in e.values()), e
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)
