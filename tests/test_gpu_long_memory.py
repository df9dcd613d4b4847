"""GPU parity on long-memory inputs, through the C ABI.

With the specified gate distribution (g = -softplus(N(0, 1)), mean -0.81 per
token) the state decays by about e^-52 per 64-token chunk: anything older than
a chunk falls below fp32 resolution, so those workloads cannot detect an error
in the state carried from chunk to chunk, or from segment to segment in the
two-level scan.  Here the log-decay is scaled down (gate_scale 0.01 .. 0, down
to the ungated delta rule), so the state entering a chunk dominates its output
and every checkpoint, and the tests cover:

* the one-TP-rank shape (T = 3,584, 8 heads, C = 256), every head, cold and
  resumed at two boundaries, bitwise resume = recompute;
* every segment length the two-level scan takes (C = 100, 192, 1,024, 1,792:
  2, 3, 16 and 14 chunks per segment) on a ragged length;
* a ragged varlen batch resumed from mixed boundaries (cold included);
* T = 32,768 with 16 heads, every head checked against the oracle;
* fp32 with mid-chunk checkpoints (C = 16).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.boundary import strict_prefix_boundary as brute_boundary
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, compare, host, oracle_run, out_err, state_err

pytestmark = pytest.mark.gpu
TB = TOL[la.LA_BF16]


def _resume_from_own_checkpoint(x, res, C, B):
    """Resume over [B, N) from the cold run's checkpoint at B (single sequence)."""
    N = x.total_tokens
    row = B // C - 1
    r2 = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], res.ckpt[row:row + 1].clone(), C)
    torch.cuda.synchronize()
    return r2


@pytest.mark.parametrize("gate_scale", [0.01, 0.0])
def test_tp_rank_shape_long_memory(gate_scale):
    x = wl.random_inputs(31, [3584], 8, 128, 128, gate_scale=gate_scale)
    C, N = 256, 3584
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TB, f"long memory gate_scale={gate_scale} T=3584 cold")
    o_ref, fin_ref, ck_ref = ref
    for B in (la.strict_prefix_boundary(N, C, N), 1792):
        r2 = _resume_from_own_checkpoint(x, res, C, B)
        e = {"o": out_err(host(r2.o), o_ref[B:], [0, N - B]), "final": state_err(host(r2.final_state), fin_ref),
             "ckpt": state_err(host(r2.ckpt), ck_ref[B // C:])}
        print(f"[parity] long memory gate_scale={gate_scale} resume at {B}: "
              + " ".join(f"{k} {v:.2e}" for k, v in e.items()), flush=True)
        assert all(v <= TB for v in e.values()), e
        assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)
        assert torch.equal(r2.ckpt, res.ckpt[B // C:])


@pytest.mark.parametrize("C", [100, 192, 1024, 1792])
def test_segment_lengths_long_memory(C):
    N = 4000     # a multiple of neither 64 nor C: ragged last chunk and segment
    x = wl.random_inputs(32 + C, [N], 2, 128, 128, gate_scale=0.01)
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TB, f"long memory C={C} T={N} cold")
    B = la.strict_prefix_boundary(N, C, N)
    assert B == brute_boundary(N, C, N) and B > 0
    r2 = _resume_from_own_checkpoint(x, res, C, B)
    o_ref, fin_ref, _ = ref
    assert out_err(host(r2.o), o_ref[B:], [0, N - B]) <= TB
    assert state_err(host(r2.final_state), fin_ref) <= TB
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_varlen_mixed_resume_long_memory():
    lens = [1000, 3584, 257, 4196, 64, 1]
    C = 256
    x = wl.random_inputs(33, lens, 4, 128, 128, gate_scale=0.005)
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TB, "long memory varlen cold")
    o_ref, fin_ref, ck_ref = ref
    # resume every sequence from its own strict-prefix checkpoint (0 = cold)
    starts = [la.strict_prefix_boundary(n, C, n) for n in lens]
    states = torch.zeros((len(lens), 4, 128, 128), dtype=torch.float32, device="cuda")
    for i, B in enumerate(starts):
        if B:
            states[i] = res.ckpt[int(res.ckpt_offsets[i]) + B // C - 1]
    suf = [x.seq(i).tokens(starts[i], lens[i]) for i in range(len(lens))]
    cat = lambda f: np.concatenate([getattr(s, f) for s in suf])
    cu = np.concatenate([[0], np.cumsum([n - b for n, b in zip(lens, starts)])]).astype(np.int32)
    xs = wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"), cu, x.io_dtype)
    r2 = api.prefill_resume(api.to_device(xs), starts, states, C)
    torch.cuda.synchronize()
    worst = {"o": 0.0, "final": 0.0}
    for i, (n, B) in enumerate(zip(lens, starts)):
        a, b = int(x.cu_seqlens[i]), int(x.cu_seqlens[i + 1])
        worst["o"] = max(worst["o"], out_err(host(r2.o[cu[i]:cu[i + 1]]), o_ref[a + B:b], [0, n - B]))
        worst["final"] = max(worst["final"], state_err(host(r2.final_state[i:i + 1]), fin_ref[i:i + 1]))
        # batch invariance and resume = recompute, bit for bit
        assert torch.equal(r2.o[cu[i]:cu[i + 1]], res.o[a + B:b])
        assert torch.equal(r2.final_state[i], res.final_state[i])
    print(f"[parity] long memory varlen resume {starts}: " + " ".join(f"{k} {v:.2e}" for k, v in worst.items()),
          flush=True)
    assert all(v <= TB for v in worst.values()), worst


def test_long_prefill_long_memory_all_heads():
    N, H, C = 32768, 16, 1024
    x = wl.random_inputs(34, [N], H, 128, 128, gate_scale=0.001)
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    B = la.strict_prefix_boundary(N, C, N)
    r2 = _resume_from_own_checkpoint(x, res, C, B)
    o_ref, s_ref, ck_ref = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=C)
    e = {"o": out_err(host(res.o), o_ref, [0, N]),
         "final": state_err(host(res.final_state), s_ref[None]),
         "ckpt": state_err(host(res.ckpt), ck_ref),
         "resume_o": out_err(host(r2.o), o_ref[B:], [0, N - B])}
    print(f"[parity] long memory T={N} all {H} heads: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()),
          flush=True)
    assert all(v <= TB for v in e.values()), e
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_fp32_mid_chunk_checkpoints_long_memory():
    x = wl.random_inputs(35, [1000], 2, 64, 64, io_dtype=wl.F32, gate_scale=0.01)
    C = 16
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_F32], "long memory fp32 C=16 T=1000")
    B = la.strict_prefix_boundary(1000, C, 1000)
    r2 = _resume_from_own_checkpoint(x, res, C, B)
    o_ref, fin_ref, _ = ref
    assert out_err(host(r2.o), o_ref[B:], [0, 1000 - B]) <= TOL[la.LA_F32]
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)
