"""GPU parity of decode continuation (one token per sequence per call) against
the fp64 oracle's token loop, through the C ABI.

Decoding T tokens from a state is the recurrence over those tokens from that
state, which the oracle computes directly (its token loop with state_in).
Covered: 64- and 256-token continuations after a strict-prefix resume of the
one-TP-rank workload (the continuation lengths the paper compares), the
continuation equality the paper checks (cold and reloaded runs continue bit
for bit identically), a 16-sequence batch with both recurrence variants and a
scale, every head-dimension pair, fp32 inputs, and long-memory tokens.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, host, slice_err

pytestmark = pytest.mark.gpu


def _decode_gpu(shape, tok: wl.Inputs, n_seqs, T, state):
    """Run T decode steps; tok holds n_seqs sequences of T tokens (packed).
    Returns o [n_seqs, T, H, dv] and leaves the final state in ``state``."""
    xd = api.to_device(tok)
    H, dv = tok.n_heads, tok.dv
    o = torch.empty((n_seqs, T, H, dv), dtype=xd.q.dtype, device="cuda")
    step_o = torch.empty((n_seqs, H, dv), dtype=xd.q.dtype, device="cuda")
    base = torch.arange(n_seqs, device="cuda") * T
    for t in range(T):
        idx = base + t
        la.la_decode_step(shape, xd.q[idx].contiguous(), xd.k[idx].contiguous(), xd.v[idx].contiguous(),
                          xd.g[idx].contiguous(), xd.beta[idx].contiguous(), state, step_o)
        o[:, t] = step_o
    torch.cuda.synchronize()
    return o


def _decode_oracle(tok: wl.Inputs, n_seqs, T, states, variant=0, scale=1.0):
    outs, finals = [], []
    for i in range(n_seqs):
        s = tok.seq(i)
        o, fin, _ = oracle.gdr_prefill_seq(s.q, s.k, s.v, s.g, s.beta, state_in=states[i], variant=variant,
                                           scale=scale)
        outs.append(o)
        finals.append(fin)
    return np.stack(outs), np.stack(finals)


def _errs(o, o_ref, st, st_ref):
    eo = max(slice_err(o[i, :, h], o_ref[i, :, h]) for i in range(o.shape[0]) for h in range(o.shape[2]))
    es = max(slice_err(st[i, h], st_ref[i, h]) for i in range(st.shape[0]) for h in range(st.shape[1]))
    return eo, es


@pytest.mark.parametrize("T,gate_scale", [(64, 1.0), (256, 1.0), (256, 0.01)])
def test_continuation_after_resume(T, gate_scale):
    w = wl.tp_rank_3584()
    x, C, N, H = w.inputs, w.interval, w.inputs.total_tokens, w.inputs.n_heads
    cold = api.prefill(api.to_device(x), C)
    B = la.strict_prefix_boundary(N, C, N)
    row = B // C - 1
    res = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], cold.ckpt[row:row + 1].clone(), C)
    torch.cuda.synchronize()
    tok = wl.random_inputs(40 + T, [T], H, 128, 128, gate_scale=gate_scale)
    shape = la.make_shape(1, H, 128, 128, C)
    s_cold = cold.final_state.clone()
    s_res = res.final_state.clone()
    o_cold = _decode_gpu(shape, tok, 1, T, s_cold)
    o_res = _decode_gpu(shape, tok, 1, T, s_res)
    # the paper's acceptance check: cold and reloaded runs continue identically
    assert torch.equal(o_cold, o_res) and torch.equal(s_cold, s_res)
    _, fin_ref, _ = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta)
    o_ref, st_ref = _decode_oracle(tok, 1, T, fin_ref[None])
    eo, es = _errs(host(o_res), o_ref, host(s_res), st_ref)
    print(f"[parity] decode {T} tokens after resume at {B} (gate_scale {gate_scale}): o {eo:.2e} state {es:.2e}",
          flush=True)
    assert eo <= TOL[la.LA_BF16] and es <= TOL[la.LA_BF16]


@pytest.mark.parametrize("variant", [0, 1])
def test_batched_decode_variants_and_scale(variant):
    n, H, T = 16, 8, 32
    rng = np.random.default_rng(41)
    states = (rng.standard_normal((n, H, 128, 128)) * 0.1).astype(np.float32)
    tok = wl.random_inputs(42, [T] * n, H, 128, 128, gate_scale=0.05)
    shape = la.make_shape(n, H, 128, 128, 256, variant=variant, scale=0.125)
    st = torch.from_numpy(states).cuda()
    o = _decode_gpu(shape, tok, n, T, st)
    o_ref, st_ref = _decode_oracle(tok, n, T, states, variant=variant, scale=0.125)
    eo, es = _errs(host(o), o_ref, host(st), st_ref)
    print(f"[parity] decode batch 16 x 8 heads, variant {variant}, scale 1/8: o {eo:.2e} state {es:.2e}",
          flush=True)
    assert eo <= TOL[la.LA_BF16] and es <= TOL[la.LA_BF16]


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64)])
def test_decode_head_dims(dk, dv):
    n, H, T = 3, 4, 48
    tok = wl.random_inputs(43 + dk + dv, [T] * n, H, dk, dv, gate_scale=0.02)
    shape = la.make_shape(n, H, dk, dv, 256)
    states = np.zeros((n, H, dk, dv), np.float32)
    st = torch.zeros((n, H, dk, dv), dtype=torch.float32, device="cuda")
    o = _decode_gpu(shape, tok, n, T, st)
    o_ref, st_ref = _decode_oracle(tok, n, T, states)
    eo, es = _errs(host(o), o_ref, host(st), st_ref)
    print(f"[parity] decode dk={dk} dv={dv}: o {eo:.2e} state {es:.2e}", flush=True)
    assert eo <= TOL[la.LA_BF16] and es <= TOL[la.LA_BF16]


def test_decode_fp32_after_tiny_prefill():
    w = wl.tiny_fp32()
    x, C = w.inputs, w.interval
    res = api.prefill(api.to_device(x), C)
    torch.cuda.synchronize()
    T = 256
    tok = wl.random_inputs(44, [T], 1, 64, 64, io_dtype=wl.F32, gate_scale=0.01)
    shape = la.make_shape(1, 1, 64, 64, C, io_dtype=la.LA_F32)
    st = res.final_state.clone()
    o = _decode_gpu(shape, tok, 1, T, st)
    _, fin_ref, _ = oracle.gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta)
    o_ref, st_ref = _decode_oracle(tok, 1, T, fin_ref[None])
    eo, es = _errs(host(o), o_ref, host(st), st_ref)
    print(f"[parity] decode fp32 256 tokens after the tiny prefill: o {eo:.2e} state {es:.2e}", flush=True)
    assert eo <= TOL[la.LA_F32] and es <= TOL[la.LA_F32]
