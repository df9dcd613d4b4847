"""Pins for the fp64 oracle, checked against things other than the oracle.

The paper prints no numeric value for any state or output, so the oracle's
recurrence is pinned by mathematics:

* a backward unrolling that never forms the state (O(T^2) per output),
* closed forms (orthonormal keys, a repeated key, beta = 0, one token,
  the delta rule's overwrite property),
* special cases where the two variants must coincide (g = 0),
* invariants the paper's position semantics fix (section 2.2): a state for
  prefix [0, B) continues from B, so resuming from a checkpoint reproduces
  the full run bit for bit, and the checkpoint at P equals the final state
  of a run over [0, P),
* agreement with a 40-digit decimal evaluation on tiny inputs.

Every test here runs on the CPU.
"""
from decimal import Decimal, getcontext

import numpy as np
import pytest

import oracle
from oracle.gdr import LITERAL, DECAYED_DELTA, gdr_prefill_seq
from paper_2609_15030_amd import workloads as wl


def _rand(seed, T, H, dk, dv, io=wl.F32):
    x = wl.random_inputs(seed, [T], H, dk, dv, io)
    return x.q, x.k, x.v, x.g, x.beta


def unrolled_outputs(q, k, v, g, beta, variant, scale=1.0, S0=None, probe=None):
    """o_t by walking the transposed transition maps backwards from q_t.

    With M_s = a_s I - b_s k_s k_s^T (a_s = exp(g_s); b_s = beta_s for the
    literal rule, beta_s * a_s for the decayed one) the state is
    S_t = M_t S_{t-1} + beta_t k_t v_t^T, hence
    o_t = scale * (sum_s beta_s (k_s . r_s) v_s + S0^T r_0),
    where r_t = q_t and r_{s-1} = M_s r_s (M_s is symmetric).
    ``probe`` replaces q_t by an arbitrary vector (to read S_t^T x).
    """
    T, H, dk = q.shape
    dv = v.shape[2]
    q, k, v, g, beta = (np.asarray(a, np.float64) for a in (q, k, v, g, beta))
    out = np.zeros((T, H, dv))
    for h in range(H):
        for t in range(T):
            r = (q[t, h] if probe is None else probe[h]).copy()
            acc = np.zeros(dv)
            for s in range(t, -1, -1):
                ks = k[s, h]
                a = np.exp(g[s, h])
                b = beta[s, h] * (a if variant == DECAYED_DELTA else 1.0)
                acc += beta[s, h] * np.dot(ks, r) * v[s, h]
                r = a * r - b * ks * np.dot(ks, r)
            if S0 is not None:
                acc += S0[h].T @ r
            out[t, h] = scale * acc
    return out


@pytest.mark.parametrize("variant", [LITERAL, DECAYED_DELTA])
@pytest.mark.parametrize("seed,T,H,dk,dv", [(11, 40, 2, 8, 8), (12, 33, 1, 16, 4), (13, 24, 3, 4, 12)])
def test_token_loop_matches_backward_unrolling(variant, seed, T, H, dk, dv):
    q, k, v, g, beta = _rand(seed, T, H, dk, dv)
    rng = np.random.default_rng(seed)
    S0 = rng.standard_normal((H, dk, dv))
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta, state_in=S0, variant=variant, scale=0.7)
    ref = unrolled_outputs(q, k, v, g, beta, variant, scale=0.7, S0=S0)
    assert np.max(np.abs(o - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))
    # the final state, read one row at a time: S_T^T e_i = row i of S_T
    for i in range(dk):
        e = np.zeros((H, dk))
        e[:, i] = 1.0
        rows = unrolled_outputs(q, k, v, g, beta, variant, S0=S0, probe=e)[-1]
        assert np.allclose(S[:, i, :], rows, rtol=0, atol=1e-12 * max(1.0, np.abs(S).max()))


def test_orthonormal_keys_reduce_to_decayed_linear_attention():
    """Orthogonal keys never interfere: S_t = sum_s exp(G_t - G_s) beta_s k_s v_s^T."""
    T, dk, dv = 12, 16, 5
    rng = np.random.default_rng(5)
    basis, _ = np.linalg.qr(rng.standard_normal((dk, dk)))
    k = basis.T[:T][:, None, :].astype(np.float32)            # orthonormal rows
    q = rng.standard_normal((T, 1, dk)).astype(np.float32)
    v = rng.standard_normal((T, 1, dv)).astype(np.float32)
    g = -rng.uniform(0.0, 2.0, (T, 1)).astype(np.float32)
    beta = rng.uniform(0.1, 1.0, (T, 1)).astype(np.float32)
    kd, qd, vd = (a.astype(np.float64)[:, 0] for a in (k, q, v))
    G = np.cumsum(g[:, 0].astype(np.float64))
    for variant in (LITERAL, DECAYED_DELTA):
        o, S, _ = gdr_prefill_seq(q, k, v, g, beta, variant=variant)
        for t in range(T):
            St = sum(np.exp(G[t] - G[s]) * beta[s, 0] * np.outer(kd[s], vd[s]) for s in range(t + 1))
            assert np.allclose(o[t, 0], St.T @ qd[t], rtol=1e-6, atol=1e-6)
        assert np.allclose(S[0], St, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("variant", [LITERAL, DECAYED_DELTA])
def test_repeated_unit_key_gives_scalar_recurrence(variant):
    """With one repeated key, S_t = k w_t^T and w_t follows a first-order
    recurrence (kk = k.k of the stored key, 1 up to fp32 rounding):
    literal: w_t = (a_t - beta_t kk) w_{t-1} + beta_t v_t;
    decayed: w_t = a_t (1 - beta_t kk) w_{t-1} + beta_t v_t.
    """
    T, dk, dv = 30, 8, 6
    rng = np.random.default_rng(7)
    kv = rng.standard_normal(dk)
    kv /= np.linalg.norm(kv)
    k = np.tile(kv.astype(np.float32), (T, 1))[:, None, :]
    kd = k[0, 0].astype(np.float64)
    q = rng.standard_normal((T, 1, dk)).astype(np.float32)
    v = rng.standard_normal((T, 1, dv)).astype(np.float32)
    g = -rng.uniform(0, 1.5, (T, 1)).astype(np.float32)
    beta = rng.uniform(0, 1, (T, 1)).astype(np.float32)
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta, variant=variant)
    kk = float(np.dot(kd, kd))
    w = np.zeros(dv)
    for t in range(T):
        a, b = np.exp(float(g[t, 0])), float(beta[t, 0])
        decay = (a - b * kk) if variant == LITERAL else a * (1 - b * kk)
        w = decay * w + b * v[t, 0].astype(np.float64)
        assert np.allclose(o[t, 0], w * np.dot(kd, q[t, 0]), rtol=1e-9, atol=1e-12)
    assert np.allclose(S[0], np.outer(kd, w), rtol=1e-9, atol=1e-12)


def test_zero_gate_makes_variants_coincide():
    q, k, v, g, beta = _rand(21, 50, 2, 8, 8)
    g = np.zeros_like(g)
    o0, s0, _ = gdr_prefill_seq(q, k, v, g, beta, variant=LITERAL)
    o1, s1, _ = gdr_prefill_seq(q, k, v, g, beta, variant=DECAYED_DELTA)
    assert np.array_equal(o0, o1) and np.array_equal(s0, s1)


def test_variants_differ_when_gated():
    q, k, v, g, beta = _rand(22, 50, 2, 8, 8)
    o0, _, _ = gdr_prefill_seq(q, k, v, g, beta, variant=LITERAL)
    o1, _, _ = gdr_prefill_seq(q, k, v, g, beta, variant=DECAYED_DELTA)
    assert np.max(np.abs(o0 - o1)) > 1e-3


def test_zero_beta_is_pure_decay_of_initial_state():
    """beta = 0: S_t = exp(G_t) S_0 with G_t summed from the first token of the call."""
    q, k, v, g, beta = _rand(23, 20, 2, 6, 5)
    beta = np.zeros_like(beta)
    rng = np.random.default_rng(3)
    S0 = rng.standard_normal((2, 6, 5))
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta, state_in=S0, start=37, scale=1.3)
    G = np.cumsum(g.astype(np.float64), axis=0)
    for t in range(20):
        for h in range(2):
            ref = 1.3 * np.exp(G[t, h]) * (S0[h].T @ q[t, h].astype(np.float64))
            assert np.allclose(o[t, h], ref, rtol=1e-12, atol=1e-14)
    assert np.allclose(S, np.exp(G[-1])[:, None, None] * S0, rtol=1e-12, atol=1e-14)


def test_single_token_from_zero_state():
    q, k, v, g, beta = _rand(24, 1, 3, 8, 4)
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta, scale=0.5)
    for h in range(3):
        kd, qd, vd = (a[0, h].astype(np.float64) for a in (k, q, v))
        b = float(beta[0, h])
        assert np.allclose(S[h], b * np.outer(kd, vd), rtol=1e-15, atol=0)
        assert np.allclose(o[0, h], 0.5 * b * np.dot(kd, qd) * vd, rtol=1e-14, atol=1e-16)


def test_delta_rule_overwrites_association():
    """alpha = 1, beta = 1, unit key: writing v1 then v2 under key k leaves S^T k = v2."""
    dk, dv = 8, 3
    rng = np.random.default_rng(9)
    kv = rng.standard_normal(dk)
    kv /= np.linalg.norm(kv)
    k = np.stack([kv, kv]).astype(np.float32)[:, None, :]
    v = rng.standard_normal((2, 1, dv)).astype(np.float32)
    q = k.copy()
    g = np.zeros((2, 1), np.float32)
    beta = np.ones((2, 1), np.float32)
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta)
    kk = float(np.dot(k[0, 0].astype(np.float64), k[0, 0].astype(np.float64)))
    assert np.allclose(o[0, 0], kk * v[0, 0], atol=1e-6)     # S_1^T k = v1 (|k|^2 ~ 1)
    assert np.allclose(o[1, 0], v[1, 0], atol=1e-6)          # S_2^T k = v2, v1 forgotten


@pytest.mark.parametrize("variant", [LITERAL, DECAYED_DELTA])
def test_resume_from_checkpoint_is_bit_exact(variant):
    """Section 2.2: a state for prefix [0, B) supports continuation from B."""
    x = wl.tiny_fp32().inputs
    o, S, ck = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=16, variant=variant)
    assert ck.shape == (16, 1, 64, 64)
    for B in (16, 64, 240):
        row = B // 16 - 1
        o2, S2, ck2 = gdr_prefill_seq(x.q[B:], x.k[B:], x.v[B:], x.g[B:], x.beta[B:],
                                      start=B, interval=16, state_in=ck[row], variant=variant)
        assert np.array_equal(o2, o[B:])
        assert np.array_equal(S2, S)
        assert np.array_equal(ck2, ck[row + 1:])


def test_checkpoint_equals_state_of_prefix_run():
    x = wl.random_inputs(31, [200], 2, 8, 8, wl.BF16)
    _, _, ck = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=48)
    assert ck.shape[0] == 200 // 48
    for j in range(ck.shape[0]):
        P = 48 * (j + 1)
        _, SP, _ = gdr_prefill_seq(x.q[:P], x.k[:P], x.v[:P], x.g[:P], x.beta[:P])
        assert np.array_equal(ck[j], SP)


def test_checkpoint_rows_follow_absolute_positions():
    """Checkpoints sit at absolute multiples of C in (start, end]."""
    x = wl.random_inputs(32, [70], 1, 4, 4)
    S0 = np.random.default_rng(1).standard_normal((1, 4, 4))
    _, _, ck = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, start=32, interval=16, state_in=S0)
    assert ck.shape[0] == (32 + 70) // 16 - 2          # P = 48, 64, 80, 96
    _, S48, _ = gdr_prefill_seq(x.q[:16], x.k[:16], x.v[:16], x.g[:16], x.beta[:16],
                                start=32, state_in=S0)
    assert np.array_equal(ck[0], S48)


def test_thread_count_does_not_change_results():
    x = wl.random_inputs(33, [300], 6, 16, 16, wl.BF16)
    a = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=64, n_threads=1)
    *b, used = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=64, n_threads=4,
                               return_threads=True)
    assert used == 4
    for u, w in zip(a, b):
        assert np.array_equal(u, w)


def test_prefix_double_application_diverges():
    """The pre-fix failure (section 3.2): the restored state already covers
    [0, N) while the scheduler feeds token N - 1 again.  The oracle must see
    a different state from the correct one (the failure is observable)."""
    x = wl.random_inputs(34, [64], 2, 8, 8)
    _, S_full, ck = gdr_prefill_seq(x.q, x.k, x.v, x.g, x.beta, interval=32)
    _, S_bad, _ = gdr_prefill_seq(x.q[63:], x.k[63:], x.v[63:], x.g[63:], x.beta[63:],
                                  start=63, state_in=ck[-1])
    assert np.max(np.abs(S_bad - S_full)) > 1e-3
    _, S_ok, _ = gdr_prefill_seq(x.q[32:], x.k[32:], x.v[32:], x.g[32:], x.beta[32:],
                                 start=32, state_in=ck[0])
    assert np.array_equal(S_ok, S_full)


def test_matches_forty_digit_decimal_evaluation():
    """fp64 rounding only: a 40-digit evaluation of the same recurrence agrees
    to near machine precision on a tiny case (checks the loop's accumulation,
    not the formula, which the tests above pin)."""
    getcontext().prec = 40
    q, k, v, g, beta = _rand(41, 16, 1, 4, 3)
    o, S, _ = gdr_prefill_seq(q, k, v, g, beta)
    D = lambda a: Decimal(float(a))
    Sd = [[Decimal(0)] * 3 for _ in range(4)]
    for t in range(16):
        a = D(g[t, 0]).exp()
        b = D(beta[t, 0])
        kt = [D(x) for x in k[t, 0]]
        pred = [sum(Sd[r][c] * kt[r] for r in range(4)) for c in range(3)]
        u = [b * (D(v[t, 0, c]) - pred[c]) for c in range(3)]
        Sd = [[a * Sd[r][c] + kt[r] * u[c] for c in range(3)] for r in range(4)]
        qt = [D(x) for x in q[t, 0]]
        ot = [sum(Sd[r][c] * qt[r] for r in range(4)) for c in range(3)]
        assert np.allclose(o[t, 0], [float(x) for x in ot], rtol=1e-13, atol=1e-15)
    assert np.allclose(S[0], [[float(x) for x in row] for row in Sd], rtol=1e-13, atol=1e-15)


def test_varlen_front_end_matches_per_sequence_calls():
    x = wl.random_inputs(42, [17, 64, 1, 90], 2, 8, 8, wl.BF16)
    starts = [0, 64, 32, 0]
    o, fin, cks = oracle.gdr_prefill(x, starts=starts, interval=32)
    for i in range(4):
        xi = x.seq(i)
        oi, si, ci = gdr_prefill_seq(xi.q, xi.k, xi.v, xi.g, xi.beta, start=starts[i], interval=32)
        a, b = x.cu_seqlens[i], x.cu_seqlens[i + 1]
        assert np.array_equal(o[a:b], oi) and np.array_equal(fin[i], si)
        assert (ci is None and cks[i] is None) or np.array_equal(ci, cks[i])
