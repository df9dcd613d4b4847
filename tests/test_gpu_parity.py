"""GPU parity: the gfx950 prefill against the fp64 oracle, through the C ABI.

Covers the tiny fp32 workload (mid-chunk checkpoints, resume at 240), the
one-TP-rank workload (T = 3,584, resume at the strict-prefix boundary 3,328),
ragged lengths, small and non-dividing checkpoint intervals, both recurrence
variants, every built head-dimension pair, and the invariants the paper's
position semantics fix: resume from a checkpoint equals recompute, and the
restored state is the state for exactly the prefix [0, B).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

from parity import TOL, compare, host, oracle_run, out_err, state_err

pytestmark = pytest.mark.gpu


def _run_cold(x, C, variant=0, scale=1.0):
    xd = api.to_device(x)
    res = api.prefill(xd, C, variant, scale)
    torch.cuda.synchronize()
    return xd, res


def test_tiny_fp32_full_prefill_and_resume_at_240():
    w = wl.tiny_fp32()
    x, C = w.inputs, w.interval
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_F32], "tiny fp32 cold")
    # strict-prefix restore at B = 240 from the GPU's own checkpoint
    B = la.strict_prefix_boundary(256, C, w.available[0])
    assert B == 240
    row = B // C - 1
    state = res.ckpt[row:row + 1].clone()
    xs = api.to_device(x.tokens(B, 256))
    r2 = api.prefill_resume(xs, [B], state, C)
    torch.cuda.synchronize()
    o_ref, fin_ref, ck_ref = ref
    assert out_err(host(r2.o), o_ref[B:], [0, 256 - B]) <= TOL[la.LA_F32]
    assert state_err(host(r2.final_state), fin_ref) <= TOL[la.LA_F32]
    assert state_err(host(r2.ckpt), ck_ref[row + 1:]) <= TOL[la.LA_F32]
    # resume equals recompute on the GPU, bit for bit (same chunk grid)
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_tp_rank_bf16_cold_and_complete_hit_resume():
    w = wl.tp_rank_3584()
    x, C = w.inputs, w.interval
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], "T=3584 H=8 bf16 cold")
    B = la.strict_prefix_boundary(3584, C, 3584)
    assert B == 3328
    state = res.ckpt[B // C - 1:B // C].clone()
    xs = api.to_device(x.tokens(B, 3584))
    r2 = api.prefill_resume(xs, [B], state, C)
    torch.cuda.synchronize()
    o_ref, fin_ref, _ = ref
    eo = out_err(host(r2.o), o_ref[B:], [0, 3584 - B])
    es = state_err(host(r2.final_state), fin_ref)
    print(f"[parity] T=3584 resume at {B}: o {eo:.3e} final {es:.3e}", flush=True)
    assert eo <= TOL[la.LA_BF16] and es <= TOL[la.LA_BF16]
    assert torch.equal(r2.o, res.o[B:]) and torch.equal(r2.final_state, res.final_state)


def test_resume_from_oracle_checkpoint():
    """Restore the oracle's own fp64 checkpoint (rounded to the fp32 state
    dtype) and resume: the GPU continues the oracle's run."""
    x = wl.random_inputs(501, [700], 4, 128, 128, wl.BF16)
    C, B = 128, 512
    o_ref, fin_ref, ck_ref = oracle_run(x, interval=C)
    state = torch.from_numpy(ck_ref[B // C - 1:B // C].astype(np.float32)).cuda()
    xs = api.to_device(x.tokens(B, 700))
    r = api.prefill_resume(xs, [B], state, C)
    torch.cuda.synchronize()
    assert out_err(host(r.o), o_ref[B:], [0, 700 - B]) <= TOL[la.LA_BF16]
    assert state_err(host(r.final_state), fin_ref) <= TOL[la.LA_BF16]
    assert state_err(host(r.ckpt), ck_ref[B // C:]) <= TOL[la.LA_BF16]


@pytest.mark.parametrize("io", [wl.BF16, wl.F32])
def test_ragged_varlen_batch(io):
    lens = [1, 63, 64, 65, 200, 0, 130, 7]
    d = 128 if io == wl.BF16 else 64
    x = wl.random_inputs(502, lens, 3, d, d, io)
    C = 64
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    tol = TOL[la.LA_BF16 if io == wl.BF16 else la.LA_F32]
    compare(res, ref, x.cu_seqlens, tol, f"ragged varlen {io}")
    # the empty sequence's final state is the zero state
    assert torch.count_nonzero(res.final_state[5]) == 0


@pytest.mark.parametrize("C", [16, 48, 100, 192, 1])
def test_checkpoint_intervals(C):
    x = wl.random_inputs(503, [300, 77], 2, 128, 128, wl.BF16)
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], f"C={C}")


@pytest.mark.parametrize("variant", [la.LA_GDR_LITERAL, la.LA_GDR_DECAYED_DELTA])
@pytest.mark.parametrize("io", [wl.BF16, wl.F32])
def test_variants_and_scale(variant, io):
    x = wl.random_inputs(504, [333], 2, 64, 64, io)
    xd, res = _run_cold(x, 64, variant=variant, scale=0.125)
    ref = oracle_run(x, interval=64, variant=variant, scale=0.125)
    tol = TOL[la.LA_BF16 if io == wl.BF16 else la.LA_F32]
    compare(res, ref, x.cu_seqlens, tol, f"variant={variant} {io} scale=1/8")


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
def test_head_dims(dk, dv):
    x = wl.random_inputs(505, [190, 64], 2, dk, dv, wl.BF16)
    xd, res = _run_cold(x, 64)
    ref = oracle_run(x, interval=64)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], f"dk={dk} dv={dv}")


def test_fp32_wide_heads():
    x = wl.random_inputs(506, [257], 2, 128, 128, wl.F32)
    xd, res = _run_cold(x, 64)
    compare(res, oracle_run(x, interval=64), x.cu_seqlens, TOL[la.LA_F32], "fp32 d=128")


def test_run_to_run_determinism_and_batch_invariance():
    lens = [300, 1000, 64]
    x = wl.random_inputs(507, lens, 4, 128, 128, wl.BF16)
    xd = api.to_device(x)
    a = api.prefill(xd, 256)
    o1, f1, c1 = a.o.clone(), a.final_state.clone(), a.ckpt.clone()
    b = api.prefill(xd, 256)
    torch.cuda.synchronize()
    assert torch.equal(o1, b.o) and torch.equal(f1, b.final_state) and torch.equal(c1, b.ckpt)
    # sequence 1 alone gives bit-identical rows to sequence 1 inside the batch
    alone = api.prefill(api.to_device(x.seq(1)), 256)
    torch.cuda.synchronize()
    s, e = int(x.cu_seqlens[1]), int(x.cu_seqlens[2])
    assert torch.equal(alone.o, o1[s:e]) and torch.equal(alone.final_state[0], f1[1])
    off = int(a.ckpt_offsets[1])
    assert torch.equal(alone.ckpt, c1[off:off + alone.n_ckpt_rows])


def test_resume_rejects_empty_suffix_and_misaligned_state():
    x = wl.random_inputs(508, [64], 1, 64, 64, wl.BF16)
    xd = api.to_device(x)
    st = torch.zeros((1, 1, 64, 64), device="cuda")
    p = api.Prefill(xd, 64, starts=[64])
    p.o.fill_(7.0)
    o_before = p.o.clone()
    # misaligned: B = 32 is not a multiple of C = 64
    p.starts[:] = 32
    p.start_dev.fill_(32)
    with pytest.raises(la.LinAttnError) as e:
        p.run(st)
    assert e.value.status == la.LA_ERR_MISALIGNED_STATE
    torch.cuda.synchronize()
    assert torch.equal(p.o, o_before)       # nothing launched, outputs untouched
    # empty suffix: the pre-fix failure (B = N with one more token scheduled) is unrepresentable
    xe = api.DeviceInputs(xd.q[:0], xd.k[:0], xd.v[:0], xd.g[:0], xd.beta[:0],
                          torch.zeros(2, dtype=torch.int32, device="cuda"),
                          np.zeros(2, np.int32), xd.io_dtype)
    shape = la.make_shape(1, 1, 64, 64, 64)
    ws = torch.empty(la.la_prefill_workspace_bytes(shape, 0), dtype=torch.uint8, device="cuda")
    starts = np.array([64], np.int64)
    st_code = la.la_prefill_resume(shape, xd.q, xd.k, xd.v, xd.g, xd.beta, xe.cu_dev, xe.cu_host,
                                   torch.from_numpy(starts).cuda(), starts, st, xd.q, None, None,
                                   None, None, ws, check=False)
    assert st_code == la.LA_ERR_EMPTY_SUFFIX


def test_prefix_double_application_is_detected():
    """The pre-fix failure reproduced on the GPU: restoring the state for [0, N)
    and feeding token N - 1 again gives a different state from the oracle's;
    the strict-prefix restore matches it."""
    x = wl.random_inputs(509, [512], 2, 128, 128, wl.BF16)
    C, N = 256, 512
    xd, res = _run_cold(x, C)
    _, fin_ref, _ = oracle_run(x, interval=C)
    full = res.ckpt[1:2].clone()                     # state for [0, 512) = [0, N)
    bad = api.prefill_resume(api.to_device(x.tokens(N - 1, N)), [N - 1], full, 1)
    torch.cuda.synchronize()
    assert state_err(host(bad.final_state), fin_ref) > 0.05
    B = la.strict_prefix_boundary(N, C, N)
    good = api.prefill_resume(api.to_device(x.tokens(B, N)), [B], res.ckpt[B // C - 1:B // C].clone(), C)
    torch.cuda.synchronize()
    assert state_err(host(good.final_state), fin_ref) <= TOL[la.LA_BF16]


def test_many_chains_in_several_rounds():
    """A batch of 320 (sequence, head) chains: more fused-scan workgroups
    than CUs, so they run in several rounds.  Parity with the oracle on
    every head; a sequence alone gives the same bits as inside the batch;
    and every sequence resumed at its strict-prefix boundary from the
    batch's own checkpoints reproduces the cold run's tail and final state
    bit for bit."""
    rng = np.random.default_rng(511)
    lens = [int(n) for n in rng.integers(1, 400, size=40)]
    H, C = 8, 64
    x = wl.random_inputs(511, lens, H, 128, 128, wl.BF16)
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], "40 seqs x 8 heads, several rounds")
    cu = x.cu_seqlens
    i = int(np.argmax(lens))
    alone = api.prefill(api.to_device(x.seq(i)), C)
    torch.cuda.synchronize()
    s, e = int(cu[i]), int(cu[i + 1])
    off = int(res.ckpt_offsets[i])
    assert torch.equal(alone.o, res.o[s:e]) and torch.equal(alone.final_state[0], res.final_state[i])
    assert torch.equal(alone.ckpt, res.ckpt[off:off + alone.n_ckpt_rows])
    # strict-prefix resume of every sequence from the batch's checkpoints
    starts = [la.strict_prefix_boundary(n, C, n) for n in lens]
    rows = [np.arange(int(cu[j]) + b, int(cu[j + 1])) for j, b in enumerate(starts)]
    idx = np.concatenate(rows)
    xs = wl.Inputs(x.q[idx], x.k[idx], x.v[idx], x.g[idx], x.beta[idx],
                   np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32), x.io_dtype)
    state = torch.zeros((len(lens), H, 128, 128), dtype=torch.float32, device="cuda")
    for j, b in enumerate(starts):
        if b > 0:
            state[j] = res.ckpt[int(res.ckpt_offsets[j]) + b // C - 1]
    r2 = api.prefill_resume(api.to_device(xs), starts, state, C)
    torch.cuda.synchronize()
    assert torch.equal(r2.o, res.o[torch.from_numpy(idx).cuda()])
    assert torch.equal(r2.final_state, res.final_state)


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
def test_fused_scan_batch_head_dims(dk, dv):
    """33 sequences x 8 heads for every built head-dimension pair, on the
    fused scan (the form is asserted): parity with the oracle on every head,
    and a sequence alone gives the same bits as inside the batch."""
    rng = np.random.default_rng(600 + dk + dv)
    lens = [int(n) for n in rng.integers(64, 700, size=33)]
    C = 128
    x = wl.random_inputs(600 + dk + dv, lens, 8, dk, dv, wl.BF16)
    assert la.la_prefill_form(la.make_shape(33, 8, dk, dv, C)) == la.LA_FORM_FUSED_SCAN
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], f"33 seqs x 8 heads dk={dk} dv={dv}, fused scan")
    i = int(np.argmax(lens))
    alone = api.prefill(api.to_device(x.seq(i)), C)
    torch.cuda.synchronize()
    s, e = int(x.cu_seqlens[i]), int(x.cu_seqlens[i + 1])
    assert torch.equal(alone.o, res.o[s:e]) and torch.equal(alone.final_state[0], res.final_state[i])


@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 64), (128, 128)])
def test_two_level_head_dims(dk, dv):
    """The two-level fused scan (C = 512: 8 chunks per interval, segments of
    8 chunks) for head-dimension pairs that split the map's columns
    differently: parity on every head, and a resume from the run's own
    checkpoint reproduces its tail bit for bit."""
    lens = [1500, 700, 2048]
    C = 512
    x = wl.random_inputs(620 + dk + dv, lens, 3, dk, dv, wl.BF16)
    assert la.la_prefill_form(la.make_shape(3, 3, dk, dv, C)) == la.LA_FORM_FUSED_TWO_LEVEL
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], f"two-level dk={dk} dv={dv}")
    i, B = 2, 1536
    xs = api.to_device(x.seq(i).tokens(B, lens[i]))
    off = int(res.ckpt_offsets[i])
    r2 = api.prefill_resume(xs, [B], res.ckpt[off + B // C - 1:off + B // C].clone(), C)
    torch.cuda.synchronize()
    s = int(x.cu_seqlens[i])
    assert torch.equal(r2.o, res.o[s + B:s + lens[i]]) and torch.equal(r2.final_state[0], res.final_state[i])


def _concat(parts):
    """The sequences of several packed inputs, in order, as one batch."""
    cat = lambda f: np.concatenate([getattr(x, f) for x in parts])
    lens = np.concatenate([np.diff(x.cu_seqlens) for x in parts])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return wl.Inputs(cat("q"), cat("k"), cat("v"), cat("g"), cat("beta"), cu, parts[0].io_dtype)


def test_column_widths_give_the_same_bits():
    """One 300-token sequence (C = 128: two checkpoints) run in calls whose
    chain counts fix the fused scan's widths: alone (8 chains, 32-column
    workgroups), among 32 sequences of its length (256 even chains, 64
    columns), among 64 sequences (512 chains, 128 columns), and in two
    mixed-width launches, once as the longest sequence (its chains at 32
    columns, the short ones' at 64) and once behind a longer one (its
    chains at 64).  Parity with the oracle, and its output, checkpoints and
    final state equal bit for bit across all five calls."""
    H, C, L = 8, 128, 300
    x = wl.random_inputs(641, [L], H, 128, 128, wl.BF16)
    rng = np.random.default_rng(642)
    same = wl.random_inputs(643, [L] * 31, H, 128, 128, wl.BF16)
    mixed = wl.random_inputs(644, [int(n) for n in rng.integers(1, 400, size=63)], H, 128, 128, wl.BF16)
    short = wl.random_inputs(645, [64] * 15, H, 128, 128, wl.BF16)
    longer = wl.random_inputs(646, [1000], H, 128, 128, wl.BF16)
    cases = ((x, (32, 8)), (_concat([same, x]), (64, 0)), (_concat([mixed, x]), (128, 0)),
             (_concat([short, x]), (64, 8)), (_concat([longer, short, x]), (64, 8)))
    runs = []
    for batch, widths in cases:
        shape = la.make_shape(batch.n_seqs, H, 128, 128, C, la.LA_BF16)
        assert la.la_prefill_scan_columns(shape, batch.cu_seqlens) == widths, widths
        _, res = _run_cold(batch, C)
        i = batch.n_seqs - 1
        s, e = int(batch.cu_seqlens[i]), int(batch.cu_seqlens[i + 1])
        off = int(res.ckpt_offsets[i])
        runs.append((res.o[s:e], res.final_state[i:i + 1], res.ckpt[off:off + L // C], widths))
    o_ref, fin_ref, ck_ref = oracle_run(x, interval=C)
    o, fin, ck, _ = runs[0]
    assert out_err(host(o), o_ref, [0, L]) <= TOL[la.LA_BF16]
    assert state_err(host(fin), fin_ref) <= TOL[la.LA_BF16]
    assert state_err(host(ck), ck_ref) <= TOL[la.LA_BF16]
    for o2, fin2, ck2, widths in runs[1:]:
        assert torch.equal(o2, o) and torch.equal(fin2, fin) and torch.equal(ck2, ck), widths


def test_column_width_does_not_change_bits():
    """64 sequences x 8 heads (512 chains: the fused scan runs 128-column
    workgroups) against one of them alone (8 chains: 32-column workgroups):
    parity with the oracle on every head, and the lone sequence's output,
    checkpoints and final state equal its rows in the batch bit for bit."""
    rng = np.random.default_rng(640)
    lens = [int(n) for n in rng.integers(1, 300, size=64)]
    H, C = 8, 128
    x = wl.random_inputs(640, lens, H, 128, 128, wl.BF16)
    xd, res = _run_cold(x, C)
    ref = oracle_run(x, interval=C)
    compare(res, ref, x.cu_seqlens, TOL[la.LA_BF16], "64 seqs x 8 heads, 128-column workgroups")
    cu = x.cu_seqlens
    for i in (int(np.argmax(lens)), 5):
        alone = api.prefill(api.to_device(x.seq(i)), C)
        torch.cuda.synchronize()
        s, e = int(cu[i]), int(cu[i + 1])
        off = int(res.ckpt_offsets[i])
        assert torch.equal(alone.o, res.o[s:e]) and torch.equal(alone.final_state[0], res.final_state[i])
        if alone.n_ckpt_rows:
            assert torch.equal(alone.ckpt, res.ckpt[off:off + alone.n_ckpt_rows])


@pytest.mark.parametrize("seed", [650, 651, 652, 653, 654, 655])
def test_random_batches_against_the_oracle_and_alone(seed):
    """Seeded random batches (2-24 sequences of 0-900 tokens, 1, 3 or 8
    heads, C in {64, 128, 192, 256}, d = 128 bf16): whatever widths the
    batch's chains get, every sequence matches the oracle, and a sequence
    run alone (its own widths) gives the same bits."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 25))
    H = int(rng.choice([1, 3, 8]))
    C = int(rng.choice([64, 128, 192, 256]))
    lens = [int(v) for v in rng.integers(0, 901, size=n)]
    x = wl.random_inputs(seed, lens, H, 128, 128, wl.BF16)
    shape = la.make_shape(n, H, 128, 128, C, la.LA_BF16)
    print(f"[parity] seed {seed}: {n} seqs x {H} heads, C={C}, widths "
          f"{la.la_prefill_scan_columns(shape, x.cu_seqlens)}", flush=True)
    _, res = _run_cold(x, C)
    compare(res, oracle_run(x, interval=C), x.cu_seqlens, TOL[la.LA_BF16], f"random batch {seed}")
    i = int(np.argmax(lens))
    alone = api.prefill(api.to_device(x.seq(i)), C)
    torch.cuda.synchronize()
    s, e = int(x.cu_seqlens[i]), int(x.cu_seqlens[i + 1])
    off = int(res.ckpt_offsets[i])
    assert torch.equal(alone.o, res.o[s:e]) and torch.equal(alone.final_state[0], res.final_state[i])
    if alone.n_ckpt_rows:
        assert torch.equal(alone.ckpt, res.ckpt[off:off + alone.n_ckpt_rows])
