"""GPU tests of la_prefill_stages: the stages of one prefill call run
separately, on different streams ordered by events, give the monolithic
call's results bit for bit.  The resume case prepares its suffix on a side
stream while the state it starts from is still being restored, the overlap
the stage split exists for.
"""
import numpy as np
import pytest
import torch

from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la
from paper_2609_15030_amd import workloads as wl

pytestmark = pytest.mark.gpu
P, S, O = la.LA_STAGE_PREPARE, la.LA_STAGE_SCAN, la.LA_STAGE_OUTPUT


def _equal(a, b):
    return (torch.equal(a.o, b.o) and torch.equal(a.final_state, b.final_state)
            and (a.ckpt is None or torch.equal(a.ckpt, b.ckpt)))


@pytest.mark.parametrize("lens,C", [([3584], 256), ([4096, 1500], 1024), ([1000, 3584, 257], 256)])
def test_cold_stages_across_streams_equal_monolithic(lens, C):
    x = wl.random_inputs(60 + C, lens, 8, 128, 128, gate_scale=0.01)
    xd = api.to_device(x)
    ref = api.Prefill(xd, C).run()
    p = api.Prefill(xd, C)
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    p.run(stream=main, stages=P | S)
    done_scan = torch.cuda.Event()
    done_scan.record(main)
    side.wait_event(done_scan)
    with torch.cuda.stream(side):
        p.run(stream=side, stages=O)
    main.wait_stream(side)
    torch.cuda.synchronize()
    res = api.PrefillResult(p.o, p.final, p.ckpt, p.ckpt_offsets, p.n_ckpt_rows)
    torch.cuda.synchronize()
    assert _equal(res, ref)


@pytest.mark.parametrize("C", [256, 1024])
def test_resume_prepared_while_state_restores(C):
    N, H = 4096, 8
    x = wl.random_inputs(70 + C, [N], H, 128, 128, gate_scale=0.01)
    cold = api.prefill(api.to_device(x), C)
    B = la.strict_prefix_boundary(N, C, N)
    j = B // C - 1
    n_ck = cold.n_ckpt_rows
    pool = torch.empty((n_ck * H, 128 * 128), device="cuda")
    ids = torch.arange(n_ck * H, dtype=torch.int32, device="cuda")
    la.la_state_save_paged(cold.ckpt, pool, ids)
    torch.cuda.synchronize()
    xs = api.to_device(x.tokens(B, N))
    ref = api.prefill_resume(xs, [B], cold.ckpt[j:j + 1].clone(), C)
    # restore on the main stream while the suffix is prepared on a side stream
    state = torch.full((1, H, 128, 128), float("nan"), device="cuda")
    r = api.Prefill(xs, C, starts=[B])
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    side.wait_stream(main)                 # the suffix inputs were copied on main
    with torch.cuda.stream(side):
        r.run(state, stream=side, stages=P)
    la.la_state_restore_paged(pool, ids[j * H:(j + 1) * H].contiguous(), state, stream=main)
    main.wait_stream(side)
    r.run(state, stream=main, stages=S | O)
    torch.cuda.synchronize()
    assert torch.equal(r.o, ref.o) and torch.equal(r.final, ref.final_state) and torch.equal(r.ckpt, ref.ckpt)
    assert torch.equal(r.o, cold.o[B:]) and torch.equal(r.final, cold.final_state)


@pytest.mark.parametrize("dk,dv,io", [(64, 64, wl.BF16), (64, 128, wl.BF16), (128, 64, wl.BF16), (128, 128, wl.BF16),
                                      (64, 64, wl.F32), (64, 128, wl.F32)])
def test_scan_output_wave_equals_split_output_kernel(dk, dv, io):
    """One call with the scan and output stages together reads the output
    out in the scan kernel's output wave; split calls run the output kernel
    on the state and U the scan left in the workspace.  Same bits, on a
    ragged varlen batch (partial last chunks, a 1-token and an empty
    sequence)."""
    lens = [1000, 0, 257, 64, 1]
    C = 256 if io == wl.BF16 else 64
    x = wl.random_inputs(90 + dk + dv, lens, 3, dk, dv, io_dtype=io, gate_scale=0.02)
    xd = api.to_device(x)
    ref = api.Prefill(xd, C).run()
    p = api.Prefill(xd, C)
    p.run(stages=P | S)
    p.run(stages=O)
    torch.cuda.synchronize()
    res = api.PrefillResult(p.o, p.final, p.ckpt, p.ckpt_offsets, p.n_ckpt_rows)
    assert _equal(ref, res)


def test_split_handoff_exact_at_batch_scale():
    """The scan stage on its own hands the state entering every chunk and U
    to the output stage through the workspace (16-byte words per lane).
    Regression: a store-data hazard once left a few of those words wrong on
    some runs (about 1 KiB in a 700 MiB workspace), so small batches rarely
    showed it.  Three stage-split runs of the 16-sequence varlen batch must
    equal the one-call result bit for bit."""
    w = wl.batched_varlen()
    xd = api.to_device(w.inputs)
    ref = api.Prefill(xd, w.interval).run()
    ref_o, ref_f, ref_c = ref.o.clone(), ref.final_state.clone(), ref.ckpt.clone()
    p = api.Prefill(xd, w.interval)
    for _ in range(3):
        p.run(stages=P)
        p.run(stages=S)
        p.run(stages=O)
        torch.cuda.synchronize()
        assert torch.equal(p.o, ref_o) and torch.equal(p.final, ref_f) and torch.equal(p.ckpt, ref_c)
