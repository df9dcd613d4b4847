"""Shared helpers for the GPU parity tests (tests only).

Error metric: normwise per slice.  For every (sequence, head) slice of an
output, and every (row, head) slice of a state/checkpoint array, the error is
max |x - ref| / max |ref|; a test bounds the maximum over slices.  (A
per-element relative error is unusable for bf16 data: correct results show
large ratios next to near-zero reference entries.)

Tolerances: 2e-2 for bf16 inputs and 1e-4 for fp32 inputs.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_15030_amd import api
from paper_2609_15030_amd import linattn as la

TOL = {la.LA_BF16: 2e-2, la.LA_F32: 1e-4}


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def slice_err(x: np.ndarray, ref: np.ndarray) -> float:
    den = np.max(np.abs(ref))
    num = np.max(np.abs(x - ref))
    if den == 0:
        return float(num)
    return float(num / den)


def out_err(o: np.ndarray, ref: np.ndarray, cu) -> float:
    """max over (sequence, head) of the normwise error of o rows."""
    worst = 0.0
    for i in range(len(cu) - 1):
        a, b = int(cu[i]), int(cu[i + 1])
        if b == a:
            continue
        for h in range(ref.shape[1]):
            worst = max(worst, slice_err(o[a:b, h], ref[a:b, h]))
    return worst


def state_err(s: np.ndarray, ref: np.ndarray) -> float:
    """max over (row, head) of the normwise error of [rows, H, dk, dv] states."""
    worst = 0.0
    for r in range(ref.shape[0]):
        for h in range(ref.shape[1]):
            worst = max(worst, slice_err(s[r, h], ref[r, h]))
    return worst


def oracle_run(x, starts=None, interval=0, states_in=None, variant=0, scale=1.0):
    o, fin, cks = oracle.gdr_prefill(x, starts=starts, interval=interval, states_in=states_in,
                                     variant=variant, scale=scale)
    cks = [c for c in cks if c is not None]
    ck = np.concatenate(cks, axis=0) if cks else None
    return o, fin, ck


def compare(res: api.PrefillResult, ref, cu, tol, what=""):
    o_ref, fin_ref, ck_ref = ref
    eo = out_err(host(res.o), o_ref, cu)
    es = state_err(host(res.final_state), fin_ref)
    ec = 0.0
    if ck_ref is not None:
        assert res.ckpt is not None and res.ckpt.shape[0] == ck_ref.shape[0], what
        ec = state_err(host(res.ckpt), ck_ref)
    else:
        assert res.ckpt is None or res.ckpt.shape[0] == 0, what
    print(f"[parity] {what}: o {eo:.3e}  final {es:.3e}  ckpt {ec:.3e}  (tol {tol:g})", flush=True)
    assert eo <= tol and es <= tol and ec <= tol, (what, eo, es, ec)
    return eo, es, ec
