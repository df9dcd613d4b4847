"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of ``oracle/gdr_oracle.c`` (a flipped
sign, a dropped term, a transposed operand, swapped variants, a wrong
operand in the read-out, a mis-numbered checkpoint row), compiles it with
gcc on the CPU, and runs a small battery of the pin checks against it.  At
least one check must fail for every planted mistake, and all of them must
pass for the unmodified source.  Every planted mistake keeps all memory
accesses in bounds for the shapes used here (dk == dv).
"""
import functools
import os
import subprocess

import numpy as np
import pytest

from oracle.gdr import DECAYED_DELTA, LITERAL, _SRC, gdr_prefill_seq, load_library
from paper_2609_15030_amd import workloads as wl

from test_oracle_pins import unrolled_outputs

MUTATIONS = {
    "delta_sign": ("((double)vt[c] - pred[c])", "((double)vt[c] + pred[c])"),
    "dropped_beta": ("pred[c] = beta * (", "pred[c] = ("),
    "dropped_decay": ("Sr[c] = alpha * Sr[c] + kr * pred[c]", "Sr[c] = Sr[c] + kr * pred[c]"),
    "variants_swapped": ("if (j->variant == 1)", "if (j->variant == 0)"),
    "readout_uses_key": ("const double qr = (double)qt[r];", "const double qr = (double)kt[r];"),
    "transposed_prediction": ("pred[c] += Sr[c] * kr;", "pred[c] += S[(size_t)c * dv + r] * kr;"),
    "gate_sign": ("exp((double)j->g[", "exp(-(double)j->g["),
    "scale_dropped": ("ot[c] *= j->scale;", ";"),
    "checkpoint_rows_reversed": ("const int64_t row = len / j->C - j->start / j->C - 1;",
                                 "const int64_t row = (j->start + j->T) / j->C - len / j->C;"),
}


def _battery(run):
    """Returns the names of the pin checks that fail for ``run``."""
    failed = []
    d = 8
    for variant in (LITERAL, DECAYED_DELTA):
        x = wl.random_inputs(101 + variant, [24], 2, d, d, wl.F32)
        S0 = np.random.default_rng(variant).standard_normal((2, d, d))
        o, _, _ = run(x.q, x.k, x.v, x.g, x.beta, state_in=S0, variant=variant, scale=0.7)
        ref = unrolled_outputs(x.q, x.k, x.v, x.g, x.beta, variant, scale=0.7, S0=S0)
        if not np.allclose(o, ref, rtol=1e-10, atol=1e-10):
            failed.append(f"unrolling[{variant}]")
    # repeated key, literal: w_t = (a - b kk) w + b v
    rng = np.random.default_rng(7)
    kv = rng.standard_normal(d)
    kv /= np.linalg.norm(kv)
    T = 12
    k = np.tile(kv.astype(np.float32), (T, 1))[:, None, :]
    q = rng.standard_normal((T, 1, d)).astype(np.float32)
    v = rng.standard_normal((T, 1, d)).astype(np.float32)
    g = -rng.uniform(0, 1.5, (T, 1)).astype(np.float32)
    beta = rng.uniform(0, 1, (T, 1)).astype(np.float32)
    o, _, _ = run(q, k, v, g, beta, variant=LITERAL)
    kd = k[0, 0].astype(np.float64)
    kk = float(kd @ kd)
    w = np.zeros(d)
    for t in range(T):
        a, b = np.exp(float(g[t, 0])), float(beta[t, 0])
        w = (a - b * kk) * w + b * v[t, 0].astype(np.float64)
    if not np.allclose(o[-1, 0], w * float(kd @ q[-1, 0]), rtol=1e-9, atol=1e-12):
        failed.append("repeated_key")
    # checkpoint at P equals the final state of a run over [0, P)
    x = wl.random_inputs(103, [64], 1, d, d, wl.F32)
    _, _, ck = run(x.q, x.k, x.v, x.g, x.beta, interval=16)
    _, S16, _ = run(x.q[:16], x.k[:16], x.v[:16], x.g[:16], x.beta[:16])
    if not np.array_equal(ck[0], S16):
        failed.append("checkpoint_is_prefix_state")
    return failed


def _build_variant(tmp_path, name, old, new):
    src = open(_SRC).read()
    assert src.count(old) == 1, name
    path = os.path.join(tmp_path, f"mut_{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    so = os.path.join(tmp_path, f"mut_{name}.so")
    subprocess.run(["gcc", "-O1", "-shared", "-fPIC", path, "-o", so, "-lm", "-lpthread"],
                   check=True)
    return load_library(so)


def test_unmodified_oracle_passes_battery():
    assert _battery(gdr_prefill_seq) == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    lib = _build_variant(str(tmp_path), name, old, new)
    failed = _battery(functools.partial(gdr_prefill_seq, lib=lib))
    assert failed, f"mutation {name} passed every pin"
