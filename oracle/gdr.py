"""ctypes front end of the fp64 token-by-token oracle (``gdr_oracle.c``).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The recurrence, the output read-out and the checkpoint rule are documented in
``gdr_oracle.c``; this file only marshals NumPy arrays and builds the C file
with gcc when the shared object is missing or older than its source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gdr_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

LITERAL = 0
DECAYED_DELTA = 1


def oracle_library_path() -> str:
    return _LIB


def build_oracle(force: bool = False) -> str:
    """Compile gdr_oracle.c with gcc (plain C, -O2, no BLAS)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-shared", "-fPIC", _SRC,
                        "-o", tmp, "-lm", "-lpthread"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def load_library(path: str):
    """Load an oracle shared object (the built one, or a test's variant of it)."""
    lib = ctypes.CDLL(path)
    f = lib.oracle_gdr_prefill
    P = ctypes.c_void_p
    f.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_int32, ctypes.c_double, P, P, P, P, P,
                  ctypes.c_int64, ctypes.c_int64, P, P, P, P,
                  ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
    f.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        _lib = load_library(build_oracle())
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def n_checkpoints(start: int, end: int, C: int) -> int:
    """Count of absolute multiples of C in (start, end]."""
    return 0 if C <= 0 else end // C - start // C


def gdr_prefill_seq(q, k, v, g, beta, *, start: int = 0, interval: int = 0,
                    state_in: Optional[np.ndarray] = None, variant: int = LITERAL,
                    scale: float = 1.0, want_o: bool = True, want_ckpt: bool = True,
                    n_threads: int = 0, return_threads: bool = False, lib=None):
    """One sequence: tokens at absolute positions [start, start + T).

    q, k: [T, H, dk]; v: [T, H, dv]; g, beta: [T, H] (any float dtype; read
    as float32, i.e. the stored values).  state_in: [H, dk, dv] (converted
    to fp64) or None for the zero state.

    Returns (o [T, H, dv] fp64 or None, final state [H, dk, dv] fp64,
    checkpoints [n_ckpt, H, dk, dv] fp64 or None) and, if asked, the
    number of threads used.
    """
    q, k, v, g, beta = map(_f32, (q, k, v, g, beta))
    T, H, dk = q.shape
    dv = v.shape[2]
    assert k.shape == (T, H, dk) and v.shape[:2] == (T, H)
    assert g.shape == (T, H) and beta.shape == (T, H)
    s_in = None
    if state_in is not None:
        s_in = np.ascontiguousarray(state_in, dtype=np.float64)
        assert s_in.shape == (H, dk, dv)
    o = np.empty((T, H, dv), np.float64) if want_o else None
    st = np.empty((H, dk, dv), np.float64)
    nck = n_checkpoints(start, start + T, interval)
    ck = np.empty((nck, H, dk, dv), np.float64) if (want_ckpt and nck > 0) else None
    used = ctypes.c_int32(0)
    rc = (lib or _load()).oracle_gdr_prefill(T, H, dk, dv, variant, float(scale),
                                    _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                    int(start), int(interval), _ptr(s_in),
                                    _ptr(o), _ptr(st), _ptr(ck),
                                    int(n_threads), ctypes.byref(used))
    if rc != 0:
        raise RuntimeError(f"oracle_gdr_prefill failed with {rc}")
    if return_threads:
        return o, st, ck, used.value
    return o, st, ck


def gdr_prefill(inputs, *, starts: Optional[Sequence[int]] = None, interval: int = 0,
                states_in: Optional[np.ndarray] = None, variant: int = LITERAL,
                scale: float = 1.0, n_threads: int = 0):
    """Packed varlen front end over ``gdr_prefill_seq``.

    ``inputs`` follows ``paper_2609_15030_amd.workloads.Inputs``: the tokens of
    sequence i are rows cu_seqlens[i]:cu_seqlens[i+1], at absolute positions
    starts[i] + (0, 1, ...).  states_in: [n_seqs, H, dk, dv] or None.

    Returns (o [T_total, H, dv], final states [n_seqs, H, dk, dv],
    list of per-sequence checkpoint arrays (or None)).
    """
    cu = np.asarray(inputs.cu_seqlens)
    n = len(cu) - 1
    starts = [0] * n if starts is None else list(starts)
    T, H, dv = inputs.total_tokens, inputs.n_heads, inputs.dv
    o = np.empty((T, H, dv), np.float64)
    finals = np.empty((n, H, inputs.dk, dv), np.float64)
    ckpts = []
    for i in range(n):
        a, b = int(cu[i]), int(cu[i + 1])
        oi, si, ci = gdr_prefill_seq(
            inputs.q[a:b], inputs.k[a:b], inputs.v[a:b], inputs.g[a:b], inputs.beta[a:b],
            start=starts[i], interval=interval,
            state_in=None if states_in is None else states_in[i],
            variant=variant, scale=scale, n_threads=n_threads)
        o[a:b] = oi
        finals[i] = si
        ckpts.append(ci)
    return o, finals, ckpts
