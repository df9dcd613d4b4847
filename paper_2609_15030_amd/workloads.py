"""Seeded synthetic inputs for the strict-prefix linear-attention prefill.

This module only draws random numbers and packs them into arrays.  It holds
none of the method's arithmetic (no recurrence, no boundary rule, no paging):
both the fp64 oracle and the GPU path read the same arrays from here, and
nothing else is shared between them.

Recipe (one call per workload, every draw from NumPy's PCG64):

* q, k ~ N(0, 1), each (token, head) row L2-normalised in fp64; v ~ N(0, 1);
  beta = sigmoid(N(0, 1)); g = -softplus(N(0, 1)).  This is the distribution
  the gated delta rule workloads are specified with.
* Storage rounding: fp64 -> fp32 (round to nearest even), and for bf16
  workloads fp32 -> bf16 (round to nearest even).  The stored values are the
  ground truth for both paths; arrays are returned as float32 holding exactly
  representable values of the storage dtype.  g and beta are always fp32.
* Draw order: q, k, v, beta logits, g logits; then (varlen workload only)
  lengths, restore modes, kept-checkpoint counts and the page permutation
  from a spawned child generator.
* Seeds: ``SeedSequence(i)`` for workload i; the nine-length sweep spawns
  nine children of ``SeedSequence(2)``.

The paper itself prints no tensor data: its prompts are synthetic templates
fed to a real model (the paper's evaluation section).  These random tensors
stand in for one tensor-parallel rank's linear-attention inputs at the
prompt lengths the paper studies (3,584 tokens, the nine boundary lengths,
the 32,768-token maximum model length).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round a finite array to bf16 (nearest even) and return it as float32.

    Works on the fp32 bit pattern: add 0x7FFF plus the lowest kept bit, then
    clear the 16 dropped bits (no overflow for finite values)."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    lsb = (u >> 16) & 1
    u += np.uint32(0x7FFF)
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of a float32 array that already holds bf16 values."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    return (x32.view(np.uint32) >> 16).astype(np.uint16)


def _store(x: np.ndarray, io_dtype: str) -> np.ndarray:
    x32 = x.astype(np.float32)
    return round_to_bf16(x32) if io_dtype == BF16 else x32


@dataclasses.dataclass
class Inputs:
    """Packed varlen inputs: tokens of all sequences concatenated.

    q, k: [T_total, H, dk]; v: [T_total, H, dv]; g, beta: [T_total, H].
    cu_seqlens: int32 [n_seqs + 1] prefix offsets into the token axis.
    """
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray
    cu_seqlens: np.ndarray
    io_dtype: str

    @property
    def n_heads(self) -> int:
        return self.q.shape[1]

    @property
    def dk(self) -> int:
        return self.q.shape[2]

    @property
    def dv(self) -> int:
        return self.v.shape[2]

    @property
    def total_tokens(self) -> int:
        return self.q.shape[0]

    @property
    def n_seqs(self) -> int:
        return len(self.cu_seqlens) - 1

    def seq(self, i: int) -> "Inputs":
        a, b = int(self.cu_seqlens[i]), int(self.cu_seqlens[i + 1])
        return Inputs(self.q[a:b], self.k[a:b], self.v[a:b], self.g[a:b],
                      self.beta[a:b], np.array([0, b - a], np.int32),
                      self.io_dtype)

    def tokens(self, a: int, b: int) -> "Inputs":
        """Tokens [a, b) of a single-sequence input, as a new one-sequence input."""
        assert self.n_seqs == 1
        return Inputs(self.q[a:b], self.k[a:b], self.v[a:b], self.g[a:b],
                      self.beta[a:b], np.array([0, b - a], np.int32),
                      self.io_dtype)

    def heads(self, hs) -> "Inputs":
        hs = list(hs)
        return Inputs(np.ascontiguousarray(self.q[:, hs]),
                      np.ascontiguousarray(self.k[:, hs]),
                      np.ascontiguousarray(self.v[:, hs]),
                      np.ascontiguousarray(self.g[:, hs]),
                      np.ascontiguousarray(self.beta[:, hs]),
                      self.cu_seqlens.copy(), self.io_dtype)


def _normals(rng, shape, io_dtype, unit_rows):
    """N(0,1) draws in fp64, optionally L2-normalised per last-axis row, then
    rounded to the storage dtype.  Drawn in blocks of rows (the block size
    does not change the values: PCG64 fills arrays in C order)."""
    T = shape[0]
    out = np.empty(shape, np.float32)
    step = max(1, (1 << 22) // int(np.prod(shape[1:])))
    for a in range(0, T, step):
        b = min(T, a + step)
        x = rng.standard_normal((b - a,) + tuple(shape[1:]))
        if unit_rows:
            x /= np.linalg.norm(x, axis=-1, keepdims=True)
        out[a:b] = _store(x, io_dtype)
    return out


def draw(rng: np.random.Generator, seqlens, n_heads: int, dk: int, dv: int,
         io_dtype: str, gate_scale: float = 1.0) -> Inputs:
    """Draw one packed input with the distributions stated in the module doc.

    ``gate_scale`` multiplies the log-decay (g = -softplus(N(0, 1)) * scale,
    in fp64 before rounding): 1 is the specified distribution, whose state
    forgets everything older than a chunk (mean g = -0.81 per token); small
    scales give long-memory inputs whose state is carried across many chunks."""
    seqlens = [int(n) for n in seqlens]
    T = int(sum(seqlens))
    q = _normals(rng, (T, n_heads, dk), io_dtype, True)
    k = _normals(rng, (T, n_heads, dk), io_dtype, True)
    v = _normals(rng, (T, n_heads, dv), io_dtype, False)
    b_logit = rng.standard_normal((T, n_heads))
    g_logit = rng.standard_normal((T, n_heads))
    beta = (1.0 / (1.0 + np.exp(-b_logit))).astype(np.float32)
    g = (-np.logaddexp(0.0, g_logit) * gate_scale).astype(np.float32)
    cu = np.zeros(len(seqlens) + 1, np.int32)
    cu[1:] = np.cumsum(seqlens)
    return Inputs(q, k, v, g, beta, cu, io_dtype)


def random_inputs(seed: int, seqlens, n_heads: int, dk: int, dv: int,
                  io_dtype: str = BF16, gate_scale: float = 1.0) -> Inputs:
    """Inputs for ad-hoc test shapes (edge cases, ragged tails, long memory)."""
    return draw(np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed))),
                seqlens, n_heads, dk, dv, io_dtype, gate_scale)


@dataclasses.dataclass
class Workload:
    """One named workload: inputs plus its checkpoint/cache parameters.

    ``interval`` is the cache-block (checkpoint) size C.  ``available`` is,
    per sequence, the length of the contiguous cached prefix the lookup may
    use (tokens); ``page_perm`` and ``pool_pages`` describe the paged state
    pool where that workload has one.
    """
    name: str
    inputs: Inputs
    interval: int
    chunk: int = 64
    available: Optional[List[int]] = None
    modes: Optional[List[str]] = None
    kept: Optional[List[int]] = None
    page_perm: Optional[np.ndarray] = None
    pool_pages: int = 0
    max_ckpt_per_seq: int = 0


def _gen(seed_seq: np.random.SeedSequence) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_seq))


def tiny_fp32() -> Workload:
    """1 head, dk = dv = 64, T = 256, fp32, C = 16 (full hit, restored at 240)."""
    rng = _gen(np.random.SeedSequence(0))
    x = draw(rng, [256], 1, 64, 64, F32)
    return Workload("tiny_fp32_T256_H1_d64_C16", x, interval=16,
                    available=[256], modes=["complete"])


def tp_rank_3584() -> Workload:
    """One TP rank's share: 8 heads, d = 128, T = 3,584, bf16, C = 256."""
    rng = _gen(np.random.SeedSequence(1))
    x = draw(rng, [3584], 8, 128, 128, BF16)
    return Workload("tp_rank_T3584_H8_d128_bf16_C256", x, interval=256,
                    available=[3584], modes=["complete"])


def nine_length_sweep() -> List[Workload]:
    """Nine serial runs T = 512 * i (i = 1..9), 8 heads, d = 128, bf16, C = 256."""
    children = np.random.SeedSequence(2).spawn(9)
    out = []
    for i, ss in enumerate(children):
        T = 512 * (i + 1)
        x = draw(_gen(ss), [T], 8, 128, 128, BF16)
        out.append(Workload(f"sweep_T{T}_H8_d128_bf16_C256", x, interval=256,
                            available=[T], modes=["complete"],
                            pool_pages=(T // 256) * 8))
    return out


def long_prefill(heads: Optional[int] = None) -> Workload:
    """16 heads, d = 128, T = 32,768, bf16, C = 1,024.

    ``heads`` keeps only the first ``heads`` heads of the same draw (the draw
    itself always covers all 16 heads, so values do not depend on it)."""
    rng = _gen(np.random.SeedSequence(3))
    x = draw(rng, [32768], 16, 128, 128, BF16)
    if heads is not None:
        x = x.heads(range(heads))
    return Workload("long_T32768_H16_d128_bf16_C1024", x, interval=1024,
                    available=[32768], modes=["complete"])


VARLEN_POOL_PAGES = 4096
VARLEN_CKPT_SLOTS = 32          # 8,192 / 256 checkpoint slots per sequence


def batched_varlen(with_data: bool = True) -> Workload:
    """16 sequences, lengths uniform in [1024, 8192] rounded down to 16,
    8 heads, d = 128, bf16, C = 256, with a 4,096-page pool addressed through
    a random permutation page table, and a per-sequence restore mode.

    ``with_data=False`` skips the tensor draw (inputs hold 0-token arrays but
    the true cu_seqlens); the metadata does not depend on it."""
    root = np.random.SeedSequence(4)
    data_ss, meta_ss = root.spawn(2)
    meta = _gen(meta_ss)
    n_seqs, C = 16, 256
    lens = (16 * (meta.integers(1024, 8193, size=n_seqs) // 16)).tolist()
    modes = [("cold", "complete", "partial")[int(m)]
             for m in meta.integers(0, 3, size=n_seqs)]
    kept = []
    for n, mode in zip(lens, modes):
        usable = (n - 1) // C          # checkpoints strictly inside the prompt
        kept.append(int(meta.integers(0, usable)) if mode == "partial" else
                    (usable if mode == "complete" else 0))
    perm = meta.permutation(VARLEN_POOL_PAGES).astype(np.int32)
    if with_data:
        x = draw(_gen(data_ss), lens, 8, 128, 128, BF16)
    else:
        x = draw(_gen(data_ss), [0], 8, 128, 128, BF16)
        x.cu_seqlens = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    available = [k * C if m != "complete" else n
                 for n, m, k in zip(lens, modes, kept)]
    return Workload("varlen16_H8_d128_bf16_C256", x, interval=C,
                    available=available, modes=modes, kept=kept,
                    page_perm=perm, pool_pages=VARLEN_POOL_PAGES,
                    max_ckpt_per_seq=VARLEN_CKPT_SLOTS)


def page_slot(seq: int, ckpt: int, head: int, n_heads: int = 8,
              slots: int = VARLEN_CKPT_SLOTS) -> int:
    """Index into the page permutation for (sequence, checkpoint, head)."""
    return (seq * slots + ckpt) * n_heads + head
