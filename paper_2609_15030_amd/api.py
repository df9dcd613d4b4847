"""Torch-facing helpers over the C ABI: move inputs to the device, allocate
outputs, checkpoint rows and workspace, and call the entry points.

Allocation and marshalling only; all computation happens in liblinattn.so.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np
import torch

from . import linattn as la
from .workloads import BF16, Inputs


@dataclasses.dataclass
class DeviceInputs:
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    g: torch.Tensor
    beta: torch.Tensor
    cu_dev: torch.Tensor
    cu_host: np.ndarray
    io_dtype: int

    @property
    def n_seqs(self) -> int:
        return len(self.cu_host) - 1

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
        return int(self.cu_host[-1])


def torch_dtype(io_dtype: int):
    return torch.bfloat16 if io_dtype == la.LA_BF16 else torch.float32


def to_device(x: Inputs, device="cuda") -> DeviceInputs:
    """Exact conversion: the arrays already hold values of the storage dtype."""
    io = la.LA_BF16 if x.io_dtype == BF16 else la.LA_F32
    td = torch_dtype(io)

    def dev(a, dt):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt).contiguous()

    cu = np.ascontiguousarray(x.cu_seqlens, dtype=np.int32)
    return DeviceInputs(dev(x.q, td), dev(x.k, td), dev(x.v, td), dev(x.g, torch.float32),
                        dev(x.beta, torch.float32), dev(cu, torch.int32), cu, io)


def checkpoint_rows(lengths: Sequence[int], starts: Optional[Sequence[int]], interval: int):
    """Row offsets for the checkpoints of each sequence and the total, as the
    library numbers them (la_checkpoint_rows)."""
    cu = np.concatenate([[0], np.cumsum(np.asarray(lengths, np.int64))]).astype(np.int32)
    return la.la_checkpoint_rows(cu, None if starts is None else np.asarray(starts, np.int64), interval)


@dataclasses.dataclass
class PrefillResult:
    o: torch.Tensor
    final_state: torch.Tensor
    ckpt: Optional[torch.Tensor]
    ckpt_offsets: np.ndarray
    n_ckpt_rows: int


class Prefill:
    """Reusable buffers for repeated prefill calls of one shape."""

    def __init__(self, x: DeviceInputs, interval: int, variant: int = la.LA_GDR_LITERAL,
                 scale: float = 1.0, starts: Optional[Sequence[int]] = None,
                 emit_ckpt: bool = True):
        self.x = x
        self.shape = la.make_shape(x.n_seqs, x.n_heads, x.dk, x.dv, interval, x.io_dtype,
                                   variant, scale)
        dev = x.q.device
        lens = np.diff(x.cu_host).tolist()
        self.starts = None if starts is None else np.asarray(starts, np.int64)
        self.ckpt_offsets, self.n_ckpt_rows = checkpoint_rows(lens, starts, interval)
        self.ckpt_off_dev = torch.from_numpy(self.ckpt_offsets).to(dev)
        self.start_dev = None if starts is None else torch.from_numpy(self.starts).to(dev)
        self.o = torch.empty((x.total_tokens, x.n_heads, x.dv), dtype=x.q.dtype, device=dev)
        self.final = torch.empty((x.n_seqs, x.n_heads, x.dk, x.dv), dtype=torch.float32, device=dev)
        self.ckpt = None
        if emit_ckpt and self.n_ckpt_rows > 0:
            self.ckpt = torch.empty((self.n_ckpt_rows, x.n_heads, x.dk, x.dv), dtype=torch.float32,
                                    device=dev)
        nbytes = la.la_prefill_workspace_bytes(self.shape, x.total_tokens)
        assert nbytes > 0
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)

    def run(self, state_in: Optional[torch.Tensor] = None, stream=None) -> PrefillResult:
        """la_prefill (cold) or la_prefill_resume (with start positions)."""
        x = self.x
        ck = self.ckpt
        if self.starts is None:
            la.la_prefill(self.shape, x.q, x.k, x.v, x.g, x.beta, x.cu_dev, x.cu_host, self.o,
                          self.final, ck, self.ckpt_off_dev if ck is not None else None,
                          self.ckpt_offsets if ck is not None else None, self.workspace, stream)
        else:
            assert state_in is not None
            la.la_prefill_resume(self.shape, x.q, x.k, x.v, x.g, x.beta, x.cu_dev, x.cu_host,
                                 self.start_dev, self.starts, state_in, self.o, self.final, ck,
                                 self.ckpt_off_dev if ck is not None else None,
                                 self.ckpt_offsets if ck is not None else None, self.workspace,
                                 stream)
        return PrefillResult(self.o, self.final, ck, self.ckpt_offsets, self.n_ckpt_rows)


    def run_paged(self, pool: torch.Tensor, ckpt_page_ids: Optional[torch.Tensor] = None,
                  state_page_ids: Optional[torch.Tensor] = None, err_count: Optional[torch.Tensor] = None,
                  stream=None) -> PrefillResult:
        """la_prefill_paged: checkpoints to pool pages (rows numbered as
        ckpt_offsets), starting states from pool pages (a resume).  The
        result's ckpt is None: the checkpoints live in the pool."""
        x = self.x
        pages = la.make_pages(pool, ckpt_page_ids, state_page_ids, err_count)
        with_ck = ckpt_page_ids is not None
        la.la_prefill_paged(self.shape, pages, x.q, x.k, x.v, x.g, x.beta, x.cu_dev, x.cu_host, self.start_dev,
                            self.starts, self.o, self.final, self.ckpt_off_dev if with_ck else None,
                            self.ckpt_offsets if with_ck else None, self.workspace, stream)
        return PrefillResult(self.o, self.final, None, self.ckpt_offsets, self.n_ckpt_rows)


def prefill(x: DeviceInputs, interval: int, variant: int = la.LA_GDR_LITERAL, scale: float = 1.0,
            emit_ckpt: bool = True) -> PrefillResult:
    return Prefill(x, interval, variant, scale, None, emit_ckpt).run()


def prefill_resume(x: DeviceInputs, starts: Sequence[int], state_in: torch.Tensor, interval: int,
                   variant: int = la.LA_GDR_LITERAL, scale: float = 1.0,
                   emit_ckpt: bool = True) -> PrefillResult:
    return Prefill(x, interval, variant, scale, starts, emit_ckpt).run(state_in)
