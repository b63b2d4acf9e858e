"""One-layer decode session on one GPU, driven through the C ABI.

A DecodeSession builds a partitioned cache sized for a workload, routes its
prefilled context once (bulk write: CPU prefix to the host pool, GPU suffix to
HBM), and then runs decode steps: append the new token's K/V into the GPU
partition, attend the GPU range, merge with a partial computed elsewhere for
the CPU range.  All device work runs in libwsk.so; torch only provides device
memory and the current stream.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import torch

from . import wsk
from .workloads import GQA, MLA, Prefill, Workload


def _cdiv(a: int, b: int) -> int:
    return -(-a // b)


class DecodeSession:
    def __init__(self, w: Workload, prefill: Prefill, device: int = 0, extra_tokens: Optional[int] = None,
                 block_tokens: int = 64, splits: Optional[Sequence[int]] = None, pool_slack: int = 0):
        self.w = w
        self.device = device
        self.dev = torch.device("cuda", device)
        self.B = len(prefill.lengths)
        extra = w.steps if extra_tokens is None else extra_tokens
        self.splits = list(prefill.splits if splits is None else splits)
        bk = block_tokens
        dev_blocks = sum(_cdiv(L + extra, bk) - min(s, L + extra) // bk
                         for L, s in zip(prefill.lengths, self.splits)) + pool_slack
        host_blocks = sum(_cdiv(min(s, L), bk) for L, s in zip(prefill.lengths, self.splits)) + pool_slack
        self.max_len = max(prefill.lengths) + extra
        if w.kind == MLA:
            spec = wsk.make_spec(wsk.KIND_MLA, w.n_q_heads, 1, w.head_dim, bk, self.B, self.max_len, dev_blocks,
                                 host_blocks, w.softmax_scale, latent_dim=w.latent_dim, rope_dim=w.rope_dim)
        else:
            spec = wsk.make_spec(wsk.KIND_GQA, w.n_q_heads, w.n_kv_heads, w.head_dim, bk, self.B, self.max_len,
                                 dev_blocks, host_blocks, w.softmax_scale)
        self.spec = spec
        torch.cuda.set_device(device)
        self.h = wsk.wsk_init(spec, device)
        self.lengths = list(prefill.lengths)
        for b in range(self.B):
            wsk.wsk_seq_open(self.h, b, self.splits[b])
            wsk.wsk_write(self.h, b, 0, prefill.k[b], None if prefill.v is None else prefill.v[b])
        self.ids = list(range(self.B))
        self._ws = torch.empty(0, dtype=torch.uint8, device=self.dev)

    # -- shapes -----------------------------------------------------------------
    @property
    def out_width(self) -> int:
        return self.w.latent_dim if self.w.kind == MLA else self.w.head_dim

    @property
    def q_width(self) -> int:
        return self.w.row_elems if self.w.kind == MLA else self.w.head_dim

    # -- operations ---------------------------------------------------------------
    def gpu_range(self, b: int):
        return min(self.splits[b], self.lengths[b]), self.lengths[b]

    def append(self, k_new: torch.Tensor, v_new: Optional[torch.Tensor], ids: Optional[List[int]] = None):
        ids = self.ids if ids is None else ids
        wsk.wsk_append(self.h, ids, k_new, v_new)
        for b in ids:
            self.lengths[b] += 1

    def workspace(self, ids, start, end) -> torch.Tensor:
        """Device workspace for an attend call; grown with room for one more chunk
        partial per sequence, so that decode steps that cross into a new chunk do
        not allocate."""
        need = wsk.wsk_attend_workspace(self.h, ids, start, end)
        if self._ws.numel() < need:
            spare = len(ids) * self.w.n_q_heads * (self.out_width + 1) * 4 + 512
            self._ws = torch.empty(need + spare, dtype=torch.uint8, device=self.dev)
        return self._ws

    def _ranges(self, start, end, ids):
        ids = self.ids if ids is None else ids
        if start is None:
            start = [self.gpu_range(b)[0] for b in ids]
        if end is None:
            end = [self.lengths[b] for b in ids]
        return ids, start, end

    def _outputs(self, n, o, lse):
        H = self.w.n_q_heads
        if o is None:
            o = torch.empty(n, H, self.out_width, dtype=torch.float32, device=self.dev)
        if lse is None:
            lse = torch.empty(n, H, dtype=torch.float32, device=self.dev)
        return o, lse

    def attend(self, q: torch.Tensor, start: Optional[Sequence[int]] = None, end: Optional[Sequence[int]] = None,
               ids: Optional[List[int]] = None, o: Optional[torch.Tensor] = None,
               lse: Optional[torch.Tensor] = None):
        ids, start, end = self._ranges(start, end, ids)
        o, lse = self._outputs(len(ids), o, lse)
        ws = self.workspace(ids, start, end)
        wsk.wsk_attend(self.h, ids, start, end, q, o, lse, ws)
        return o, lse

    def attend_pass1(self, q: torch.Tensor, start=None, end=None, ids=None):
        """Pass 1 only (chunk partials in the session workspace); attend_pass2 with
        the same ranges completes it."""
        ids, start, end = self._ranges(start, end, ids)
        wsk.wsk_attend_pass1(self.h, ids, start, end, q, self.workspace(ids, start, end))

    def attend_pass2(self, start=None, end=None, ids=None, o=None, lse=None, o_x=None, lse_x=None):
        """Pass 2; with (o_x, lse_x) the CPU-range partial is merged in as well."""
        ids, start, end = self._ranges(start, end, ids)
        o, lse = self._outputs(len(ids), o, lse)
        wsk.wsk_attend_pass2(self.h, ids, start, end, o, lse, self.workspace(ids, start, end), o_x, lse_x)
        return o, lse

    @staticmethod
    def merge(o_a, lse_a, o_b, lse_b, o_out=None, lse_out=None, o_bf16=None):
        o_out = torch.empty_like(o_b) if o_out is None else o_out
        lse_out = torch.empty_like(lse_b) if lse_out is None else lse_out
        wsk.wsk_merge(o_a, lse_a, o_b, lse_b, o_out, lse_out, o_bf16)
        return o_out, lse_out

    def close(self):
        if self.h:
            torch.cuda.synchronize(self.dev)
            wsk.wsk_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def to_device_bf16(bits: np.ndarray, device) -> torch.Tensor:
    """Raw bf16 bits (uint16) -> device bf16 tensor, same bytes."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(device)
