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
                 block_tokens: int = 64, splits: Optional[Sequence[int]] = None, pool_slack: int = 0,
                 load_ends: Optional[Sequence[int]] = None, evict_tokens: int = 0, pingpong_blocks: int = 0,
                 arena_blocks: int = 0):
        """load_ends: per sequence, the end of its load-region range [s, load_end)
        (default: no load range); evict_tokens: the eviction batch D, which
        also sizes the CPU and load pools for every batch the extra tokens can
        evict."""
        self.w = w
        self.device = device
        self.dev = torch.device("cuda", device)
        self.B = len(prefill.lengths)
        extra = w.steps if extra_tokens is None else extra_tokens
        self.splits = list(prefill.splits if splits is None else splits)
        self.load_ends = list(self.splits if load_ends is None else load_ends)
        bk = block_tokens
        Ls = prefill.lengths
        evict_blocks = _cdiv(extra, bk) + 1 if evict_tokens else 0
        dev_blocks = sum(_cdiv(L + extra, bk) - min(e, L + extra) // bk
                         for L, e in zip(Ls, self.load_ends)) + pool_slack
        host_blocks = sum(_cdiv(min(s, L), bk) + evict_blocks for L, s in zip(Ls, self.splits)) + pool_slack
        load_blocks = sum((_cdiv(e, bk) - s // bk if e > s else 0) + evict_blocks
                          for s, e in zip(self.splits, self.load_ends)) if load_ends is not None else 0
        if load_blocks:
            load_blocks += pool_slack
            arena_blocks = arena_blocks or max(1, min(load_blocks, 1024))
            pingpong_blocks = pingpong_blocks or 512
        else:
            arena_blocks = pingpong_blocks = 0
        self.max_len = max(max(Ls) + extra, max(self.load_ends))
        common = dict(evict_tokens=evict_tokens, load_pool_blocks=load_blocks, load_arena_blocks=arena_blocks,
                      pingpong_blocks=pingpong_blocks)
        if w.kind == MLA:
            spec = wsk.make_spec(wsk.KIND_MLA, w.n_q_heads, 1, w.head_dim, bk, self.B, self.max_len, dev_blocks,
                                 host_blocks, w.softmax_scale, latent_dim=w.latent_dim, rope_dim=w.rope_dim,
                                 **common)
        else:
            spec = wsk.make_spec(wsk.KIND_GQA, w.n_q_heads, w.n_kv_heads, w.head_dim, bk, self.B, self.max_len,
                                 dev_blocks, host_blocks, w.softmax_scale, **common)
        self.spec = spec
        torch.cuda.set_device(device)
        self.h = wsk.wsk_init(spec, device)
        self.lengths = list(Ls)
        for b in range(self.B):
            wsk.wsk_seq_open_window(self.h, b, self.splits[b], self.load_ends[b])
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
        """The D-window [w, L): the GPU-pool range of sequence b."""
        segs = wsk.wsk_seq_segments(self.h, b)
        w = segs[-1][0] if segs and segs[-1][2] == wsk.PART_GPU else self.lengths[b]
        return w, self.lengths[b]

    def attend_gpu(self, q: torch.Tensor, ids: Optional[List[int]] = None, o_x=None, lse_x=None, o=None, lse=None):
        """Every GPU-side position (D-window in place, load region streamed), merged
        with (o_x, lse_x) when given."""
        ids = self.ids if ids is None else ids
        o, lse = self._outputs(len(ids), o, lse)
        need = wsk.wsk_attend_gpu_workspace(self.h, ids)
        if self._ws.numel() < need:
            self._ws = torch.empty(need + 4096, dtype=torch.uint8, device=self.dev)
        wsk.wsk_attend_gpu(self.h, ids, q, o, lse, self._ws, o_x, lse_x)
        return o, lse

    def decode_step(self, q: torch.Tensor, k_new: torch.Tensor, v_new: Optional[torch.Tensor], o_x=None, lse_x=None,
                    o=None, lse=None, ids: Optional[List[int]] = None):
        """Append + attend every GPU-side position (the new row included) + merge,
        in one call (wsk_decode_step); the workspace keeps room for one more
        chunk partial per sequence, so that steps do not allocate."""
        ids = self.ids if ids is None else ids
        o, lse = self._outputs(len(ids), o, lse)
        need = wsk.wsk_decode_step_workspace(self.h, ids)
        if self._ws.numel() < need:
            spare = len(ids) * self.w.n_q_heads * (self.out_width + 1) * 4 + 512
            self._ws = torch.empty(need + spare, dtype=torch.uint8, device=self.dev)
        wsk.wsk_decode_step(self.h, ids, q, k_new, v_new, o, lse, self._ws, o_x, lse_x)
        for b in ids:
            self.lengths[b] += 1
        return o, lse

    def decode_step_mla(self, q: torch.Tensor, k_new: torch.Tensor, w_uv: torch.Tensor, o: torch.Tensor,
                        lse: torch.Tensor, o_lat=None, o_x=None, lse_x=None, ids: Optional[List[int]] = None):
        """MLA decode step with the output expansion folded into its pass 2
        (wsk_decode_step_mla): o [n, H, dv] = W_UV[h]^T O_lat; o_lat, when
        given, receives the merged latent output."""
        ids = self.ids if ids is None else ids
        need = wsk.wsk_decode_step_workspace(self.h, ids)
        if self._ws.numel() < need:
            spare = len(ids) * self.w.n_q_heads * (self.out_width + 1) * 4 + 512
            self._ws = torch.empty(need + spare, dtype=torch.uint8, device=self.dev)
        wsk.wsk_decode_step_mla(self.h, ids, q, k_new, w_uv, o, lse, self._ws, o_lat=o_lat, o_x=o_x, lse_x=lse_x)
        for b in ids:
            self.lengths[b] += 1
        return o, lse

    def attend_gpu_pass1(self, q: torch.Tensor, ids: Optional[List[int]] = None):
        """Pass 1 of attend_gpu (transfers and kernels enqueued, partials in the
        session workspace); attend_gpu_pass2 with the same ids completes it."""
        ids = self.ids if ids is None else ids
        need = wsk.wsk_attend_gpu_workspace(self.h, ids)
        if self._ws.numel() < need:
            self._ws = torch.empty(need + 4096, dtype=torch.uint8, device=self.dev)
        wsk.wsk_attend_gpu_pass1(self.h, ids, q, self._ws)

    def attend_gpu_pass2(self, ids: Optional[List[int]] = None, o_x=None, lse_x=None, o=None, lse=None):
        ids = self.ids if ids is None else ids
        o, lse = self._outputs(len(ids), o, lse)
        wsk.wsk_attend_gpu_pass2(self.h, ids, o, lse, self._ws, o_x, lse_x)
        return o, lse

    def flush(self, parts: Sequence[int], ids: Optional[List[int]] = None):
        ids = self.ids if ids is None else ids
        return wsk.wsk_flush(self.h, ids, parts)

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
