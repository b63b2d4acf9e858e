"""Oracle of write-time partition routing -- TEST INFRASTRUCTURE ONLY.

A plain model of where each cached token lives, written from the paper and
sharing nothing with the HIP library's host code.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg import it.

What the paper fixes (Sec. 3 "write-time principle"; Sec. 4.1 "The Format Is
the Partition"; Sec. 4.2; Sec. 4.3 semantics (i)-(iii); Sec. 5.1):
  * every byte gets exactly one final physical residency, chosen when it is
    written, and placed data never moves afterwards;
  * each region is made of fixed-size blocks, the one granularity for routing;
  * the CPU takes one sequence range and the GPU the adjacent one, the GPU's
    share including the newest (decode-time) entries;
  * blocks are reclaimed in place when a session ends.

Readings where the paper is silent:
  * the CPU partition is the prefix [0, s) and the GPU partition is [s, L);
    position p routes to the CPU iff p < s, and s is fixed per sequence;
  * with a load range (the paper's pinned load region, Sec. 4.2), positions
    [s, load_end) route to the load region and p >= load_end to the GPU pool
    (the D-window); load_end is fixed per sequence and block-aligned;
  * an eviction ("flush", Sec. 4.2) moves the whole batch [w, w') of the
    D-window, w' = floor((w + D) / Bk) * Bk, to the CPU partition or the load
    region when w' <= L; the batch's blocks take slots in the destination
    (lowest free first, sequences in ascending id whatever order the call
    lists them in, blocks ascending -- the order an append uses; a block
    that already has a slot there keeps it), their GPU-pool slots are freed,
    and those positions live in the destination from then on;
  * blocks sit on an absolute grid: logical block k covers [k*Bk, (k+1)*Bk);
    a block straddling s has a slot in both pools, each holding only the
    positions of its own side;
  * a slot is taken when its (pool, sequence, logical block) is first touched,
    lowest free slot first; positions are touched in call order, sequences of
    one multi-sequence call in ascending id, positions of one sequence in
    ascending order;
  * a call that cannot get every slot it needs fails and changes nothing;
  * closing a sequence returns all its slots to the free sets.
"""
from __future__ import annotations

import heapq
from typing import Dict, List, Tuple

CPU = 0
GPU = 1
LOAD = 2


class RouteError(Exception):
    """A refused operation; ``code`` is one of EINVAL, ENOMEM, ERANGE, ESTATE."""

    def __init__(self, code: str, msg: str):
        super().__init__("%s: %s" % (code, msg))
        self.code = code


class RouteModel:
    def __init__(self, block_tokens: int, host_blocks: int, device_blocks: int, load_blocks: int = 0,
                 evict_tokens: int = 0):
        self.bk = block_tokens
        self.evict = evict_tokens
        self.capacity = {CPU: host_blocks, GPU: device_blocks, LOAD: load_blocks}
        # free slots of each pool as a min-heap: the lowest free slot is on top
        self.free = {CPU: list(range(host_blocks)), GPU: list(range(device_blocks)), LOAD: list(range(load_blocks))}
        self.split: Dict[int, int] = {}
        self.load_end: Dict[int, int] = {}
        self.window: Dict[int, int] = {}
        self.length: Dict[int, int] = {}
        self.homes: Dict[int, List[int]] = {}     # home of every written position
        # (part, seq, logical block) -> slot
        self.slot: Dict[Tuple[int, int, int], int] = {}

    def _home_at_write(self, seq: int, p: int) -> int:
        if p < self.split[seq]:
            return CPU
        return LOAD if p < self.load_end[seq] else GPU

    # -- allocation -------------------------------------------------------
    def _plan(self, seq: int, pos0: int, n: int, pending: Dict):
        """Take slots for positions [pos0, pos0+n) of seq, touching them in order.
        The first position of each new (partition, block) takes the lowest free slot."""
        for p in range(pos0, pos0 + n):
            part = self._home_at_write(seq, p)
            key = (part, seq, p // self.bk)
            if key in self.slot or key in pending:
                continue
            if not self.free[part]:
                raise RouteError("ENOMEM", "pool exhausted")
            pending[key] = heapq.heappop(self.free[part])

    def _undo(self, pending: Dict):
        for (part, _, _), slot in pending.items():
            heapq.heappush(self.free[part], slot)

    def _commit(self, pending: Dict):
        self.slot.update(pending)

    # -- operations -----------------------------------------------------------
    def open(self, seq: int, split: int, load_end: int = None):
        load_end = split if load_end is None else load_end
        if split < 0 or load_end < split:
            raise RouteError("EINVAL", "bad split or load_end")
        if load_end > split:
            if self.capacity[LOAD] == 0:
                raise RouteError("ESTATE", "no load region")
            if load_end % self.bk:
                raise RouteError("EINVAL", "load_end not block-aligned")
        if seq in self.split:
            raise RouteError("ESTATE", "already open")
        self.split[seq] = split
        self.load_end[seq] = load_end
        self.window[seq] = load_end
        self.length[seq] = 0
        self.homes[seq] = []

    def write(self, seq: int, pos0: int, n: int):
        """Bulk write of n positions at the tail of seq (prefill routing)."""
        if seq not in self.split:
            raise RouteError("ESTATE", "not open")
        if n < 0:
            raise RouteError("EINVAL", "negative count")
        if pos0 != self.length[seq]:
            raise RouteError("ERANGE", "not at tail")
        pending = {}
        try:
            self._plan(seq, pos0, n, pending)
        except RouteError:
            self._undo(pending)
            raise
        self._commit(pending)
        self.homes[seq].extend(self._home_at_write(seq, p) for p in range(pos0, pos0 + n))
        self.length[seq] += n

    def flush(self, seqs: List[int], parts: List[int]) -> List[int]:
        """Evict one D-batch of each listed sequence's D-window; returns the positions moved."""
        if len(set(seqs)) != len(seqs):
            raise RouteError("EINVAL", "duplicate sequence")
        if self.evict <= 0:
            raise RouteError("ESTATE", "no eviction batch")
        for sq, part in zip(seqs, parts):
            if sq not in self.split:
                raise RouteError("ESTATE", "not open")
            if part not in (CPU, LOAD):
                raise RouteError("EINVAL", "bad destination")
            if part == LOAD and self.capacity[LOAD] == 0:
                raise RouteError("ESTATE", "no load region")
        dest = dict(zip(seqs, parts))
        batch, pending = {}, {}
        try:
            for sq in sorted(seqs):          # slots are taken in ascending sequence id
                part = dest[sq]
                w = self.window[sq]
                w1 = (w + self.evict) // self.bk * self.bk
                if w1 > self.length[sq]:
                    batch[sq] = None
                    continue
                batch[sq] = (w, w1)
                for blk in range(w // self.bk, w1 // self.bk):
                    key = (part, sq, blk)
                    if key in self.slot or key in pending:
                        continue
                    if not self.free[part]:
                        raise RouteError("ENOMEM", "pool exhausted")
                    pending[key] = heapq.heappop(self.free[part])
        except RouteError:
            self._undo(pending)
            raise
        self._commit(pending)
        moved = []
        for sq, part in zip(seqs, parts):
            b = batch[sq]
            if b is None:
                moved.append(0)
                continue
            w, w1 = b
            for blk in range(w // self.bk, w1 // self.bk):
                heapq.heappush(self.free[GPU], self.slot.pop((GPU, sq, blk)))
            for p in range(w, w1):
                self.homes[sq][p] = part
            self.window[sq] = w1
            moved.append(w1 - w)
        return moved

    def append(self, seqs: List[int]):
        """One new position at the tail of every listed sequence (decode routing)."""
        if len(set(seqs)) != len(seqs):
            raise RouteError("EINVAL", "duplicate sequence")
        for sq in seqs:
            if sq not in self.split:
                raise RouteError("ESTATE", "not open")
        pending = {}
        try:
            for sq in sorted(seqs):
                self._plan(sq, self.length[sq], 1, pending)
        except RouteError:
            self._undo(pending)
            raise
        self._commit(pending)
        for sq in seqs:
            self.homes[sq].append(self._home_at_write(sq, self.length[sq]))
            self.length[sq] += 1

    def close(self, seq: int):
        if seq not in self.split:
            raise RouteError("ESTATE", "not open")
        for key in [k for k in self.slot if k[1] == seq]:
            heapq.heappush(self.free[key[0]], self.slot.pop(key))
        for d in (self.split, self.load_end, self.window, self.length, self.homes):
            del d[seq]

    def route(self, seq: int, pos: int) -> Tuple[int, int, int, int]:
        """(part, logical block, slot, offset) of a written position."""
        if seq not in self.split or not (0 <= pos < self.length[seq]):
            raise RouteError("ERANGE", "out of range")
        part = self.homes[seq][pos]
        blk = pos // self.bk
        return part, blk, self.slot[(part, seq, blk)], pos % self.bk

    def table(self, part: int, seq: int, n_blocks: int) -> List[int]:
        """Row of the block table of one partition: slot per logical block, -1 if absent."""
        return [self.slot.get((part, seq, k), -1) for k in range(n_blocks)]
