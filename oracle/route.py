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


class RouteError(Exception):
    """A refused operation; ``code`` is one of EINVAL, ENOMEM, ERANGE, ESTATE."""

    def __init__(self, code: str, msg: str):
        super().__init__("%s: %s" % (code, msg))
        self.code = code


class RouteModel:
    def __init__(self, block_tokens: int, host_blocks: int, device_blocks: int):
        self.bk = block_tokens
        self.capacity = {CPU: host_blocks, GPU: device_blocks}
        # free slots of each pool as a min-heap: the lowest free slot is on top
        self.free = {CPU: list(range(host_blocks)), GPU: list(range(device_blocks))}
        self.split: Dict[int, int] = {}
        self.length: Dict[int, int] = {}
        # (part, seq, logical block) -> slot
        self.slot: Dict[Tuple[int, int, int], int] = {}

    # -- allocation -------------------------------------------------------
    def _plan(self, seq: int, pos0: int, n: int, pending: Dict):
        """Take slots for positions [pos0, pos0+n) of seq, touching them in order.
        The first position of each new (partition, block) takes the lowest free slot."""
        s = self.split[seq]
        for p in range(pos0, pos0 + n):
            part = CPU if p < s else GPU
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
    def open(self, seq: int, split: int):
        if seq in self.split:
            raise RouteError("ESTATE", "already open")
        if split < 0:
            raise RouteError("EINVAL", "bad split")
        self.split[seq] = split
        self.length[seq] = 0

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
        self.length[seq] += n

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
            self.length[sq] += 1

    def close(self, seq: int):
        if seq not in self.split:
            raise RouteError("ESTATE", "not open")
        for key in [k for k in self.slot if k[1] == seq]:
            heapq.heappush(self.free[key[0]], self.slot.pop(key))
        del self.split[seq]
        del self.length[seq]

    def route(self, seq: int, pos: int) -> Tuple[int, int, int, int]:
        """(part, logical block, slot, offset) of a written position."""
        if seq not in self.split or not (0 <= pos < self.length[seq]):
            raise RouteError("ERANGE", "out of range")
        part = CPU if pos < self.split[seq] else GPU
        blk = pos // self.bk
        return part, blk, self.slot[(part, seq, blk)], pos % self.bk

    def table(self, part: int, seq: int, n_blocks: int) -> List[int]:
        """Row of the block table of one partition: slot per logical block, -1 if absent."""
        return [self.slot.get((part, seq, k), -1) for k in range(n_blocks)]
