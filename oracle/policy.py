"""Oracle of the roofline CPU/GPU split policy -- TEST INFRASTRUCTURE ONLY.

A plain model, written from the paper and sharing nothing with the HIP
library's host code.  Only the test suite imports it.

What the paper fixes (Sec. 5.2, Eq. 1; Sec. 5.3, Eq. 2 and the text after it):
  * per decode step the CPU engine takes r*A*L + C_cpu and the GPU engine
    (1-r)*B*L + C_gpu, with A and B per-token costs, L the placed length and
    r the CPU share; the step waits for the slower of the two;
  * the balancing share is r(L) = clamp(B/(A+B) + (C_gpu - C_cpu)/((A+B) L), 0, 1);
  * decode evictions are routed batch by batch so that the running fraction
    of CPU-placed batches follows the marginal share p = B/(A+B); starting
    from a share R0 at length L0, the cumulative share is then
    R(L) = p + (R0 - p) L0 / L;
  * A is tracked online by back-computing it from a sliding average of the
    CPU component's per-step latency.

Readings where the paper leaves a choice:
  * batch routing: the next batch goes to the CPU iff that leaves the running
    CPU fraction strictly closer to p than sending it to the GPU, i.e. iff
    c + 1/2 < p (k + 1) after k batches of which c went to the CPU;
  * the A estimate over a window of w steps (t_i, n_i) -- measured CPU
    latency and CPU-side token count -- is (sum t_i - w C_cpu) / sum n_i;
    with no CPU tokens in the window, or a non-positive result, the previous
    estimate is kept.
"""
from __future__ import annotations

from collections import deque


def latency(r: float, L: float, A: float, B: float, c_cpu: float, c_gpu: float):
    """Eq. 1: (T_cpu, T_gpu) of one decode step at CPU share r and length L."""
    return r * A * L + c_cpu, (1.0 - r) * B * L + c_gpu


def share(L: float, A: float, B: float, c_cpu: float, c_gpu: float) -> float:
    """Eq. 2: the CPU share that equalises the two engines' latencies, clamped to [0, 1]."""
    delta = c_gpu - c_cpu
    x = B / (A + B) + delta / ((A + B) * L)
    return min(1.0, max(0.0, x))


def marginal_share(A: float, B: float) -> float:
    """The converged value of Eq. 2 (L -> infinity): p = B / (A + B)."""
    return B / (A + B)


def cumulative_share(L: float, L0: float, R0: float, p: float) -> float:
    """R(L) = p + (R0 - p) L0 / L (Sec. 5.3)."""
    return p + (R0 - p) * L0 / L


class BatchRouter:
    """Destination of successive eviction batches (reading above)."""

    def __init__(self):
        self.k = 0      # batches routed
        self.c = 0      # of which to the CPU

    def route(self, p: float) -> int:
        """0 = CPU, 1 = GPU."""
        to_cpu = self.c + 0.5 < p * (self.k + 1)
        self.k += 1
        if to_cpu:
            self.c += 1
            return 0
        return 1


class AEstimator:
    """Sliding-window estimate of the CPU per-token cost A (reading above)."""

    def __init__(self, A0: float, c_cpu: float, window: int):
        self.A = A0
        self.c_cpu = c_cpu
        self.samples = deque(maxlen=window)

    def observe(self, t_cpu: float, n_cpu: int) -> float:
        self.samples.append((t_cpu, n_cpu))
        st = 0.0
        sn = 0
        for t, n in self.samples:
            st += t
            sn += n
        if sn > 0:
            a = (st - len(self.samples) * self.c_cpu) / sn
            if a > 0.0:
                self.A = a
        return self.A
