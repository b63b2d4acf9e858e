"""Helpers shared by the GPU tests: device readback, error metrics, printing."""
import ctypes
import sys

import numpy as np
import torch

_hip = None

# Tolerances of the decode outputs against the fp64 oracle (bf16 inputs, fp32
# accumulation): largest absolute error and the L1 ratio sum|x-r| / sum|r|.
# The L1 ratio is bounded over the whole output and, separately, over every
# output row (one query head of one sequence), so an error confined to one
# head cannot hide under the average of the others.
MAX_ABS = 1e-2
MEAN_REL = 1e-3
# Elementwise relative errors |x - r| / max(|r|, REL_FLOOR) are reported next
# to the L1 ratio (they blow up where |r| is near 0, so they are not bounded).
REL_FLOOR = 1e-6
# LSE is reported with the outputs; fp32 softmax statistics are good to ~1e-6
# relative on LSE values of order 10, so 1e-4 absolute leaves a wide margin.
LSE_ABS = 1e-4


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def d2h(ptr: int, nbytes: int) -> np.ndarray:
    """Copy nbytes of device memory at ptr to a host uint8 array (hipMemcpy)."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    out = np.empty(nbytes, np.uint8)
    torch.cuda.synchronize()
    rc = _hip.hipMemcpy(out.ctypes.data, ptr, nbytes, 2)   # hipMemcpyDeviceToHost
    assert rc == 0, rc
    return out


def errors(x: np.ndarray, ref: np.ndarray):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    d = np.abs(x - ref)
    return float(d.max()), float(d.sum() / max(np.abs(ref).sum(), 1e-300))


def row_l1_ratios(x, ref) -> np.ndarray:
    """L1 ratio of every output row (the last axis is the output width); rows
    whose reference is all zero (an empty range) are left out."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    w = ref.shape[-1] if ref.ndim else 1
    d = np.abs(x - ref).reshape(-1, w).sum(axis=1)
    r = np.abs(ref).reshape(-1, w).sum(axis=1)
    keep = r > 0
    return d[keep] / r[keep]


def elementwise_rel(x, ref):
    """Mean and largest |x - r| / max(|r|, REL_FLOOR)."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    e = np.abs(x - ref) / np.maximum(np.abs(ref), REL_FLOOR)
    return float(e.mean()), float(e.max())


def assert_close(x, ref, what: str):
    ma, mr = errors(x, ref)
    rows = row_l1_ratios(x, ref)
    worst = float(rows.max()) if rows.size else 0.0
    em, ex = elementwise_rel(x, ref)
    say("  %-28s max_abs %.3e  mean_rel %.3e  worst row %.3e  elementwise rel mean %.3e max %.3e"
        % (what, ma, mr, worst, em, ex))
    assert np.all(np.isfinite(x)), what
    assert ma <= MAX_ABS and mr <= MEAN_REL, (what, ma, mr)
    assert worst <= MEAN_REL, (what, "row L1 ratio", worst, int(rows.argmax()))
    return ma, mr


def assert_lse(x, ref, what: str):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    inf_ref = np.isinf(ref)
    assert np.array_equal(np.isinf(x), inf_ref), what
    d = np.abs(x[~inf_ref] - ref[~inf_ref]).max() if (~inf_ref).any() else 0.0
    say("  %-28s max_abs %.3e" % (what + " (lse)", d))
    assert d <= LSE_ABS, (what, d)


def bf16_to_f64(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
