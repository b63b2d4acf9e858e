"""Helpers shared by the GPU tests: device readback, error metrics, printing."""
import ctypes
import sys

import numpy as np
import torch

_hip = None

# Tolerances of the decode outputs against the fp64 oracle (bf16 inputs, fp32
# accumulation): largest absolute error and the L1 ratio sum|x-r| / sum|r|.
MAX_ABS = 1e-2
MEAN_REL = 1e-3
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


def assert_close(x, ref, what: str):
    ma, mr = errors(x, ref)
    say("  %-28s max_abs %.3e  mean_rel %.3e" % (what, ma, mr))
    assert np.all(np.isfinite(x)), what
    assert ma <= MAX_ABS and mr <= MEAN_REL, (what, ma, mr)
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
