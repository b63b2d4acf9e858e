"""fp64 CPU oracle of the partitioned-KV decode path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (``paper_2609_14507_amd``)
never does, and this package imports nothing from the product.

``wsk_oracle.c`` holds the arithmetic (attention, LSE merge, MLA absorb and
expand, bf16 rounding); ``route.py`` holds the write-time routing rule.  This
module only builds and loads the C library and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wsk_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (IEEE fp64: no fast-math).  sanitize=True
    builds it with clang's ASan and UBSan instead (the runtime the sanitized
    HIP library uses, so that one process can load both)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        if sanitize:
            cc = ["/opt/rocm/llvm/bin/clang", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                  "-fno-omit-frame-pointer", "-g", "-fopenmp=libgomp"]
        else:
            cc = ["gcc", "-fopenmp"]
        subprocess.check_call(cc + ["-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
                                    "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        d, i64, i32 = ctypes.POINTER(ctypes.c_double), ctypes.c_int64, ctypes.c_int
        u16 = ctypes.POINTER(ctypes.c_uint16)
        L.oracle_attend.argtypes = [i32, i32, i32, i32, d, u16, i64, i64, u16, i64, i64,
                                    i64, i64, ctypes.c_double, d, d]
        L.oracle_merge.argtypes = [i64, i32, d, d, d, d, d, d]
        L.oracle_mla_absorb.argtypes = [i32, i32, i32, u16, u16, d]
        L.oracle_mla_expand.argtypes = [i32, i32, i32, d, u16, d]
        L.oracle_round_bf16.argtypes = [i64, d, u16]
        L.oracle_set_threads.argtypes = [i32]
        for f in (L.oracle_attend, L.oracle_merge, L.oracle_mla_absorb,
                  L.oracle_mla_expand, L.oracle_round_bf16, L.oracle_max_threads, L.oracle_set_threads):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of raw bf16 bits to fp64."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def attend(q, k, v, a: int, e: int, scale: float, G: int, dv: int = None):
    """Exact attention of every query head over key positions [a, e).

    q : [H, dk] (fp64, or uint16 bf16 bits which are widened exactly)
    k : token-major cache of one sequence, [T, Hkv, dk] (GQA) or [T, dk_row] (MLA rows)
    v : [T, Hkv, dv] (GQA) or None (MLA: the first ``dv`` elements of each key row)
    Returns (O [H, dv] fp64, LSE [H] fp64).
    """
    q = np.ascontiguousarray(bf16_to_f64(q) if q.dtype == np.uint16 else q, dtype=np.float64)
    H, dk = q.shape
    k = np.ascontiguousarray(k, dtype=np.uint16)
    if v is None:                       # MLA: one shared latent row per token
        assert k.ndim == 2 and dv is not None
        k_row, k_head = k.shape[1], 0
        vv, v_row, v_head = k, k.shape[1], 0
    else:
        assert k.ndim == 3 and k.shape[2] == dk
        k_row, k_head = k.shape[1] * k.shape[2], k.shape[2]
        vv = np.ascontiguousarray(v, dtype=np.uint16)
        dv = vv.shape[2]
        v_row, v_head = vv.shape[1] * vv.shape[2], vv.shape[2]
    o = np.empty((H, dv), np.float64)
    lse = np.empty(H, np.float64)
    rc = lib().oracle_attend(H, G, dk, dv, _p(q, ctypes.c_double),
                             _p(k, ctypes.c_uint16), k_row, k_head,
                             _p(vv, ctypes.c_uint16), v_row, v_head,
                             int(a), int(e), float(scale),
                             _p(o, ctypes.c_double), _p(lse, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle_attend failed")
    return o, lse


def merge(o_a, lse_a, o_b, lse_b):
    """LSE merge of two partials over disjoint key sets (fp64)."""
    o_a = np.ascontiguousarray(o_a, np.float64)
    o_b = np.ascontiguousarray(o_b, np.float64)
    lse_a = np.ascontiguousarray(lse_a, np.float64).reshape(-1)
    lse_b = np.ascontiguousarray(lse_b, np.float64).reshape(-1)
    width = o_a.shape[-1]
    rows = o_a.size // width
    o = np.empty_like(o_a)
    lse = np.empty(rows, np.float64)
    rc = lib().oracle_merge(rows, width, _p(o_a, ctypes.c_double), _p(lse_a, ctypes.c_double),
                            _p(o_b, ctypes.c_double), _p(lse_b, ctypes.c_double),
                            _p(o, ctypes.c_double), _p(lse, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle_merge failed")
    return o, lse.reshape(o_a.shape[:-1])


def mla_absorb(q_nope, w_uk):
    """q_lat[h] = W_UK[h]^T q_nope[h] in fp64 (unrounded).  q_nope [H, dn], w_uk [H, dn, dl] bf16."""
    q_nope = np.ascontiguousarray(q_nope, np.uint16)
    w_uk = np.ascontiguousarray(w_uk, np.uint16)
    H, dn, dl = w_uk.shape
    out = np.empty((H, dl), np.float64)
    rc = lib().oracle_mla_absorb(H, dn, dl, _p(q_nope, ctypes.c_uint16),
                                 _p(w_uk, ctypes.c_uint16), _p(out, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle_mla_absorb failed")
    return out


def mla_expand(o_lat, w_uv):
    """O[h] = W_UV[h]^T O_lat[h] in fp64.  o_lat [H, dl] fp64, w_uv [H, dl, dv] bf16."""
    o_lat = np.ascontiguousarray(o_lat, np.float64)
    w_uv = np.ascontiguousarray(w_uv, np.uint16)
    H, dl, dv = w_uv.shape
    out = np.empty((H, dv), np.float64)
    rc = lib().oracle_mla_expand(H, dl, dv, _p(o_lat, ctypes.c_double),
                                 _p(w_uv, ctypes.c_uint16), _p(out, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle_mla_expand failed")
    return out


def round_bf16(x) -> np.ndarray:
    """fp64 -> bf16 bits, round to nearest even."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    lib().oracle_round_bf16(x.size, _p(x, ctypes.c_double), _p(out, ctypes.c_uint16))
    return out


def max_threads() -> int:
    return int(lib().oracle_max_threads())


def set_threads(n: int):
    """OpenMP threads of later oracle calls (timing only)."""
    assert lib().oracle_set_threads(int(n)) == 0
