"""Python binding of the C ABI in include/wsk.h (argument marshalling only).

Every function here has the name of the C entry point it calls.  Device
buffers are torch tensors (PyTorch supplies device memory and the HIP stream);
host buffers are numpy arrays.  All compute runs in libwsk.so: if the library
is missing this module raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwsk.so")

WSK_OK, WSK_EINVAL, WSK_ENOMEM, WSK_ERANGE, WSK_EHIP, WSK_ESTATE = 0, -1, -2, -3, -4, -5
ERROR_NAMES = {WSK_EINVAL: "EINVAL", WSK_ENOMEM: "ENOMEM", WSK_ERANGE: "ERANGE",
               WSK_EHIP: "EHIP", WSK_ESTATE: "ESTATE"}
KIND_GQA, KIND_MLA = 0, 1
PART_CPU, PART_GPU, PART_LOAD = 0, 1, 2
LAYOUT_ROWS, LAYOUT_TILED64, LAYOUT_MLA32 = 0, 1, 2


class WskError(RuntimeError):
    def __init__(self, code: int, msg: str):
        self.code = code
        self.name = ERROR_NAMES.get(code, str(code))
        super().__init__("%s: %s" % (self.name, msg))


class wsk_partition_spec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("latent_dim", ctypes.c_int32), ("rope_dim", ctypes.c_int32),
                ("block_tokens", ctypes.c_int32), ("max_seqs", ctypes.c_int32), ("max_seq_len", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("device_pool_blocks", ctypes.c_int64),
                ("host_pool_blocks", ctypes.c_int64), ("softmax_scale", ctypes.c_float),
                ("evict_tokens", ctypes.c_int32), ("load_arena_blocks", ctypes.c_int32),
                ("pingpong_blocks", ctypes.c_int32), ("load_pool_blocks", ctypes.c_int64)]


class wsk_load_info(ctypes.Structure):
    _fields_ = [("pinned_bytes", ctypes.c_int64), ("slots_used", ctypes.c_int64), ("h2d_bytes", ctypes.c_int64),
                ("d2h_bytes", ctypes.c_int64), ("pin_seconds", ctypes.c_double), ("arenas", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class wsk_loc(ctypes.Structure):
    _fields_ = [("part", ctypes.c_int32), ("logical_block", ctypes.c_int32), ("slot", ctypes.c_int32),
                ("offset", ctypes.c_int32)]


class wsk_roofline(ctypes.Structure):
    _fields_ = [("A", ctypes.c_double), ("B", ctypes.c_double), ("c_cpu", ctypes.c_double),
                ("c_gpu", ctypes.c_double)]


class wsk_view(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("table", ctypes.POINTER(ctypes.c_int32)),
                ("slot_bytes", ctypes.c_int64), ("head_bytes", ctypes.c_int64), ("v_bytes", ctypes.c_int64),
                ("row_bytes", ctypes.c_int64), ("start", ctypes.c_int32), ("end", ctypes.c_int32),
                ("block_tokens", ctypes.c_int32), ("is_device", ctypes.c_int32),
                ("layout", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None
_VP, _I32, _I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
_PI32 = ctypes.POINTER(ctypes.c_int32)
_SIGS = {
    "wsk_last_error": ([], ctypes.c_char_p),
    "wsk_init": ([ctypes.POINTER(wsk_partition_spec), ctypes.c_int, ctypes.POINTER(_VP)], ctypes.c_int),
    "wsk_destroy": ([_VP], ctypes.c_int),
    "wsk_get_spec": ([_VP, ctypes.POINTER(wsk_partition_spec)], ctypes.c_int),
    "wsk_seq_open": ([_VP, _I32, _I32], ctypes.c_int),
    "wsk_seq_open_window": ([_VP, _I32, _I32, _I32], ctypes.c_int),
    "wsk_seq_segments": ([_VP, _I32, _I32, _PI32, _PI32, _PI32, _PI32], ctypes.c_int),
    "wsk_flush": ([_VP, _I32, _PI32, _PI32, _PI32, _VP], ctypes.c_int),
    "wsk_attend_gpu_workspace": ([_VP, _I32, _PI32, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
    "wsk_attend_gpu": ([_VP, _I32, _PI32, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP], ctypes.c_int),
    "wsk_attend_gpu_pass1": ([_VP, _I32, _PI32, _VP, _VP, ctypes.c_size_t, _VP], ctypes.c_int),
    "wsk_attend_gpu_pass2": ([_VP, _I32, _PI32, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP], ctypes.c_int),
    "wsk_decode_step_workspace": ([_VP, _I32, _PI32, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
    "wsk_decode_step_noalloc": ([_VP, _I32, _PI32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP], ctypes.c_int),
    "wsk_decode_step": ([_VP, _I32, _PI32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP],
                        ctypes.c_int),
    "wsk_decode_step_mla": ([_VP, _I32, _PI32, _VP, _VP, _VP, _VP, _VP, _I32, _VP, _VP, _VP, _VP, ctypes.c_size_t,
                             _VP], ctypes.c_int),
    "wsk_cpu_attend_all": ([_VP, _I32, _PI32, _VP, _VP, _VP, _I32], ctypes.c_int),
    "wsk_load_slot": ([_VP, _I32, ctypes.POINTER(_VP)], ctypes.c_int),
    "wsk_load_stats": ([_VP, ctypes.POINTER(wsk_load_info)], ctypes.c_int),
    "wsk_seq_close": ([_VP, _I32], ctypes.c_int),
    "wsk_seq_info": ([_VP, _I32, _PI32, _PI32], ctypes.c_int),
    "wsk_reserve": ([_VP, _I32, _I32], ctypes.c_int),
    "wsk_write": ([_VP, _I32, _I32, _I32, _VP, _VP, _VP], ctypes.c_int),
    "wsk_append": ([_VP, _I32, _PI32, _VP, _VP, _VP], ctypes.c_int),
    "wsk_route": ([_VP, _I32, _I32, ctypes.POINTER(wsk_loc)], ctypes.c_int),
    "wsk_views": ([_VP, _I32, ctypes.POINTER(wsk_view), ctypes.POINTER(wsk_view)], ctypes.c_int),
    "wsk_attend_workspace": ([_VP, _I32, _PI32, _PI32, _PI32, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
    "wsk_attend": ([_VP, _I32, _PI32, _PI32, _PI32, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP], ctypes.c_int),
    "wsk_stream_read": ([_VP, ctypes.c_size_t, _I32, _VP, _VP], ctypes.c_int),
    "wsk_host_read": ([_VP, ctypes.c_size_t, _I32, ctypes.POINTER(ctypes.c_uint64)], ctypes.c_int),
    "wsk_attend_blocks_workspace": ([_VP, _I32, _PI32, _PI32, _PI32, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
    "wsk_attend_blocks": ([_VP, _I32, _PI32, _PI32, _PI32, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP],
                          ctypes.c_int),
    "wsk_cpu_attend": ([_VP, _I32, _PI32, _PI32, _PI32, _VP, _VP, _VP, _I32], ctypes.c_int),
    "wsk_roofline_share": ([ctypes.POINTER(wsk_roofline), ctypes.c_int64, ctypes.POINTER(ctypes.c_double)],
                           ctypes.c_int),
    "wsk_policy_create": ([ctypes.POINTER(wsk_roofline), _I32, ctypes.POINTER(_VP)], ctypes.c_int),
    "wsk_policy_destroy": ([_VP], ctypes.c_int),
    "wsk_policy_observe": ([_VP, ctypes.c_double, ctypes.c_int64, ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "wsk_policy_route_batch": ([_VP, ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    "wsk_policy_model": ([_VP, ctypes.POINTER(wsk_roofline)], ctypes.c_int),
    "wsk_attend_pass1": ([_VP, _I32, _PI32, _PI32, _PI32, _VP, _VP, ctypes.c_size_t, _VP], ctypes.c_int),
    "wsk_attend_pass2": ([_VP, _I32, _PI32, _PI32, _PI32, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP],
                         ctypes.c_int),
    "wsk_merge": ([_I32, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP], ctypes.c_int),
    "wsk_mla_absorb": ([_I32, _I32, _I32, _I32, _VP, _VP, _VP, _I64, _VP], ctypes.c_int),
    "wsk_mla_expand": ([_I32, _I32, _I32, _I32, _VP, _VP, _VP, _VP], ctypes.c_int),
}


def lib() -> ctypes.CDLL:
    """Load libwsk.so (built by paper_2609_14507_amd.build); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libwsk.so is not built (%s): run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(rc: int):
    if rc != WSK_OK:
        raise WskError(rc, lib().wsk_last_error().decode())


def _ptr(t) -> Optional[int]:
    """Device pointer of a torch tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    """hipStream_t handle: the given one, else torch's current stream once torch has
    initialised the GPU, else NULL (the legacy default stream)."""
    if stream is not None:
        return stream
    import torch
    if torch.cuda.is_initialized():
        return torch.cuda.current_stream().cuda_stream
    return None


def _i32_array(xs: Sequence[int]):
    a = (ctypes.c_int32 * max(1, len(xs)))(*[int(x) for x in xs])
    return a


def wsk_last_error() -> str:
    return lib().wsk_last_error().decode()


def make_spec(kind: int, n_q_heads: int, n_kv_heads: int, head_dim: int, block_tokens: int, max_seqs: int,
              max_seq_len: int, device_pool_blocks: int, host_pool_blocks: int, softmax_scale: float,
              latent_dim: int = 0, rope_dim: int = 0, evict_tokens: int = 0, load_pool_blocks: int = 0,
              load_arena_blocks: int = 0, pingpong_blocks: int = 0) -> wsk_partition_spec:
    return wsk_partition_spec(kind, n_q_heads, n_kv_heads, head_dim, latent_dim, rope_dim, block_tokens,
                              max_seqs, max_seq_len, 0, device_pool_blocks, host_pool_blocks, softmax_scale,
                              evict_tokens, load_arena_blocks, pingpong_blocks, load_pool_blocks)


def wsk_init(spec: wsk_partition_spec, device: int) -> int:
    h = ctypes.c_void_p()
    _check(lib().wsk_init(ctypes.byref(spec), device, ctypes.byref(h)))
    return h.value


def wsk_destroy(h: int):
    _check(lib().wsk_destroy(h))


def wsk_get_spec(h: int) -> wsk_partition_spec:
    s = wsk_partition_spec()
    _check(lib().wsk_get_spec(h, ctypes.byref(s)))
    return s


def wsk_seq_open(h: int, seq: int, split: int):
    _check(lib().wsk_seq_open(h, seq, split))


def wsk_seq_open_window(h: int, seq: int, split: int, load_end: int):
    _check(lib().wsk_seq_open_window(h, seq, split, load_end))


def wsk_seq_segments(h: int, seq: int):
    """[(start, end, part), ...] covering [0, L)."""
    n = ctypes.c_int32()
    _check(lib().wsk_seq_segments(h, seq, 0, None, None, None, ctypes.byref(n)))
    cap = max(1, n.value)
    a, e, p = (ctypes.c_int32 * cap)(), (ctypes.c_int32 * cap)(), (ctypes.c_int32 * cap)()
    _check(lib().wsk_seq_segments(h, seq, cap, a, e, p, ctypes.byref(n)))
    return [(a[k], e[k], p[k]) for k in range(n.value)]


def wsk_flush(h: int, seq_ids, parts, stream=None):
    """Evict one D-batch per listed sequence; returns the positions moved per sequence."""
    moved = (ctypes.c_int32 * max(1, len(seq_ids)))()
    _check(lib().wsk_flush(h, len(seq_ids), _i32_array(seq_ids), _i32_array(parts), moved, _stream(stream)))
    return [moved[i] for i in range(len(seq_ids))]


def wsk_attend_gpu_workspace(h: int, seq_ids) -> int:
    b = ctypes.c_size_t()
    _check(lib().wsk_attend_gpu_workspace(h, len(seq_ids), _i32_array(seq_ids), ctypes.byref(b)))
    return b.value


def wsk_attend_gpu(h: int, seq_ids, q, o, lse, ws, o_x=None, lse_x=None, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().wsk_attend_gpu(h, len(seq_ids), _i32_array(seq_ids), _ptr(q), _ptr(o_x), _ptr(lse_x), _ptr(o),
                                _ptr(lse), _ptr(ws), nbytes, _stream(stream)))


def wsk_attend_gpu_pass1(h: int, seq_ids, q, ws, stream=None):
    nbytes = ws.numel() * ws.element_size()
    _check(lib().wsk_attend_gpu_pass1(h, len(seq_ids), _i32_array(seq_ids), _ptr(q), _ptr(ws), nbytes,
                                      _stream(stream)))


def wsk_attend_gpu_pass2(h: int, seq_ids, o, lse, ws, o_x=None, lse_x=None, stream=None):
    nbytes = ws.numel() * ws.element_size()
    _check(lib().wsk_attend_gpu_pass2(h, len(seq_ids), _i32_array(seq_ids), _ptr(o_x), _ptr(lse_x), _ptr(o),
                                      _ptr(lse), _ptr(ws), nbytes, _stream(stream)))


def wsk_decode_step_workspace(h: int, seq_ids) -> int:
    b = ctypes.c_size_t()
    _check(lib().wsk_decode_step_workspace(h, len(seq_ids), _i32_array(seq_ids), ctypes.byref(b)))
    return b.value


def wsk_decode_step(h: int, seq_ids, q, k_new, v_new, o, lse, ws, o_x=None, lse_x=None, stream=None):
    """Append + attend every GPU-side position (the new row included) + merge, in one call."""
    nbytes = ws.numel() * ws.element_size()
    _check(lib().wsk_decode_step(h, len(seq_ids), _i32_array(seq_ids), _ptr(q), _ptr(k_new), _ptr(v_new),
                                 _ptr(o_x), _ptr(lse_x), _ptr(o), _ptr(lse), _ptr(ws), nbytes, _stream(stream)))


def wsk_decode_step_noalloc(h: int, seq_ids, q, k_new, v_new, o, lse, o_x=None, lse_x=None, stream=None):
    """wsk_decode_step with its chunk partials in the library's own device scratch (no workspace)."""
    _check(lib().wsk_decode_step_noalloc(h, len(seq_ids), _i32_array(seq_ids), _ptr(q), _ptr(k_new), _ptr(v_new),
                                         _ptr(o_x), _ptr(lse_x), _ptr(o), _ptr(lse), _stream(stream)))


def wsk_decode_step_mla(h: int, seq_ids, q, k_new, w_uv, o, lse, ws, o_lat=None, o_x=None, lse_x=None,
                        stream=None):
    """MLA decode step with the output expansion: o fp32 [n, H, dv] from w_uv bf16 [H, 512, dv];
    o_lat (optional) receives the merged latent output."""
    nbytes = ws.numel() * ws.element_size()
    dv = w_uv.shape[2]
    _check(lib().wsk_decode_step_mla(h, len(seq_ids), _i32_array(seq_ids), _ptr(q), _ptr(k_new), _ptr(o_x),
                                     _ptr(lse_x), _ptr(w_uv), dv, _ptr(o_lat), _ptr(lse), _ptr(o), _ptr(ws), nbytes,
                                     _stream(stream)))


def wsk_cpu_attend_all(h: int, seq_ids, q, o, lse, threads: int = 0):
    """CPU engine over every CPU-partition position; host numpy arrays as for wsk_cpu_attend."""
    for a, dt in ((q, np.uint16), (o, np.float32), (lse, np.float32)):
        if a.dtype != dt or not a.flags["C_CONTIGUOUS"]:
            raise ValueError("host arrays must be C-contiguous with the documented dtypes")
    _check(lib().wsk_cpu_attend_all(h, len(seq_ids), _i32_array(seq_ids), q.ctypes.data, o.ctypes.data,
                                    lse.ctypes.data, threads))


def wsk_load_slot(h: int, slot: int) -> int:
    p = _VP()
    _check(lib().wsk_load_slot(h, slot, ctypes.byref(p)))
    return p.value


def wsk_load_stats(h: int) -> wsk_load_info:
    info = wsk_load_info()
    _check(lib().wsk_load_stats(h, ctypes.byref(info)))
    return info


def wsk_seq_close(h: int, seq: int):
    _check(lib().wsk_seq_close(h, seq))


def wsk_seq_info(h: int, seq: int) -> Tuple[int, int]:
    L, s = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().wsk_seq_info(h, seq, ctypes.byref(L), ctypes.byref(s)))
    return L.value, s.value


def wsk_reserve(h: int, seq: int, n: int):
    _check(lib().wsk_reserve(h, seq, n))


def wsk_write(h: int, seq: int, pos0: int, k: np.ndarray, v: Optional[np.ndarray], stream=None):
    """k, v: host uint16 (bf16 bits), token-major [n, Hkv, D] (MLA: k [n, row], v None)."""
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = None if v is None else np.ascontiguousarray(v, dtype=np.uint16)
    n = k.shape[0]
    _check(lib().wsk_write(h, seq, pos0, n, k.ctypes.data, None if v is None else v.ctypes.data,
                           _stream(stream) if n else None))


def wsk_append(h: int, seq_ids: Sequence[int], k_new, v_new=None, stream=None):
    """k_new, v_new: device tensors (bf16), row i for seq_ids[i]."""
    ids = _i32_array(seq_ids)
    _check(lib().wsk_append(h, len(seq_ids), ids, _ptr(k_new), _ptr(v_new), _stream(stream)))


def wsk_route(h: int, seq: int, pos: int) -> Tuple[int, int, int, int]:
    loc = wsk_loc()
    _check(lib().wsk_route(h, seq, pos, ctypes.byref(loc)))
    return loc.part, loc.logical_block, loc.slot, loc.offset


def wsk_views(h: int, seq: int) -> Tuple[wsk_view, wsk_view]:
    cpu, gpu = wsk_view(), wsk_view()
    _check(lib().wsk_views(h, seq, ctypes.byref(cpu), ctypes.byref(gpu)))
    return cpu, gpu


def wsk_attend_workspace(h: int, seq_ids, start, end) -> int:
    b = ctypes.c_size_t()
    _check(lib().wsk_attend_workspace(h, len(seq_ids), _i32_array(seq_ids), _i32_array(start),
                                      _i32_array(end), ctypes.byref(b)))
    return b.value


def wsk_attend(h: int, seq_ids, start, end, q, o, lse, ws, stream=None):
    """q: device bf16 [n, H, qwidth]; o: fp32 [n, H, width]; lse fp32 [n, H]; ws: device uint8 buffer."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().wsk_attend(h, len(seq_ids), _i32_array(seq_ids), _i32_array(start), _i32_array(end),
                            _ptr(q), _ptr(o), _ptr(lse), _ptr(ws), nbytes, _stream(stream)))


def wsk_attend_pass1(h: int, seq_ids, start, end, q, ws, stream=None):
    """Pass 1 of wsk_attend: the chunk partials into ws."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().wsk_attend_pass1(h, len(seq_ids), _i32_array(seq_ids), _i32_array(start), _i32_array(end),
                                  _ptr(q), _ptr(ws), nbytes, _stream(stream)))


def wsk_attend_pass2(h: int, seq_ids, start, end, o, lse, ws, o_x=None, lse_x=None, stream=None):
    """Pass 2 of wsk_attend: merges the chunk partials in ws (and, if given,
    the partial (o_x, lse_x) over other keys) into o, lse."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().wsk_attend_pass2(h, len(seq_ids), _i32_array(seq_ids), _i32_array(start), _i32_array(end),
                                  _ptr(o_x), _ptr(lse_x), _ptr(o), _ptr(lse), _ptr(ws), nbytes, _stream(stream)))


def wsk_merge(o_a, lse_a, o_b, lse_b, o_out, lse_out, o_bf16=None, stream=None):
    """Row-wise LSE merge of fp32 device partials [rows, width] / [rows]."""
    width = o_a.shape[-1]
    rows = o_a.numel() // width
    _check(lib().wsk_merge(rows, width, _ptr(o_a), _ptr(lse_a), _ptr(o_b), _ptr(lse_b), _ptr(o_out),
                           _ptr(lse_out), _ptr(o_bf16), _stream(stream)))


def wsk_mla_absorb(q_nope, w_uk, out, out_stride: int, stream=None):
    """q_nope bf16 [n, H, dn], w_uk bf16 [H, dn, dl]; out bf16 rows at stride out_stride."""
    n, H, dn = q_nope.shape
    dl = w_uk.shape[2]
    _check(lib().wsk_mla_absorb(n, H, dn, dl, _ptr(q_nope), _ptr(w_uk), _ptr(out), out_stride, _stream(stream)))


def wsk_mla_expand(o_lat, w_uv, o, stream=None):
    """o_lat fp32 [n, H, dl], w_uv bf16 [H, dl, dv] -> o fp32 [n, H, dv]."""
    n, H, dl = o_lat.shape
    dv = w_uv.shape[2]
    _check(lib().wsk_mla_expand(n, H, dl, dv, _ptr(o_lat), _ptr(w_uv), _ptr(o), _stream(stream)))


def wsk_host_read(arr: np.ndarray, threads: int = 0) -> int:
    """Measurement aid: one plain read of a host array on the CPU engine's threads."""
    if not arr.flags["C_CONTIGUOUS"]:
        raise ValueError("array must be C-contiguous")
    out = ctypes.c_uint64()
    _check(lib().wsk_host_read(arr.ctypes.data, arr.nbytes, threads, ctypes.byref(out)))
    return out.value


def wsk_stream_read(buf, out, workgroups: int = 0, stream=None):
    """Measurement aid: one plain read of buf with the attention kernels' loads."""
    _check(lib().wsk_stream_read(_ptr(buf), buf.numel() * buf.element_size(), workgroups, _ptr(out), _stream(stream)))


def wsk_roofline_share(A: float, B: float, c_cpu: float, c_gpu: float, L: int) -> float:
    """Eq. 2: the CPU share that balances the engines at length L."""
    r = ctypes.c_double()
    _check(lib().wsk_roofline_share(ctypes.byref(wsk_roofline(A, B, c_cpu, c_gpu)), L, ctypes.byref(r)))
    return r.value


class Policy:
    """The online split policy (wsk_policy_*)."""

    def __init__(self, A: float, B: float, c_cpu: float, c_gpu: float, window: int):
        self.h = _VP()
        _check(lib().wsk_policy_create(ctypes.byref(wsk_roofline(A, B, c_cpu, c_gpu)), window,
                                       ctypes.byref(self.h)))

    def observe(self, t_cpu: float, n_cpu: int) -> float:
        a = ctypes.c_double()
        _check(lib().wsk_policy_observe(self.h, t_cpu, n_cpu, ctypes.byref(a)))
        return a.value

    def route(self) -> int:
        part = ctypes.c_int32()
        _check(lib().wsk_policy_route_batch(self.h, ctypes.byref(part)))
        return part.value

    def model(self):
        m = wsk_roofline()
        _check(lib().wsk_policy_model(self.h, ctypes.byref(m)))
        return m.A, m.B, m.c_cpu, m.c_gpu

    def close(self):
        if self.h:
            lib().wsk_policy_destroy(self.h)
            self.h = _VP()


def wsk_cpu_attend(h: int, seq_ids, start, end, q, o, lse, threads: int = 0):
    """CPU engine over the CPU partition.  q: numpy uint16 (bf16 bits) [n, H, row];
    o: numpy float32 [n, H, dv]; lse: numpy float32 [n, H] (host arrays)."""
    import numpy as np
    for a, dt in ((q, np.uint16), (o, np.float32), (lse, np.float32)):
        if a.dtype != dt or not a.flags["C_CONTIGUOUS"]:
            raise ValueError("host arrays must be C-contiguous with the documented dtypes")
    _check(lib().wsk_cpu_attend(h, len(seq_ids), _i32_array(seq_ids), _i32_array(start), _i32_array(end),
                                q.ctypes.data, o.ctypes.data, lse.ctypes.data, threads))


def _selection(sel_lists):
    begin = [0]
    flat = []
    for lst in sel_lists:
        flat.extend(int(b) for b in lst)
        begin.append(len(flat))
    return begin, flat


def wsk_attend_blocks_workspace(h: int, seq_ids, sel_lists) -> int:
    begin, flat = _selection(sel_lists)
    b = ctypes.c_size_t()
    _check(lib().wsk_attend_blocks_workspace(h, len(seq_ids), _i32_array(seq_ids), _i32_array(begin),
                                             _i32_array(flat) if flat else None, ctypes.byref(b)))
    return b.value


def wsk_attend_blocks(h: int, seq_ids, sel_lists, q, o, lse, ws, o_x=None, lse_x=None, stream=None):
    """Block-sparse attention: sel_lists[i] = logical GPU blocks of seq_ids[i] to attend."""
    begin, flat = _selection(sel_lists)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().wsk_attend_blocks(h, len(seq_ids), _i32_array(seq_ids), _i32_array(begin),
                                   _i32_array(flat) if flat else None, _ptr(q), _ptr(o_x), _ptr(lse_x), _ptr(o),
                                   _ptr(lse), _ptr(ws), nbytes, _stream(stream)))
