"""The load region on host-only caches (CPU): routing of [s, load_end) into
it, the bytes of its slots against the GPU layouts of include/wsk.h, the
segment list, arena-by-arena pinning one arena ahead, the CPU engine over
every CPU position, and the refused cases.  (The load region of a host-only
cache is plain host memory; everything that moves it to a GPU is tested in
tests/test_gpu_load.py.)"""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from tests.gpu_util import assert_close, assert_lse
from tests.layouts import gqa_elements, mla_elements

CPU, GPU, LOAD = wsk.PART_CPU, wsk.PART_GPU, wsk.PART_LOAD


def _workload(kind, H=8):
    if kind == "gqa":
        return wl.Workload("load-gqa", wl.GQA, batch=1, n_q_heads=H, n_kv_heads=2, head_dim=128, context=1)
    return wl.Workload("load-mla", wl.MLA, batch=1, n_q_heads=H, n_kv_heads=1, head_dim=128, latent_dim=512,
                       rope_dim=64, nope_dim=128, context=1, kv_std=0.5)


def _spec(w, bk, max_len, host_blocks, load_blocks, arena, nseq=4, evict=0, pingpong=8):
    common = dict(evict_tokens=evict, load_pool_blocks=load_blocks, load_arena_blocks=arena if load_blocks else 0,
                  pingpong_blocks=pingpong if load_blocks else 0)
    if w.kind == wl.MLA:
        return wsk.make_spec(wsk.KIND_MLA, w.n_q_heads, 1, w.head_dim, bk, nseq, max_len, 0, host_blocks,
                             w.softmax_scale, latent_dim=w.latent_dim, rope_dim=w.rope_dim, **common)
    return wsk.make_spec(wsk.KIND_GQA, w.n_q_heads, w.n_kv_heads, w.head_dim, bk, nseq, max_len, 0, host_blocks,
                         w.softmax_scale, **common)


def _draw(w, gen, L):
    if w.kind == wl.MLA:
        return wl.draw_bf16(gen, (L, w.row_elems), w.kv_std), None
    return wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)), wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim))


def _slot_u16(h, slot, slot_bytes):
    p = wsk.wsk_load_slot(h, slot)
    return np.frombuffer((ctypes.c_uint16 * (slot_bytes // 2)).from_address(p), dtype=np.uint16).copy()


def _slot_bytes(w, bk):
    return w.token_bytes * bk


@pytest.mark.parametrize("kind,bk", [("gqa", 64), ("gqa", 128), ("mla", 64), ("mla", 256)])
def test_prefill_routes_into_the_load_region_in_gpu_layout(kind, bk):
    w = _workload(kind)
    gen = __import__("torch").Generator().manual_seed(7 + bk)
    # (split, load_end): split inside a block, split on a boundary, no CPU
    # part, no load part
    cases = [(bk + 37, 4 * bk), (2 * bk, 3 * bk), (0, 2 * bk), (bk // 2, bk // 2)]
    spec = _spec(w, bk, 4 * bk, host_blocks=16, load_blocks=16, arena=4)
    h = wsk.wsk_init(spec, -1)
    try:
        rows = []
        for b, (s, e) in enumerate(cases):
            wsk.wsk_seq_open_window(h, b, s, e)
            k, v = _draw(w, gen, e)
            wsk.wsk_write(h, b, 0, k, v)
            rows.append((k, v))
        # segments and routing: CPU and load slots lowest-free-first in write order
        next_slot = {CPU: 0, LOAD: 0}
        sb = _slot_bytes(w, bk)
        for b, (s, e) in enumerate(cases):
            want = [(a, z, p) for a, z, p in ((0, s, CPU), (s, e, LOAD)) if z > a]
            assert wsk.wsk_seq_segments(h, b) == want
            slot_of = {}
            for p in range(e):
                part = CPU if p < s else LOAD
                key = (part, p // bk)
                if key not in slot_of:
                    slot_of[key] = next_slot[part]
                    next_slot[part] += 1
                assert wsk.wsk_route(h, b, p) == (part, p // bk, slot_of[key], p % bk), (b, p)
            # load-region bytes: every load position at its TILED64 / MLA32
            # element; nothing else written
            k, v = rows[b]
            for blk in range(s // bk, (e + bk - 1) // bk) if e > s else []:
                slot = slot_of[(LOAD, blk)]
                mem = _slot_u16(h, slot, sb)
                touched = np.zeros(mem.shape, bool)
                pos = np.arange(max(s, blk * bk), min(e, (blk + 1) * bk))
                off = pos % bk
                if w.kind == wl.MLA:
                    el = mla_elements(off, w.row_elems)
                    assert np.array_equal(mem[el], k[pos])
                    touched[el] = True
                else:
                    for g in range(w.n_kv_heads):
                        ke, ve = gqa_elements(off, w.head_dim, bk, g)
                        assert np.array_equal(mem[ke], k[pos, g])
                        assert np.array_equal(mem[ve], v[pos, g])
                        touched[ke] = True
                        touched[ve] = True
                assert not mem[~touched].any()
        # pinning: slots 0..N-1 used; arenas of 4 pinned as needed, plus one
        # ahead once the last used arena is half full
        st = wsk.wsk_load_stats(h)
        used = next_slot[LOAD]
        assert st.slots_used == used
        need = -(-used // 4)
        ahead = 1 if (used - 1) % 4 >= 2 and need < 4 else 0
        assert st.arenas == need + ahead
        assert st.pinned_bytes == st.arenas * 4 * sb
        # the CPU engine over every CPU position
        q = wl.draw_bf16(gen, (len(cases), w.n_q_heads, w.row_elems))
        dv = w.latent_dim if w.kind == wl.MLA else w.head_dim
        o = np.empty((len(cases), w.n_q_heads, dv), np.float32)
        lse = np.empty((len(cases), w.n_q_heads), np.float32)
        wsk.wsk_cpu_attend_all(h, list(range(len(cases))), q, o, lse, 2)
        g = w.n_q_heads if w.kind == wl.MLA else w.group
        for b, (s, e) in enumerate(cases):
            if s == 0:
                assert np.all(o[b] == 0) and np.all(np.isneginf(lse[b]))
                continue
            o_r, l_r = oracle.attend(q[b], rows[b][0], rows[b][1], 0, s, w.softmax_scale, g, dv=dv)
            assert_close(o[b], o_r, "cpu_attend_all b%d" % b)
            assert_lse(lse[b], l_r, "cpu_attend_all b%d" % b)
        # a range reaching into the load region is not the CPU's
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_cpu_attend(h, [0], [0], [cases[0][0] + 1], np.ascontiguousarray(q[:1]), o[:1], lse[:1])
        assert ei.value.code == wsk.WSK_ERANGE
        # closing returns the load slots: reopening takes the same ones
        wsk.wsk_seq_close(h, 0)
        s, e = cases[0]
        wsk.wsk_seq_open_window(h, 0, s, e)
        wsk.wsk_write(h, 0, 0, *rows[0])
        assert wsk.wsk_route(h, 0, s)[2] == 0
    finally:
        wsk.wsk_destroy(h)


def test_refused_load_region_cases():
    w = _workload("gqa")
    with pytest.raises(wsk.WskError) as ei:     # load region without arena or ping-pong sizes
        wsk.wsk_init(_spec(w, 64, 512, 4, 8, 0), -1)
    assert ei.value.code == wsk.WSK_EINVAL
    with pytest.raises(wsk.WskError) as ei:     # eviction batch not a multiple of the block
        wsk.wsk_init(_spec(w, 64, 512, 4, 8, 2, evict=96), -1)
    assert ei.value.code == wsk.WSK_EINVAL
    h = wsk.wsk_init(_spec(w, 64, 512, 4, 0, 0, evict=128), -1)
    try:
        with pytest.raises(wsk.WskError) as ei:  # no load region
            wsk.wsk_seq_open_window(h, 0, 10, 64)
        assert ei.value.code == wsk.WSK_ESTATE
        wsk.wsk_seq_open_window(h, 0, 10, 10)    # an empty load range needs none
        assert wsk.wsk_seq_segments(h, 0) == []
    finally:
        wsk.wsk_destroy(h)
    h = wsk.wsk_init(_spec(w, 64, 512, 4, 8, 2, evict=128), -1)
    try:
        for s, e, code in ((10, 100, wsk.WSK_EINVAL), (70, 64, wsk.WSK_EINVAL)):
            with pytest.raises(wsk.WskError) as ei:
                wsk.wsk_seq_open_window(h, 0, s, e)
            assert ei.value.code == code
        wsk.wsk_seq_open_window(h, 0, 10, 128)
        k, v = _draw(w, __import__("torch").Generator().manual_seed(1), 130)
        with pytest.raises(wsk.WskError) as ei:  # positions past load_end need a device
            wsk.wsk_write(h, 0, 0, k, v)
        assert ei.value.code == wsk.WSK_ESTATE
        wsk.wsk_write(h, 0, 0, k[:128], v[:128])
        with pytest.raises(wsk.WskError) as ei:  # eviction needs a device
            wsk.wsk_flush(h, [0], [CPU])
        assert ei.value.code == wsk.WSK_ESTATE
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_load_slot(h, 8)
        assert ei.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ei:  # its arena was never pinned
            wsk.wsk_load_slot(h, 6)
        assert ei.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_seq_open_window(h, 1, 0, 576)   # past max_seq_len
        assert ei.value.code == wsk.WSK_EINVAL
        # 6 of the 8 load slots are free: 7 blocks do not fit, and the failed
        # write changes nothing
        wsk.wsk_seq_open_window(h, 1, 0, 448)
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_write(h, 1, 0, *_draw(w, __import__("torch").Generator().manual_seed(2), 448))
        assert ei.value.code == wsk.WSK_ENOMEM
        assert wsk.wsk_seq_info(h, 1)[0] == 0
        assert wsk.wsk_load_stats(h).slots_used == 2
    finally:
        wsk.wsk_destroy(h)
