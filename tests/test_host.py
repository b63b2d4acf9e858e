"""Host-side checks of libwsk.so that need no GPU.

A cache created with device = -1 never calls HIP: routing (wsk_reserve),
wsk_route, CPU views and CPU-partition writes work, GPU calls are refused.
Routing is compared with the oracle's model of the write-time rule.
"""
import ctypes
import json
import os
import re

import numpy as np
import pytest

from oracle.route import CPU, GPU, RouteError, RouteModel
from paper_2609_14507_amd import wsk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "wsk.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(wsk_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = wsk.lib()
    names = _declared_symbols()
    assert len(names) == 44
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(wsk._SIGS)


def _spec(**kw):
    base = dict(kind=wsk.KIND_GQA, n_q_heads=8, n_kv_heads=2, head_dim=128, block_tokens=64, max_seqs=4,
                max_seq_len=1024, device_pool_blocks=16, host_pool_blocks=16, softmax_scale=0.088)
    base.update(kw)
    return wsk.make_spec(**base)


@pytest.mark.parametrize("bad", [
    dict(kind=7), dict(n_q_heads=0), dict(n_q_heads=6, n_kv_heads=4), dict(head_dim=64),
    dict(block_tokens=32), dict(block_tokens=96), dict(max_seqs=0), dict(max_seq_len=0),
    dict(device_pool_blocks=-1), dict(softmax_scale=0.0), dict(softmax_scale=float("nan")),
    dict(n_q_heads=130, n_kv_heads=2),
    dict(kind=wsk.KIND_MLA, n_q_heads=16, n_kv_heads=2, latent_dim=512, rope_dim=64),
    dict(kind=wsk.KIND_MLA, n_q_heads=16, n_kv_heads=1, latent_dim=256, rope_dim=64),
    dict(kind=wsk.KIND_MLA, n_q_heads=32, n_kv_heads=1, latent_dim=512, rope_dim=64),
])
def test_spec_validation_rejects(bad):
    with pytest.raises(wsk.WskError) as ex:
        wsk.wsk_init(_spec(**bad), -1)
    assert ex.value.code == wsk.WSK_EINVAL


def test_spec_reserved_must_be_zero():
    s = _spec()
    s.reserved = 1
    with pytest.raises(wsk.WskError):
        wsk.wsk_init(s, -1)


def test_host_only_cache_refuses_gpu_work():
    h = wsk.wsk_init(_spec(), -1)
    try:
        wsk.wsk_seq_open(h, 0, 100)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_write(h, 0, 0, np.zeros((130, 2, 128), np.uint16), np.zeros((130, 2, 128), np.uint16))
        assert ex.value.code == wsk.WSK_ESTATE
        assert wsk.wsk_seq_info(h, 0) == (0, 100)        # nothing changed
        lib = wsk.lib()
        ids = (ctypes.c_int32 * 1)(0)
        rc = lib.wsk_append(h, 1, ids, 16, 16, None)
        assert rc == wsk.WSK_ESTATE
    finally:
        wsk.wsk_destroy(h)


def _replay_golden(h, model_ops):
    """Replay the hand-derived routing fixture; data-free ops use wsk_reserve."""
    for op in model_ops:
        kind, err = op["op"], op.get("error")
        try:
            if kind == "open":
                wsk.wsk_seq_open(h, op["seq"], op["split"])
            elif kind == "write":
                L, _ = wsk.wsk_seq_info(h, op["seq"])
                if op["pos0"] != L:
                    # the position check happens before any routing
                    wsk.wsk_write(h, op["seq"], op["pos0"], np.zeros((op["n"], 2, 128), np.uint16),
                                  np.zeros((op["n"], 2, 128), np.uint16))
                else:
                    wsk.wsk_reserve(h, op["seq"], op["n"])
            elif kind == "append":
                for sq in sorted(op["seqs"]):
                    wsk.wsk_reserve(h, sq, 1)
            elif kind == "close":
                wsk.wsk_seq_close(h, op["seq"])
            elif kind == "expect_route":
                got = [list(wsk.wsk_route(h, op["seq"], p)) for p in range(len(op["routes"]))]
                assert got == op["routes"], (op, got)
            elif kind == "expect_length":
                assert wsk.wsk_seq_info(h, op["seq"])[0] == op["length"]
        except wsk.WskError as ex:
            assert err == ex.name, (op, str(ex))
            continue
        assert err is None, ("expected failure", op)


def test_routing_matches_hand_derived_fixture():
    with open(os.path.join(GOLDEN, "route_small.json")) as f:
        g = json.load(f)
    # the fixture's block size is 4; the library's smallest is 64: scale positions by 16
    scale = 64 // g["block_tokens"]
    ops = []
    for op in g["ops"]:
        op = dict(op)
        for key in ("split", "pos0", "n"):
            if key in op:
                op[key] = op[key] * scale
        if op["op"] == "expect_route":
            op["routes"] = [[r[0], r[1], r[2], r[3] * scale + d] for r in op["routes"] for d in range(scale)]
        if op["op"] == "expect_length":
            op["length"] *= scale
        ops.append(op)
    # appends add one position; scaled, each append becomes `scale` reserve rounds
    scaled = []
    for op in ops:
        if op["op"] == "append":
            scaled.extend([op] * scale)
        else:
            scaled.append(op)
    spec = _spec(max_seqs=4, max_seq_len=64 * 64, device_pool_blocks=g["device_blocks"],
                 host_pool_blocks=g["host_blocks"])
    h = wsk.wsk_init(spec, -1)
    try:
        _replay_golden(h, scaled)
    finally:
        wsk.wsk_destroy(h)


def test_routing_random_ops_match_oracle_model():
    rng = np.random.default_rng(3)
    bk, host_blocks, dev_blocks, max_seqs = 64, 40, 40, 6
    spec = _spec(max_seqs=max_seqs, max_seq_len=4096, device_pool_blocks=dev_blocks, host_pool_blocks=host_blocks)
    h = wsk.wsk_init(spec, -1)
    model = RouteModel(bk, host_blocks, dev_blocks)
    try:
        for step in range(400):
            sq = int(rng.integers(max_seqs))
            r = rng.random()
            try:
                if sq not in model.split:
                    split = int(rng.integers(0, 700))
                    model.open(sq, split)
                    wsk.wsk_seq_open(h, sq, split)
                elif r < 0.1:
                    model.close(sq)
                    wsk.wsk_seq_close(h, sq)
                else:
                    n = int(rng.integers(0, 300))
                    try:
                        model.write(sq, model.length[sq], n)
                        expect = None
                    except RouteError as ex:
                        expect = ex.code
                    try:
                        wsk.wsk_reserve(h, sq, n)
                        got = None
                    except wsk.WskError as ex:
                        got = ex.name
                    assert got == expect, step
            except RouteError:
                raise
            for s2 in model.split:
                L = model.length[s2]
                assert wsk.wsk_seq_info(h, s2) == (L, model.split[s2])
                for p in range(0, L, 7):
                    assert wsk.wsk_route(h, s2, p) == model.route(s2, p), (step, s2, p)
    finally:
        wsk.wsk_destroy(h)


def test_cpu_partition_bytes_land_at_routed_address():
    """CPU-partition rows are copied into the host pool at the slot/offset routing names,
    readable through the zero-copy view; the pool's other bytes stay zero."""
    rng = np.random.default_rng(5)
    spec = _spec(max_seqs=2, max_seq_len=1024, host_pool_blocks=8, device_pool_blocks=0)
    h = wsk.wsk_init(spec, -1)
    try:
        wsk.wsk_seq_open(h, 1, 300)
        wsk.wsk_seq_open(h, 0, 300)
        k = rng.integers(0, 65535, (150, 2, 128), dtype=np.uint16)
        v = rng.integers(0, 65535, (150, 2, 128), dtype=np.uint16)
        wsk.wsk_write(h, 1, 0, k[:70], v[:70])
        wsk.wsk_write(h, 0, 0, k[70:], v[70:])
        wsk.wsk_write(h, 1, 70, k[:5], v[:5])
        cpu, gpu = wsk.wsk_views(h, 1)
        assert (cpu.start, cpu.end, gpu.start, gpu.end) == (0, 75, 75, 75)
        assert cpu.is_device == 0 and not gpu.pool
        pool = np.ctypeslib.as_array(ctypes.cast(cpu.pool, ctypes.POINTER(ctypes.c_uint16)),
                                     shape=(8 * cpu.slot_bytes // 2,))
        touched = np.zeros(pool.shape, bool)
        for sq, rows_k, rows_v in ((1, np.concatenate([k[:70], k[:5]]), np.concatenate([v[:70], v[:5]])),
                                   (0, k[70:], v[70:])):
            cpu, _ = wsk.wsk_views(h, sq)
            for p in range(rows_k.shape[0]):
                part, blk, slot, off = wsk.wsk_route(h, sq, p)
                assert part == wsk.PART_CPU and cpu.table[blk] == slot and off == p % 64
                for g_ in range(2):
                    for which, src in ((0, rows_k), (1, rows_v)):
                        a = (slot * cpu.slot_bytes + g_ * cpu.head_bytes + which * cpu.v_bytes +
                             off * cpu.row_bytes) // 2
                        assert np.array_equal(pool[a:a + 128], src[p, g_])
                        touched[a:a + 128] = True
        assert not pool[~touched].any()
    finally:
        wsk.wsk_destroy(h)


def test_error_codes():
    h = wsk.wsk_init(_spec(host_pool_blocks=2, device_pool_blocks=2), -1)
    try:
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_seq_info(h, 0)
        assert ex.value.code == wsk.WSK_ESTATE
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_seq_open(h, 9, 0)
        assert ex.value.code == wsk.WSK_EINVAL
        wsk.wsk_seq_open(h, 0, 1000)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_seq_open(h, 0, 0)
        assert ex.value.code == wsk.WSK_ESTATE
        wsk.wsk_reserve(h, 0, 128)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_reserve(h, 0, 1)                      # third host block
        assert ex.value.code == wsk.WSK_ENOMEM
        assert wsk.wsk_seq_info(h, 0) == (128, 1000)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_route(h, 0, 128)
        assert ex.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_reserve(h, 0, 5000)
        assert ex.value.code == wsk.WSK_EINVAL
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_attend_workspace(h, [0], [0], [10])   # below the split
        assert ex.value.code == wsk.WSK_ERANGE
        assert wsk.wsk_attend_workspace(h, [0], [128], [128]) == 0
        wsk.wsk_seq_close(h, 0)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_route(h, 0, 0)
        assert ex.value.code == wsk.WSK_ESTATE
        lib = wsk.lib()
        assert lib.wsk_merge(-1, 128, None, None, None, None, None, None, None, None) == wsk.WSK_EINVAL
        assert lib.wsk_merge(4, 126, None, None, None, None, None, None, None, None) == wsk.WSK_EINVAL
        assert lib.wsk_merge(0, 128, None, None, None, None, None, None, None, None) == wsk.WSK_OK
        assert lib.wsk_mla_absorb(1, 16, 128, 500, None, None, None, 576, None) == wsk.WSK_EINVAL
        assert lib.wsk_mla_expand(1, 16, 512, 100, None, None, None, None) == wsk.WSK_EINVAL
        assert "width" in wsk.wsk_last_error() or wsk.wsk_last_error()
    finally:
        wsk.wsk_destroy(h)


def test_decode_step_mla_refusals():
    """The fused MLA step refuses a GQA cache, an unsupported dv and a NULL w_uv or o before any
    routing, and a host-only cache (no GPU) with ESTATE, leaving the sequence unchanged."""
    lib = wsk.lib()
    ids = (ctypes.c_int32 * 1)(0)
    g = wsk.wsk_init(_spec(), -1)
    try:
        wsk.wsk_seq_open(g, 0, 0)
        assert lib.wsk_decode_step_mla(g, 1, ids, 16, 16, None, None, 16, 128, None, 16, 16, 256, 1 << 20,
                                       None) == wsk.WSK_EINVAL
    finally:
        wsk.wsk_destroy(g)
    m = wsk.wsk_init(_spec(kind=wsk.KIND_MLA, n_q_heads=16, n_kv_heads=1, latent_dim=512, rope_dim=64,
                           softmax_scale=0.072), -1)
    try:
        wsk.wsk_seq_open(m, 0, 0)
        for dv, w_uv, o in ((100, 16, 16), (128, None, 16), (128, 24, 16), (128, 16, None)):
            assert lib.wsk_decode_step_mla(m, 1, ids, 16, 16, None, None, w_uv, dv, None, 16, o, 256, 1 << 20,
                                           None) == wsk.WSK_EINVAL, (dv, w_uv, o)
        assert lib.wsk_decode_step_mla(m, 1, ids, 16, 16, None, None, 16, 128, None, 16, 16, 256, 1 << 20,
                                       None) == wsk.WSK_ESTATE
        assert wsk.wsk_seq_info(m, 0)[0] == 0
    finally:
        wsk.wsk_destroy(m)


def test_workspace_grows_with_range_and_is_aligned():
    h = wsk.wsk_init(_spec(device_pool_blocks=64, max_seq_len=8192), -1)
    try:
        wsk.wsk_seq_open(h, 0, 0)
        wsk.wsk_reserve(h, 0, 4000)
        sizes = [wsk.wsk_attend_workspace(h, [0], [0], [e]) for e in (0, 1, 64, 65, 1000, 4000)]
        assert sizes[0] == 0 and all(b % 256 == 0 for b in sizes)
        assert sizes == sorted(sizes)
    finally:
        wsk.wsk_destroy(h)


def _segments_of(model, seq):
    """Runs of one home over [0, L) from the model's per-position homes."""
    out, homes = [], model.homes[seq]
    for p, part in enumerate(homes):
        if out and out[-1][2] == part and out[-1][1] == p:
            out[-1] = (out[-1][0], p + 1, part)
        else:
            out.append((p, p + 1, part))
    return out


def test_routing_with_load_region_matches_oracle_model():
    """Random open / open-with-load-range / reserve / close on a host-only cache
    with a load region: every route (part, block, slot, offset), the segment
    list and every refusal equal the oracle model's, bit for bit."""
    rng = np.random.default_rng(11)
    bk, host_blocks, dev_blocks, load_blocks, max_seqs = 64, 30, 30, 30, 5
    spec = _spec(max_seqs=max_seqs, max_seq_len=4096, device_pool_blocks=dev_blocks, host_pool_blocks=host_blocks)
    spec.load_pool_blocks, spec.load_arena_blocks, spec.pingpong_blocks = load_blocks, 7, 4
    h = wsk.wsk_init(spec, -1)
    model = RouteModel(bk, host_blocks, dev_blocks, load_blocks)
    try:
        for step in range(400):
            sq = int(rng.integers(max_seqs))
            if sq not in model.split:
                split = int(rng.integers(0, 600))
                load_end = split if rng.random() < 0.3 else int(rng.integers(split // bk, 14)) * bk
                if rng.random() < 0.1:
                    load_end = split + 1 + int(rng.integers(0, 60))       # unaligned: refused
                try:
                    model.open(sq, split, load_end)
                    expect = None
                except RouteError as ex:
                    expect = ex.code
                try:
                    wsk.wsk_seq_open_window(h, sq, split, load_end)
                    got = None
                except wsk.WskError as ex:
                    got = ex.name
                assert got == expect, (step, split, load_end)
            elif rng.random() < 0.1:
                model.close(sq)
                wsk.wsk_seq_close(h, sq)
            else:
                n = int(rng.integers(0, 300))
                try:
                    model.write(sq, model.length[sq], n)
                    expect = None
                except RouteError as ex:
                    expect = ex.code
                try:
                    wsk.wsk_reserve(h, sq, n)
                    got = None
                except wsk.WskError as ex:
                    got = ex.name
                assert got == expect, step
            for s2 in model.split:
                L = model.length[s2]
                assert wsk.wsk_seq_info(h, s2) == (L, model.split[s2])
                assert wsk.wsk_seq_segments(h, s2) == _segments_of(model, s2), (step, s2)
                for p in range(0, L, 5):
                    assert wsk.wsk_route(h, s2, p) == model.route(s2, p), (step, s2, p)
        assert wsk.wsk_load_stats(h).slots_used == load_blocks - len(model.free[2])
    finally:
        wsk.wsk_destroy(h)
