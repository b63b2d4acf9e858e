"""The CPU engine (wsk_cpu_attend) against the fp64 oracle, on the CPU: the
CPU partition of a host-only cache is attended in place, GQA and MLA, over
unaligned, single-token, empty and chunk-crossing ranges, block sizes 64 to
256; the tolerance is the one the GPU path meets (max_abs 1e-2, L1 ratio
1e-3, LSE 1e-4)."""
import numpy as np
import pytest

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from tests.gpu_util import assert_close, assert_lse


def _cache(w, lengths, bk, seed):
    """Host-only cache holding every position on the CPU side (s = L)."""
    gen = __import__("torch").Generator().manual_seed(seed)
    blocks = sum(-(-L // bk) for L in lengths)
    if w.kind == wl.MLA:
        spec = wsk.make_spec(wsk.KIND_MLA, w.n_q_heads, 1, w.head_dim, bk, len(lengths), max(lengths), 0, blocks,
                             w.softmax_scale, latent_dim=w.latent_dim, rope_dim=w.rope_dim)
    else:
        spec = wsk.make_spec(wsk.KIND_GQA, w.n_q_heads, w.n_kv_heads, w.head_dim, bk, len(lengths), max(lengths), 0,
                             blocks, w.softmax_scale)
    h = wsk.wsk_init(spec, -1)
    ks, vs = [], []
    for b, L in enumerate(lengths):
        wsk.wsk_seq_open(h, b, L)
        if w.kind == wl.MLA:
            k = wl.draw_bf16(gen, (L, w.row_elems), w.kv_std)
            v = None
        else:
            k = wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim))
            v = wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim))
        wsk.wsk_write(h, b, 0, k, v)
        ks.append(k)
        vs.append(v)
    q = wl.draw_bf16(gen, (len(lengths), w.n_q_heads, w.row_elems))
    return h, ks, vs, q


def _check(w, h, ks, vs, q, ranges, threads):
    n = len(ranges)
    dv = w.latent_dim if w.kind == wl.MLA else w.head_dim
    o = np.empty((n, w.n_q_heads, dv), np.float32)
    lse = np.empty((n, w.n_q_heads), np.float32)
    ids = [b for b, _ in ranges]
    wsk.wsk_cpu_attend(h, ids, [a for _, (a, e) in ranges], [e for _, (a, e) in ranges],
                       np.ascontiguousarray(q[ids]), o, lse, threads)
    g = w.n_q_heads if w.kind == wl.MLA else w.group
    for j, (b, (a, e)) in enumerate(ranges):
        if e == a:
            assert np.all(o[j] == 0) and np.all(np.isneginf(lse[j]))
            continue
        o_r, l_r = oracle.attend(q[b], ks[b], vs[b], a, e, w.softmax_scale, g, dv=dv)
        assert_close(o[j], o_r, "cpu engine b%d [%d,%d)" % (b, a, e))
        assert_lse(lse[j], l_r, "cpu engine b%d [%d,%d)" % (b, a, e))


@pytest.mark.parametrize("Hq,Hkv,bk", [(8, 2, 64), (32, 4, 128), (4, 4, 256), (12, 4, 64)])
def test_cpu_engine_gqa(Hq, Hkv, bk):
    w = wl.Workload("cpu-gqa", wl.GQA, batch=3, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=128, context=5000)
    lengths = [5000, 130, 1]
    h, ks, vs, q = _cache(w, lengths, bk, Hq * 7 + bk)
    try:
        _check(w, h, ks, vs, q, [(0, (0, 5000)), (1, (3, 130)), (2, (0, 1))], 4)
        _check(w, h, ks, vs, q, [(0, (2047, 4100)), (1, (64, 64)), (0, (4999, 5000)), (0, (0, 5000))], 1)
    finally:
        wsk.wsk_destroy(h)


@pytest.mark.parametrize("H,bk", [(16, 64), (5, 128)])
def test_cpu_engine_mla(H, bk):
    w = wl.Workload("cpu-mla", wl.MLA, batch=2, n_q_heads=H, n_kv_heads=1, head_dim=128, latent_dim=512,
                    rope_dim=64, nope_dim=128, context=2500, kv_std=0.5)
    h, ks, vs, q = _cache(w, [2500, 70], bk, H + bk)
    try:
        _check(w, h, ks, vs, q, [(0, (0, 2500)), (1, (1, 69))], 3)
        _check(w, h, ks, vs, q, [(0, (2047, 2049)), (1, (5, 5))], 1)
    finally:
        wsk.wsk_destroy(h)


def test_cpu_engine_errors():
    w = wl.Workload("cpu-gqa", wl.GQA, batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, context=100)
    h, ks, vs, q = _cache(w, [100], 64, 1)
    try:
        o = np.empty((1, 8, 128), np.float32)
        lse = np.empty((1, 8), np.float32)
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_cpu_attend(h, [0], [0], [101], np.ascontiguousarray(q), o, lse)
        assert ei.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_cpu_attend(h, [1], [0], [1], np.ascontiguousarray(q), o, lse)
        assert ei.value.code in (wsk.WSK_EINVAL, wsk.WSK_ESTATE)
    finally:
        wsk.wsk_destroy(h)


@pytest.mark.parametrize("nbytes", [8, 8000, (5 << 20) + 8, 3 << 22])
def test_host_read_probe_folds_every_word(nbytes):
    """wsk_host_read reads every 64-bit word once (its XOR equals numpy's),
    whole 4 MiB pieces and ragged tails alike, on any thread count."""
    a = np.random.default_rng(nbytes).integers(0, 2 ** 63, size=nbytes // 8, dtype=np.uint64)
    want = int(np.bitwise_xor.reduce(a))
    for threads in (1, 3, 0):
        assert wsk.wsk_host_read(a, threads) == want
    with pytest.raises(wsk.WskError):
        wsk.wsk_host_read(np.zeros(3, np.uint8))
