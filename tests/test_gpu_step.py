"""wsk_decode_step (append + GPU-side attention + merge in one call) against
the fp64 oracle over the whole context, step after step across block
boundaries, GQA and MLA, HBM-resident and with a load region; the pool it
leaves behind is byte-identical to the one wsk_append leaves; and its
refusals change nothing."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
from tests.gpu_util import assert_close, assert_lse, d2h, say

pytestmark = pytest.mark.gpu
DEV = 0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(DEV)
    yield
    torch.cuda.synchronize()


def _workload(kind, B, H, seed):
    if kind == "gqa":
        return wl.Workload("step-gqa", wl.GQA, batch=B, n_q_heads=H, n_kv_heads=2, head_dim=128, context=1,
                           seed=seed)
    return wl.Workload("step-mla", wl.MLA, batch=B, n_q_heads=H, n_kv_heads=1, head_dim=128, latent_dim=512,
                       rope_dim=64, nope_dim=128, context=1, kv_std=0.5, seed=seed)


def _prefill(w, lengths, splits, gen):
    if w.kind == wl.MLA:
        return wl.Prefill(list(lengths), list(splits), [wl.draw_bf16(gen, (L, w.row_elems), w.kv_std) for L in lengths],
                          None, gen)
    return wl.Prefill(list(lengths), list(splits),
                      [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths],
                      [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths], gen)


def _new_rows(w, B, gen):
    if w.kind == wl.MLA:
        return wl.draw_bf16(gen, (B, w.row_elems), w.kv_std), None
    return wl.draw_bf16(gen, (B, w.n_kv_heads, w.head_dim)), wl.draw_bf16(gen, (B, w.n_kv_heads, w.head_dim))


def _dims(w):
    return (w.latent_dim if w.kind == wl.MLA else w.head_dim), (w.n_q_heads if w.kind == wl.MLA else w.group)


def _cpu_partial(sess, q_bits):
    w = sess.w
    dv, _ = _dims(w)
    o = np.empty((sess.B, w.n_q_heads, dv), np.float32)
    lse = np.empty((sess.B, w.n_q_heads), np.float32)
    wsk.wsk_cpu_attend_all(sess.h, sess.ids, np.ascontiguousarray(q_bits), o, lse, 8)
    return torch.from_numpy(o).to(sess.dev), torch.from_numpy(lse).to(sess.dev)


def _step(sess, q, kn, vn, o_x, l_x):
    need = wsk.wsk_decode_step_workspace(sess.h, sess.ids)
    ws = torch.empty(need, dtype=torch.uint8, device=sess.dev)
    dv, _ = _dims(sess.w)
    o = torch.empty(sess.B, sess.w.n_q_heads, dv, device=sess.dev)
    lse = torch.empty(sess.B, sess.w.n_q_heads, device=sess.dev)
    wsk.wsk_decode_step(sess.h, sess.ids, q, kn, vn, o, lse, ws, o_x, l_x)
    for b in sess.ids:
        sess.lengths[b] += 1
    return o, lse


def _gpu_pool(sess):
    _, gv = wsk.wsk_views(sess.h, 0)
    return d2h(gv.pool, gv.slot_bytes * sess.spec.device_pool_blocks)


@pytest.mark.parametrize("kind,bk,load", [("gqa", 64, False), ("gqa", 128, True), ("mla", 64, False),
                                          ("mla", 256, True)])
def test_decode_steps(kind, bk, load):
    """Six steps from prefills that end 3 positions before a block boundary
    (so that a step opens a new block), a sequence with no CPU part, a D-window
    that starts inside a block and (with a load region) one that starts
    empty; each step's output against the oracle over [0, L]; a twin cache
    driven by wsk_append + wsk_attend_gpu ends with a byte-identical GPU pool
    and close outputs."""
    lengths = [4 * bk - 3, 2 * bk - 3, 3 * bk]
    splits = [bk + 11, 0, 2 * bk + 5]
    load_ends = [3 * bk, bk, 3 * bk] if load else None
    w = _workload(kind, len(lengths), 8, seed=bk)
    gen = torch.Generator().manual_seed(w.seed + 3)
    pf = _prefill(w, lengths, splits, gen)
    k_all = list(pf.k)
    v_all = None if pf.v is None else list(pf.v)
    dv, g = _dims(w)
    say("case decode step", kind, bk, load)
    kw = dict(extra_tokens=8, block_tokens=bk, load_ends=load_ends, pingpong_blocks=2, arena_blocks=3)
    with DecodeSession(w, pf, DEV, **kw) as sess, DecodeSession(w, pf, DEV, **kw) as twin:
        for step in range(6):
            q_bits = wl.draw_bf16(gen, (sess.B, w.n_q_heads, w.row_elems))
            kn, vn = _new_rows(w, sess.B, gen)
            q = to_device_bf16(q_bits, sess.dev)
            knd = to_device_bf16(kn, sess.dev)
            vnd = None if vn is None else to_device_bf16(vn, sess.dev)
            o_x, l_x = _cpu_partial(sess, q_bits)
            o, lse = _step(sess, q, knd, vnd, o_x, l_x)
            twin.append(knd, vnd)
            o2, lse2 = twin.attend_gpu(q, o_x=o_x, lse_x=l_x)
            for b in range(sess.B):
                k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                if v_all is not None:
                    v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
            o, lse, o2, lse2 = (t.cpu().numpy() for t in (o, lse, o2, lse2))
            for b in range(sess.B):
                L = sess.lengths[b]
                o_r, l_r = oracle.attend(q_bits[b], k_all[b], None if v_all is None else v_all[b], 0, L,
                                         w.softmax_scale, g, dv=dv)
                assert_close(o[b], o_r, "step %d b%d" % (step, b))
                assert_lse(lse[b], l_r, "step %d b%d" % (step, b))
                assert np.abs(o[b] - o2[b]).max() <= 1e-5 and np.abs(lse[b] - lse2[b]).max() <= 1e-5
        torch.cuda.synchronize()
        assert np.array_equal(_gpu_pool(sess), _gpu_pool(twin))
        for b in range(sess.B):
            for p in range(0, sess.lengths[b], 7):
                assert wsk.wsk_route(sess.h, b, p) == wsk.wsk_route(twin.h, b, p)


def test_decode_step_many_sequences_and_refusals():
    B = 70
    w = _workload("gqa", B, 8, seed=4)
    gen = torch.Generator().manual_seed(6)
    lengths = [int(x) for x in torch.randint(60, 300, (B,), generator=gen)]
    splits = [L // 3 for L in lengths]
    pf = _prefill(w, lengths, splits, gen)
    k_all, v_all = list(pf.k), list(pf.v)
    dv, g = _dims(w)
    say("case decode step many")
    with DecodeSession(w, pf, DEV, extra_tokens=2) as sess:
        q_bits = wl.draw_bf16(gen, (B, w.n_q_heads, w.row_elems))
        kn, vn = _new_rows(w, B, gen)
        q, knd, vnd = (to_device_bf16(x, sess.dev) for x in (q_bits, kn, vn))
        o, lse = _step(sess, q, knd, vnd, None, None)
        o, lse = o.cpu().numpy(), lse.cpu().numpy()
        for b in range(B):
            k = np.concatenate([k_all[b], kn[b:b + 1]])
            v = np.concatenate([v_all[b], vn[b:b + 1]])
            o_r, l_r = oracle.attend(q_bits[b], k, v, splits[b], lengths[b] + 1, w.softmax_scale, g, dv=dv)
            assert_close(o[b], o_r, "many b%d" % b)
            assert_lse(lse[b], l_r, "many b%d" % b)
        ws = torch.empty(wsk.wsk_decode_step_workspace(sess.h, sess.ids), dtype=torch.uint8, device=sess.dev)
        o_t = torch.empty(2, w.n_q_heads, dv, device=sess.dev)
        l_t = torch.empty(2, w.n_q_heads, device=sess.dev)
        before = [wsk.wsk_seq_info(sess.h, b)[0] for b in range(2)]
        with pytest.raises(wsk.WskError) as ei:                    # a sequence listed twice
            wsk.wsk_decode_step(sess.h, [1, 1], q[:2], knd[:2], vnd[:2], o_t, l_t, ws)
        assert ei.value.code == wsk.WSK_EINVAL
        with pytest.raises(wsk.WskError) as ei:                    # workspace too small
            wsk.wsk_decode_step(sess.h, [0, 1], q[:2], knd[:2], vnd[:2], o_t, l_t, ws[:256])
        assert ei.value.code == wsk.WSK_EINVAL
        assert [wsk.wsk_seq_info(sess.h, b)[0] for b in range(2)] == before


@pytest.mark.parametrize("all_gpu", [True, False])
def test_decode_step_full_launch_two_head_groups(all_gpu):
    """GQA decode steps over 64 sequences (the most one launch takes) with 32
    query heads per KV head (two head groups share each KV head and its new
    row), ragged lengths, steps with and without the CPU partial, against the
    oracle and against a twin cache driven by wsk_append + wsk_attend_gpu:
    close outputs, byte-identical pools, every step.  all_gpu=False adds a
    sequence whose GPU range is empty before the first step."""
    B = 64
    w = _workload("gqa", B, 64, seed=21)
    gen = torch.Generator().manual_seed(23)
    lengths = [int(x) for x in torch.randint(40, 400, (B,), generator=gen)]
    splits = [L // 3 for L in lengths]
    if not all_gpu:
        splits[5] = lengths[5]
    pf = _prefill(w, lengths, splits, gen)
    k_all, v_all = list(pf.k), list(pf.v)
    dv, g = _dims(w)
    say("case decode step full launch", all_gpu)
    with DecodeSession(w, pf, DEV, extra_tokens=4) as sess, DecodeSession(w, pf, DEV, extra_tokens=4) as twin:
        for step in range(3):
            q_bits = wl.draw_bf16(gen, (B, w.n_q_heads, w.row_elems))
            kn, vn = _new_rows(w, B, gen)
            q, knd, vnd = (to_device_bf16(x, sess.dev) for x in (q_bits, kn, vn))
            o_x, l_x = (None, None) if step == 0 else _cpu_partial(sess, q_bits)
            o, lse = _step(sess, q, knd, vnd, o_x, l_x)
            twin.append(knd, vnd)
            o2, lse2 = twin.attend_gpu(q, o_x=o_x, lse_x=l_x)
            for b in range(B):
                k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
            o, lse, o2, lse2 = (t.cpu().numpy() for t in (o, lse, o2, lse2))
            for b in range(B):
                lo = 0 if o_x is not None else splits[b]
                o_r, l_r = oracle.attend(q_bits[b], k_all[b], v_all[b], lo, sess.lengths[b], w.softmax_scale, g,
                                         dv=dv)
                assert_close(o[b], o_r, "full launch step %d b%d" % (step, b))
                assert_lse(lse[b], l_r, "full launch step %d b%d" % (step, b))
            assert np.abs(o - o2).max() <= 1e-5 and np.abs(lse - lse2).max() <= 1e-5
            torch.cuda.synchronize()
            assert np.array_equal(_gpu_pool(sess), _gpu_pool(twin))


@pytest.mark.parametrize("kind", ["gqa", "mla"])
def test_decode_loop_with_policy_eviction(kind):
    """300 decode steps through wsk_decode_step on a cache whose GPU share
    starts in the load region; whenever a D-window holds a whole batch it is
    evicted where the split policy routes it (CPU partition or load region);
    every 50 steps the whole step -- CPU engine over every CPU position,
    GPU side streamed and in place, the new row -- is checked against the
    oracle over [0, L]."""
    from oracle import policy as P
    bk, D, steps = 64, 128, 300
    lengths, splits, load_ends = [1500, 900], [300, 0], [1408, 768]
    w = _workload(kind, 2, 8, seed=13)
    gen = torch.Generator().manual_seed(17)
    pf = _prefill(w, lengths, splits, gen)
    k_all = list(pf.k)
    v_all = None if pf.v is None else list(pf.v)
    dv, g = _dims(w)
    A, Bc = 3e-9, 2e-9                                   # p = 0.4
    pol = wsk.Policy(A, Bc, 1e-5, 1e-5, 4)
    say("case decode loop", kind)
    try:
        with DecodeSession(w, pf, DEV, extra_tokens=steps, block_tokens=bk, load_ends=load_ends, evict_tokens=D,
                           pingpong_blocks=5, arena_blocks=6) as sess:
            flushed = {wsk.PART_CPU: 0, wsk.PART_LOAD: 0}
            for step in range(steps):
                q_bits = wl.draw_bf16(gen, (2, w.n_q_heads, w.row_elems))
                kn, vn = _new_rows(w, 2, gen)
                q = to_device_bf16(q_bits, sess.dev)
                o_x, l_x = _cpu_partial(sess, q_bits)
                o, lse = sess.decode_step(q, to_device_bf16(kn, sess.dev),
                                          None if vn is None else to_device_bf16(vn, sess.dev), o_x=o_x, lse_x=l_x)
                for b in range(2):
                    k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                    if v_all is not None:
                        v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
                if step % 50 == 49:
                    o, lse = o.cpu().numpy(), lse.cpu().numpy()
                    for b in range(2):
                        o_r, l_r = oracle.attend(q_bits[b], k_all[b], None if v_all is None else v_all[b], 0,
                                                 sess.lengths[b], w.softmax_scale, g, dv=dv)
                        assert_close(o[b], o_r, "loop step %d b%d" % (step, b))
                        assert_lse(lse[b], l_r, "loop step %d b%d" % (step, b))
                for b in range(2):
                    a, e = sess.gpu_range(b)
                    if e - a >= D + (-a) % bk:
                        dest = wsk.PART_CPU if pol.route() == wsk.PART_CPU else wsk.PART_LOAD
                        assert sess.flush([dest], ids=[b]) == [(a + D) // bk * bk - a]
                        flushed[dest] += 1
            assert flushed[wsk.PART_CPU] > 0 and flushed[wsk.PART_LOAD] > 0
            p = P.marginal_share(A, Bc)
            n = sum(flushed.values())
            assert abs(flushed[wsk.PART_CPU] / n - p) <= 0.5 / n + 1e-12
    finally:
        pol.close()


@pytest.mark.parametrize("H,bk,dv,load", [(16, 64, 128, False), (5, 256, 64, True), (16, 128, 256, False)])
def test_decode_step_mla_expand(H, bk, dv, load):
    """wsk_decode_step_mla: the merged latent output and LSE against the oracle over [0, L], the
    expanded output against the oracle's expansion of the exact latent output (Sec. 6.1), the latent
    output within 1e-5 of wsk_decode_step's on a twin cache, the GPU pool byte-identical to the
    twin's after every step (the fused kernel stores the new row as pass 2 does), and o_lat = NULL
    leaving the expanded output unchanged."""
    lengths = [4 * bk - 3, 2 * bk - 3, 3 * bk]
    splits = [bk + 11, 0, 2 * bk + 5]
    load_ends = [3 * bk, bk, 3 * bk] if load else None
    w = _workload("mla", len(lengths), H, seed=bk + dv)
    w = wl.Workload(w.name, w.kind, batch=w.batch, n_q_heads=H, n_kv_heads=1, head_dim=dv, latent_dim=512,
                    rope_dim=64, nope_dim=128, context=1, kv_std=0.5, seed=w.seed)
    gen = torch.Generator().manual_seed(w.seed + 5)
    pf = _prefill(w, lengths, splits, gen)
    rows_all = list(pf.k)
    _, w_uv = wl.draw_mla_weights(w, gen)
    say("case decode step mla expand H=%d bk=%d dv=%d load=%s" % (H, bk, dv, load))
    kw = dict(extra_tokens=8, block_tokens=bk, load_ends=load_ends, pingpong_blocks=2, arena_blocks=3)
    with DecodeSession(w, pf, DEV, **kw) as sess, DecodeSession(w, pf, DEV, **kw) as twin:
        w_uv_d = to_device_bf16(w_uv, sess.dev)
        for step in range(5):
            q_bits = wl.draw_bf16(gen, (sess.B, H, w.row_elems))
            kn, _ = _new_rows(w, sess.B, gen)
            q = to_device_bf16(q_bits, sess.dev)
            knd = to_device_bf16(kn, sess.dev)
            o_x, l_x = _cpu_partial(sess, q_bits)
            ws = torch.empty(wsk.wsk_decode_step_workspace(sess.h, sess.ids), dtype=torch.uint8, device=sess.dev)
            o_lat = torch.empty(sess.B, H, 512, device=sess.dev)
            lse = torch.empty(sess.B, H, device=sess.dev)
            o = torch.empty(sess.B, H, dv, device=sess.dev)
            keep = step == 3   # this step without o_lat: o and lse only
            wsk.wsk_decode_step_mla(sess.h, sess.ids, q, knd, w_uv_d, o, lse, ws, o_lat=None if keep else o_lat,
                                    o_x=o_x, lse_x=l_x)
            for b in sess.ids:
                sess.lengths[b] += 1
            o2, lse2 = _step(twin, q, knd, None, o_x, l_x)
            for b in range(sess.B):
                rows_all[b] = np.concatenate([rows_all[b], kn[b:b + 1]])
            o, lse, o_lat, o2, lse2 = (t.cpu().numpy() for t in (o, lse, o_lat, o2, lse2))
            for b in range(sess.B):
                L = sess.lengths[b]
                ol_r, l_r = oracle.attend(q_bits[b], rows_all[b], None, 0, L, w.softmax_scale, H, dv=512)
                assert_lse(lse[b], l_r, "mla expand step %d b%d" % (step, b))
                assert_close(o[b], oracle.mla_expand(ol_r, w_uv), "mla expand O step %d b%d" % (step, b))
                if not keep:
                    assert_close(o_lat[b], ol_r, "mla expand O_lat step %d b%d" % (step, b))
                    assert np.abs(o_lat[b] - o2[b]).max() <= 1e-5
                assert np.abs(lse[b] - lse2[b]).max() <= 1e-5
            torch.cuda.synchronize()
            assert np.array_equal(_gpu_pool(sess), _gpu_pool(twin)), "pool differs after step %d" % step


@pytest.mark.parametrize("dv", [128, 256])
def test_decode_step_mla_expand_many_sequences_and_refusals(dv):
    """70 MLA sequences (two pass-2 launches, outputs at their offsets) through wsk_decode_step_mla
    against the oracle; a sequence listed twice and a short workspace are refused with nothing
    changed.  The launch of 64 sequences expands each (sequence, head) in one workgroup, that of
    the other 6 in slices of dv / 2 columns (with dv = 256: every slice width the kernel has, with
    the three-sequence cases above)."""
    B, H = 70, 16
    w = _workload("mla", B, H, seed=9)
    w = wl.Workload(w.name, w.kind, batch=w.batch, n_q_heads=H, n_kv_heads=1, head_dim=dv, latent_dim=512,
                    rope_dim=64, nope_dim=128, context=1, kv_std=0.5, seed=w.seed)
    gen = torch.Generator().manual_seed(10)
    lengths = [int(x) for x in torch.randint(60, 300, (B,), generator=gen)]
    splits = [L // 3 for L in lengths]
    pf = _prefill(w, lengths, splits, gen)
    _, w_uv = wl.draw_mla_weights(w, gen)
    say("case decode step mla expand many")
    with DecodeSession(w, pf, DEV, extra_tokens=2) as sess:
        q_bits = wl.draw_bf16(gen, (B, H, w.row_elems))
        kn, _ = _new_rows(w, B, gen)
        q, knd, w_uv_d = (to_device_bf16(x, sess.dev) for x in (q_bits, kn, w_uv))
        ws = torch.empty(wsk.wsk_decode_step_workspace(sess.h, sess.ids), dtype=torch.uint8, device=sess.dev)
        o = torch.empty(B, H, dv, device=sess.dev)
        o_lat = torch.empty(B, H, 512, device=sess.dev)
        lse = torch.empty(B, H, device=sess.dev)
        wsk.wsk_decode_step_mla(sess.h, sess.ids, q, knd, w_uv_d, o, lse, ws, o_lat=o_lat)
        o, o_lat, lse = o.cpu().numpy(), o_lat.cpu().numpy(), lse.cpu().numpy()
        for b in range(B):
            rows = np.concatenate([pf.k[b], kn[b:b + 1]])
            ol_r, l_r = oracle.attend(q_bits[b], rows, None, splits[b], lengths[b] + 1, w.softmax_scale, H, dv=512)
            assert_close(o_lat[b], ol_r, "mla many O_lat b%d" % b)
            assert_close(o[b], oracle.mla_expand(ol_r, w_uv), "mla many O b%d" % b)
            assert_lse(lse[b], l_r, "mla many b%d" % b)
        o_t = torch.empty(2, H, dv, device=sess.dev)
        l_t = torch.empty(2, H, device=sess.dev)
        before = [wsk.wsk_seq_info(sess.h, b)[0] for b in range(2)]
        with pytest.raises(wsk.WskError) as ei:                    # a sequence listed twice
            wsk.wsk_decode_step_mla(sess.h, [1, 1], q[:2], knd[:2], w_uv_d, o_t, l_t, ws)
        assert ei.value.code == wsk.WSK_EINVAL
        with pytest.raises(wsk.WskError) as ei:                    # workspace too small
            wsk.wsk_decode_step_mla(sess.h, [0, 1], q[:2], knd[:2], w_uv_d, o_t, l_t, ws[:256])
        assert ei.value.code == wsk.WSK_EINVAL
        assert [wsk.wsk_seq_info(sess.h, b)[0] for b in range(2)] == before


def test_decode_step_mla_expand_empty_gpu_side():
    """Sequences whose GPU side holds nothing before the step (split = L: pass 1 has no chunk for
    them, so pass 2 merges only the new row and the CPU partial) beside ordinary ones, through
    wsk_decode_step_mla, against the oracle over [0, L]."""
    H, dv = 16, 128
    lengths = [200, 130, 64, 300]
    splits = [200, 0, 64, 150]          # sequences 0 and 2: every cached position on the CPU side
    w = _workload("mla", len(lengths), H, seed=31)
    gen = torch.Generator().manual_seed(32)
    pf = _prefill(w, lengths, splits, gen)
    _, w_uv = wl.draw_mla_weights(w, gen)
    say("case decode step mla expand, empty GPU side")
    with DecodeSession(w, pf, DEV, extra_tokens=2) as sess:
        q_bits = wl.draw_bf16(gen, (sess.B, H, w.row_elems))
        kn, _ = _new_rows(w, sess.B, gen)
        q, knd, w_uv_d = (to_device_bf16(x, sess.dev) for x in (q_bits, kn, w_uv))
        o_x, l_x = _cpu_partial(sess, q_bits)
        ws = torch.empty(wsk.wsk_decode_step_workspace(sess.h, sess.ids), dtype=torch.uint8, device=sess.dev)
        o = torch.empty(sess.B, H, dv, device=sess.dev)
        o_lat = torch.empty(sess.B, H, 512, device=sess.dev)
        lse = torch.empty(sess.B, H, device=sess.dev)
        wsk.wsk_decode_step_mla(sess.h, sess.ids, q, knd, w_uv_d, o, lse, ws, o_lat=o_lat, o_x=o_x, lse_x=l_x)
        o, o_lat, lse = o.cpu().numpy(), o_lat.cpu().numpy(), lse.cpu().numpy()
        for b in range(sess.B):
            rows = np.concatenate([pf.k[b], kn[b:b + 1]])
            ol_r, l_r = oracle.attend(q_bits[b], rows, None, 0, lengths[b] + 1, w.softmax_scale, H, dv=512)
            assert_close(o_lat[b], ol_r, "empty-side O_lat b%d" % b)
            assert_close(o[b], oracle.mla_expand(ol_r, w_uv), "empty-side O b%d" % b)
            assert_lse(lse[b], l_r, "empty-side b%d" % b)


def test_decode_step_flat_split_many_short_one_long():
    """A batch the per-sequence chunking handles badly: 70 sequences (two launches), most with a
    few GPU-side tiles, one of ~610 tiles in each launch, and one with nothing on the GPU side
    before the step.  Every non-empty range starting with a chunk of its own leaves the first
    launch's long sequence a single chunk, so the planner takes the flat split there (its runs
    cross from short sequence to short sequence, several segments per workgroup); the premise is
    asserted from the workspace size (the flat split writes more partials).  Two decode steps
    against the fp64 oracle, and a twin cache driven by wsk_append + wsk_attend_gpu (pass 1 alone,
    the same split) with close outputs and a byte-identical pool."""
    B, H = 70, 8
    gen = torch.Generator().manual_seed(51)
    lengths = [int(x) for x in torch.randint(100, 330, (B,), generator=gen)]
    splits = [int(x) for x in torch.randint(0, 64, (B,), generator=gen)]
    for b in (3, 66):
        lengths[b], splits[b] = 40000, 1000
    lengths[9], splits[9] = 700, 700          # nothing on the GPU side before the first step
    w = wl.Workload("step-gqa-flat", wl.GQA, batch=B, n_q_heads=H, n_kv_heads=4, head_dim=128, context=1, seed=52)
    pf = _prefill(w, lengths, splits, gen)
    k_all, v_all = list(pf.k), list(pf.v)
    dv, g = _dims(w)
    say("case decode step, flat split")
    with DecodeSession(w, pf, DEV, extra_tokens=3) as sess, DecodeSession(w, pf, DEV, extra_tokens=3) as twin:
        need = wsk.wsk_decode_step_workspace(sess.h, sess.ids)
        r256 = lambda x: (x + 255) // 256 * 256
        partials = max(p for p in range(1, 8192) if r256(p * H * dv * 4) + r256(p * H * 4) <= need)
        say("  %d chunk partials (one per range would be %d)" % (partials, B))
        assert partials >= B + 20, partials
        for step in range(2):
            q_bits = wl.draw_bf16(gen, (B, H, w.row_elems))
            kn, vn = _new_rows(w, B, gen)
            q, knd, vnd = (to_device_bf16(x, sess.dev) for x in (q_bits, kn, vn))
            o_x, l_x = _cpu_partial(sess, q_bits)
            o, lse = _step(sess, q, knd, vnd, o_x, l_x)
            twin.append(knd, vnd)
            o2, lse2 = twin.attend_gpu(q, o_x=o_x, lse_x=l_x)
            o, lse, o2, lse2 = (t.cpu().numpy() for t in (o, lse, o2, lse2))
            for b in range(B):
                k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
                o_r, l_r = oracle.attend(q_bits[b], k_all[b], v_all[b], 0, sess.lengths[b], w.softmax_scale, g,
                                         dv=dv)
                assert_close(o[b], o_r, "flat split step %d b%d" % (step, b))
                assert_lse(lse[b], l_r, "flat split step %d b%d" % (step, b))
            assert np.abs(o - o2).max() <= 1e-5 and np.abs(lse - lse2).max() <= 1e-5
            torch.cuda.synchronize()
            assert np.array_equal(_gpu_pool(sess), _gpu_pool(twin))


def test_decode_step_more_chunks_than_weights_kept():
    """GQA decode step with one KV head (one (KV head, head group) unit, so the whole grid serves
    one sequence): a long sequence cut into more than 64 chunk partials -- more than the weights
    the last workgroup keeps per head and more than the partials it loads before the merge, so
    both of its loops over the rest run -- and a short one, against the oracle; the chunk count
    is read back from the workspace size, so the premise is asserted."""
    H = 8
    lengths = [20100, 700]
    splits = [37, 130]
    w = wl.Workload("step-gqa-one-kv-head", wl.GQA, batch=len(lengths), n_q_heads=H, n_kv_heads=1, head_dim=128,
                    context=1, seed=43)
    gen = torch.Generator().manual_seed(44)
    pf = _prefill(w, lengths, splits, gen)
    dv, g = _dims(w)
    say("case decode step, more chunks than weights kept")
    with DecodeSession(w, pf, DEV, extra_tokens=2) as sess:
        for step in range(2):
            q_bits = wl.draw_bf16(gen, (sess.B, H, w.row_elems))
            kn, vn = _new_rows(w, sess.B, gen)
            need = wsk.wsk_decode_step_workspace(sess.h, sess.ids)
            r256 = lambda x: (x + 255) // 256 * 256
            partials = max(p for p in range(1, 4096) if r256(p * H * dv * 4) + r256(p * H * 4) <= need)
            short_tiles = -(-(lengths[1] + step) // 64) - splits[1] // 64
            say("  step %d: %d chunk partials in all" % (step, partials))
            assert partials - -(-short_tiles // 4) > 64, partials
            o_x, l_x = _cpu_partial(sess, q_bits)
            out, lse = _step(sess, to_device_bf16(q_bits, sess.dev), to_device_bf16(kn, sess.dev),
                             to_device_bf16(vn, sess.dev), o_x, l_x)
            out, lse = out.cpu().numpy(), lse.cpu().numpy()
            for b in range(sess.B):
                pf.k[b] = np.concatenate([pf.k[b], kn[b:b + 1]])
                pf.v[b] = np.concatenate([pf.v[b], vn[b:b + 1]])
                o_r, l_r = oracle.attend(q_bits[b], pf.k[b], pf.v[b], 0, sess.lengths[b], w.softmax_scale, g,
                                         dv=dv)
                assert_close(out[b], o_r, "more than 64 chunks step %d b%d" % (step, b))
                assert_lse(lse[b], l_r, "more than 64 chunks step %d b%d" % (step, b))


@pytest.mark.parametrize("kind", ["gqa", "mla"])
def test_decode_step_more_chunks_than_loaded_up_front(kind):
    """One long sequence (41 chunk partials on a 256-CU device: more than the 32 that pass 2 loads
    before using any, so its loop over the rest runs) and a short one (at most 2 chunks), through
    wsk_decode_step (GQA) and wsk_decode_step_mla (MLA), against the oracle.  The chunk count is
    read back from the workspace size (fp32 O [partials][H][width] then LSE [partials][H], each
    rounded up to 256 bytes), so the premise is asserted, not assumed."""
    H = 16 if kind == "mla" else 8
    lengths = [10300, 500]
    splits = [60, 100]
    w = _workload(kind, len(lengths), H, seed=41)
    gen = torch.Generator().manual_seed(42)
    pf = _prefill(w, lengths, splits, gen)
    dv, g = _dims(w)
    say("case decode step, more chunks than loaded up front", kind)
    with DecodeSession(w, pf, DEV, extra_tokens=2) as sess:
        q_bits = wl.draw_bf16(gen, (sess.B, H, w.row_elems))
        kn, vn = _new_rows(w, sess.B, gen)
        q, knd = to_device_bf16(q_bits, sess.dev), to_device_bf16(kn, sess.dev)
        o_x, l_x = _cpu_partial(sess, q_bits)
        need = wsk.wsk_decode_step_workspace(sess.h, sess.ids)
        r256 = lambda x: (x + 255) // 256 * 256
        partials = max(p for p in range(1, 4096) if r256(p * H * dv * 4) + r256(p * H * 4) <= need)
        short_tiles = -(-lengths[1] // 64) - splits[1] // 64
        say("  %d chunk partials in all, at most %d of the short sequence" % (partials, -(-short_tiles // 4)))
        assert partials - -(-short_tiles // 4) > 32, partials
        if kind == "mla":
            _, w_uv = wl.draw_mla_weights(w, gen)
            ws = torch.empty(wsk.wsk_decode_step_workspace(sess.h, sess.ids), dtype=torch.uint8, device=sess.dev)
            o_lat = torch.empty(sess.B, H, 512, device=sess.dev)
            lse = torch.empty(sess.B, H, device=sess.dev)
            o = torch.empty(sess.B, H, w.head_dim, device=sess.dev)
            wsk.wsk_decode_step_mla(sess.h, sess.ids, q, knd, to_device_bf16(w_uv, sess.dev), o, lse, ws,
                                    o_lat=o_lat, o_x=o_x, lse_x=l_x)
            o, out, lse = o.cpu().numpy(), o_lat.cpu().numpy(), lse.cpu().numpy()
        else:
            out, lse = _step(sess, q, knd, to_device_bf16(vn, sess.dev), o_x, l_x)
            out, lse = out.cpu().numpy(), lse.cpu().numpy()
        for b in range(sess.B):
            k = np.concatenate([pf.k[b], kn[b:b + 1]])
            v = None if vn is None else np.concatenate([pf.v[b], vn[b:b + 1]])
            o_r, l_r = oracle.attend(q_bits[b], k, v, 0, lengths[b] + 1, w.softmax_scale, g, dv=dv)
            assert_close(out[b], o_r, "%s many chunks b%d" % (kind, b))
            assert_lse(lse[b], l_r, "%s many chunks b%d" % (kind, b))
            if kind == "mla":
                assert_close(o[b], oracle.mla_expand(o_r, w_uv), "mla many chunks O b%d" % b)
