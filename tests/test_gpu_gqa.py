"""GPU parity of the GQA decode path against the fp64 oracle (runs on an MI355X).

Routing and pool bytes are compared bit for bit with the oracle's routing
model; attention outputs and merged results within max_abs <= 1e-2 and
L1-ratio <= 1e-3 (bf16 inputs, fp32 accumulation).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.route import CPU, GPU, RouteModel
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


def _kv_full(prefill, steps_k, steps_v, b):
    """Token-major K, V of sequence b including appended rows."""
    k = prefill.k[b]
    v = prefill.v[b]
    if steps_k:
        k = np.concatenate([k] + [s[b][None] for s in steps_k])
        v = np.concatenate([v] + [s[b][None] for s in steps_v])
    return k, v


def _oracle_partial(w, q_b, k, v, a, e):
    return oracle.attend(q_b, k, v, a, e, w.softmax_scale, w.group)


def _check_step(w, sess, q, ks, vs, prefill, o_gpu, lse_gpu, o_m, lse_m, ranges, label, sample=None):
    """Compare the GPU partial over `ranges` and the merged result with the oracle."""
    bs = range(sess.B) if sample is None else sample
    og, lg, om, lm, rg, rl, rm, rml = [], [], [], [], [], [], [], []
    for b in bs:
        k, v = _kv_full(prefill, ks, vs, b)
        a, e = ranges[b]
        o_r, l_r = _oracle_partial(w, q[b], k, v, a, e)
        o_f, l_f = _oracle_partial(w, q[b], k, v, 0, e)
        og.append(o_gpu[b]); lg.append(lse_gpu[b]); rg.append(o_r); rl.append(l_r)
        if o_m is not None:
            om.append(o_m[b]); lm.append(lse_m[b]); rm.append(o_f); rml.append(l_f)
    assert_close(np.stack(og), np.stack(rg), label + " gpu partial")
    assert_lse(np.stack(lg), np.stack(rl), label + " gpu partial")
    if o_m is not None:
        assert_close(np.stack(om), np.stack(rm), label + " merged")
        assert_lse(np.stack(lm), np.stack(rml), label + " merged")


def _cpu_partial_dev(w, q, prefill, splits, dev):
    """The CPU-range partial (oracle, fp64 -> fp32) copied to the device."""
    os_, ls_ = [], []
    for b in range(len(splits)):
        o, l = _oracle_partial(w, q[b], prefill.k[b], prefill.v[b], 0, splits[b])
        os_.append(o)
        ls_.append(l)
    return (torch.from_numpy(np.stack(os_).astype(np.float32)).to(dev),
            torch.from_numpy(np.stack(ls_).astype(np.float32)).to(dev))


def _check_routing_and_bytes(sess, model, prefill, ks, vs, full_pool=False):
    """Bit-exact routing against the oracle model, and the bytes at every routed
    GPU address equal the source rows; optionally every other pool byte is zero."""
    w = sess.w
    cpu_v, gpu_v = wsk.wsk_views(sess.h, 0)
    slot_bytes = gpu_v.slot_bytes
    dev_slots = sess.spec.device_pool_blocks
    pool = d2h(gpu_v.pool, slot_bytes * dev_slots).view(np.uint16)
    touched = np.zeros(pool.shape, bool) if full_pool else None
    mism = 0
    for b in range(sess.B):
        k, v = _kv_full(prefill, ks, vs, b)
        L = sess.lengths[b]
        assert k.shape[0] == L
        for p in range(L):
            r = wsk.wsk_route(sess.h, b, p)
            assert r == model.route(b, p), (b, p, r, model.route(b, p))
        # bytes of the GPU partition: every position, both K and V, at the
        # element the TILED64 formula of include/wsk.h names
        assert gpu_v.layout == wsk.LAYOUT_TILED64
        s = min(sess.splits[b], L)
        pos = np.arange(s, L)
        if pos.size == 0:
            continue
        slots = np.array([wsk.wsk_route(sess.h, b, int(p_))[2] for p_ in pos])
        off = pos % sess.spec.block_tokens
        t = off % 64
        tile_base = slots * (slot_bytes // 2) + (off // 64) * 16384
        d = np.arange(w.head_dim)
        mt = 2 * (t // 32) + (t % 8) // 4
        nk = 4 * ((t % 32) // 8) + t % 4
        k_el = (4 * mt[:, None] + d[None] // 32) * 64 + 16 * ((d[None] % 32) // 8) + nk[:, None]
        k_el = k_el * 8 + d[None] % 8
        v_el = (2 * (d[None] // 16) + t[:, None] // 32) * 64 + 16 * ((t[:, None] % 32) // 8) + d[None] % 16
        v_el = 8192 + v_el * 8 + (t[:, None] % 8)
        for g in range(w.n_kv_heads):
            head = tile_base[:, None] + g * (gpu_v.head_bytes // 2)
            ka, va = head + k_el, head + v_el
            mism += int(np.count_nonzero(pool[ka] != k[s:L, g]))
            mism += int(np.count_nonzero(pool[va] != v[s:L, g]))
            if touched is not None:
                touched[ka] = True
                touched[va] = True
    assert mism == 0, mism
    if touched is not None:
        assert not pool[~touched].any()


def _model_for(sess, prefill, appended_steps):
    m = RouteModel(sess.spec.block_tokens, sess.spec.host_pool_blocks, sess.spec.device_pool_blocks)
    for b in range(sess.B):
        m.open(b, sess.splits[b])
        m.write(b, 0, prefill.lengths[b])
    for _ in range(appended_steps):
        m.append(list(range(sess.B)))
    return m


# ---------------------------------------------------------------------------
# Tiny config: one sequence, L = 2048, split 1024; attend, merge, 1-token append
# ---------------------------------------------------------------------------

def test_c1_attend_merge_append():
    w = wl.C1
    say("case c1", w.name)
    pf = wl.make_prefill(w)
    st = wl.draw_step(w, pf.gen)
    dev = torch.device("cuda", DEV)
    with DecodeSession(w, pf, DEV) as sess:
        q = to_device_bf16(st.q, dev)
        o_cpu, l_cpu = _cpu_partial_dev(w, st.q, pf, pf.splits, dev)
        # attend the GPU partition [s, L), merge with the CPU partial
        o_g, l_g = sess.attend(q)
        o_m, l_m = sess.merge(o_cpu, l_cpu, o_g, l_g)
        ranges = [sess.gpu_range(b) for b in range(sess.B)]
        _check_step(w, sess, st.q, [], [], pf, o_g.cpu().numpy(), l_g.cpu().numpy(), o_m.cpu().numpy(),
                    l_m.cpu().numpy(), ranges, "c1")
        # then append one token and check routing + every byte of the device pool
        sess.append(to_device_bf16(st.k_new, dev), to_device_bf16(st.v_new, dev))
        model = _model_for(sess, pf, 1)
        _check_routing_and_bytes(sess, model, pf, [st.k_new], [st.v_new], full_pool=True)
        # canonical step order: append first, then attend [s, L+1) and merge
        o_g2, l_g2 = sess.attend(q)
        o_m2, l_m2 = sess.merge(o_cpu, l_cpu, o_g2, l_g2)
        ranges = [sess.gpu_range(b) for b in range(sess.B)]
        _check_step(w, sess, st.q, [st.k_new], [st.v_new], pf, o_g2.cpu().numpy(), l_g2.cpu().numpy(),
                    o_m2.cpu().numpy(), l_m2.cpu().numpy(), ranges, "c1 after append")


# ---------------------------------------------------------------------------
# Edge cases on small caches
# ---------------------------------------------------------------------------

def _small(Hq, Hkv, lengths, splits, seed, bk=64, std=1.0):
    w = wl.Workload("edge", wl.GQA, batch=len(lengths), n_q_heads=Hq, n_kv_heads=Hkv, head_dim=128,
                    context=max(lengths), seed=seed, block_tokens=bk, kv_std=std)
    gen = torch.Generator().manual_seed(seed)
    ks = [wl.draw_bf16(gen, (L, Hkv, 128), std) for L in lengths]
    vs = [wl.draw_bf16(gen, (L, Hkv, 128), std) for L in lengths]
    pf = wl.Prefill(list(lengths), list(splits), ks, vs, gen)
    return w, pf


@pytest.mark.parametrize("Hq,Hkv,bk", [(8, 2, 64), (32, 4, 64), (4, 4, 64), (32, 2, 128), (24, 4, 256),
                                        (6, 2, 64), (64, 1, 64), (48, 4, 128)])
def test_ranges_and_group_sizes(Hq, Hkv, bk):
    """Unaligned, single-token, single-tile, empty and tail ranges; G = 1, 3, 4, 6, 8, 12, 16, 64
    (G = 12 and 64: several query-head groups per KV head)."""
    lengths = [1000, 700, 130, 64, 5000, 1]
    splits = [0, 333, 65, 64, 1234, 0]
    w, pf = _small(Hq, Hkv, lengths, splits, seed=Hq * 7 + bk)
    say("case ranges Hq=%d Hkv=%d bk=%d" % (Hq, Hkv, bk))
    dev = torch.device("cuda", DEV)
    q_bits = wl.draw_bf16(pf.gen, (len(lengths), Hq, 128))
    with DecodeSession(w, pf, DEV, extra_tokens=0, block_tokens=bk) as sess:
        q = to_device_bf16(q_bits, dev)
        cases = [
            [(0, 1000), (333, 700), (65, 130), (64, 64), (1234, 5000), (0, 1)],       # whole GPU ranges
            [(999, 1000), (333, 334), (100, 101), (64, 64), (4999, 5000), (1, 1)],   # one token / empty
            [(10, 63), (400, 450), (65, 129), (64, 64), (1300, 1400), (0, 0)],       # inside one tile
            [(63, 65), (383, 385), (127, 130), (64, 64), (1279, 4097), (0, 1)],      # tile boundaries
        ]
        for ranges in cases:
            start = [a for a, _ in ranges]
            end = [e for _, e in ranges]
            o, l = sess.attend(q, start, end)
            o, l = o.cpu().numpy(), l.cpu().numpy()
            for b, (a, e) in enumerate(ranges):
                o_r, l_r = oracle.attend(q_bits[b], pf.k[b], pf.v[b], a, e, w.softmax_scale, w.group)
                if e == a:
                    assert np.all(o[b] == 0) and np.all(np.isneginf(l[b])), (b, a, e)
                    continue
                assert_close(o[b], o_r, "b%d [%d,%d)" % (b, a, e))
                assert_lse(l[b], l_r, "b%d [%d,%d)" % (b, a, e))


def test_garbage_outside_range_is_ignored():
    """Rows outside [start, end) in the same tiles hold NaN/Inf: the result is unaffected."""
    Hq, Hkv = 8, 2
    L = 600
    w, pf = _small(Hq, Hkv, [L], [0], seed=11)
    nan_k = pf.k[0].copy()
    nan_v = pf.v[0].copy()
    for p in list(range(0, 70)) + list(range(530, 600)):
        nan_k[p] = 0x7FC0 if p % 2 else 0x7F80     # NaN / +Inf
        nan_v[p] = 0x7FC0 if p % 3 else 0xFF80
    pf2 = wl.Prefill([L], [0], [nan_k], [nan_v], pf.gen)
    q_bits = wl.draw_bf16(pf.gen, (1, Hq, 128))
    dev = torch.device("cuda", DEV)
    say("case garbage rows")
    with DecodeSession(w, pf2, DEV, extra_tokens=0) as sess:
        o, l = sess.attend(to_device_bf16(q_bits, dev), [70], [530])
        o_r, l_r = oracle.attend(q_bits[0], pf.k[0], pf.v[0], 70, 530, w.softmax_scale, w.group)
        assert_close(o.cpu().numpy()[0], o_r, "garbage outside")
        assert_lse(l.cpu().numpy()[0], l_r, "garbage outside")


def test_many_sequences_split_launches_and_duplicates():
    """More sequences than one launch carries (64), repeated ids, mixed ranges."""
    n = 70
    lengths = [int(x) for x in np.random.default_rng(4).integers(1, 400, n)]
    splits = [int(L * f) for L, f in zip(lengths, np.random.default_rng(5).uniform(0, 1, n))]
    w, pf = _small(16, 4, lengths, splits, seed=21)
    dev = torch.device("cuda", DEV)
    say("case many sequences n=%d" % n)
    ids = list(range(n)) + [3, 3, 69]
    q_bits = wl.draw_bf16(pf.gen, (len(ids), 16, 128))
    with DecodeSession(w, pf, DEV, extra_tokens=0) as sess:
        start = [sess.gpu_range(b)[0] for b in ids]
        end = [sess.lengths[b] for b in ids]
        # the repeated ids attend sub-ranges of their GPU partition
        for i in (n, n + 1):
            a, e = sess.gpu_range(3)
            start[i], end[i] = a + (e - a) // 3 * (i - n), a + (e - a) // 2 * (i - n + 1)
        o, l = sess.attend(to_device_bf16(q_bits, dev), start, end, ids=ids)
        o, l = o.cpu().numpy(), l.cpu().numpy()
        ref_o, ref_l, got_o, got_l = [], [], [], []
        for i, b in enumerate(ids):
            o_r, l_r = oracle.attend(q_bits[i], pf.k[b], pf.v[b], start[i], end[i], w.softmax_scale, w.group)
            if end[i] == start[i]:
                assert np.all(o[i] == 0) and np.all(np.isneginf(l[i]))
                continue
            ref_o.append(o_r); ref_l.append(l_r); got_o.append(o[i]); got_l.append(l[i])
        assert_close(np.stack(got_o), np.stack(ref_o), "70 sequences")
        assert_lse(np.stack(got_l), np.stack(ref_l), "70 sequences")


def test_merge_kernel_cases():
    rng = np.random.default_rng(9)
    dev = torch.device("cuda", DEV)
    rows, width = 300, 128
    oa = rng.standard_normal((rows, width)).astype(np.float32)
    ob = rng.standard_normal((rows, width)).astype(np.float32)
    la = (rng.standard_normal(rows) * 5).astype(np.float32)
    lb = (rng.standard_normal(rows) * 5).astype(np.float32)
    la[:10] = -np.inf                      # empty CPU side
    lb[10:20] = -np.inf                    # empty GPU side
    la[20:25] = -np.inf
    lb[20:25] = -np.inf                    # both empty
    lb[25:30] = la[25:30] + 80             # one side dominates
    say("case merge kernel")
    ro, rl = oracle.merge(oa.astype(np.float64), la.astype(np.float64), ob.astype(np.float64), lb.astype(np.float64))
    t = lambda x: torch.from_numpy(x).to(dev)
    o_out, l_out = torch.empty(rows, width, device=dev), torch.empty(rows, device=dev)
    bf = torch.empty(rows, width, dtype=torch.int16, device=dev)
    wsk.wsk_merge(t(oa), t(la), t(ob), t(lb), o_out, l_out, bf)
    got = o_out.cpu().numpy()
    assert np.array_equal(got[:10], ob[:10]) and np.array_equal(got[10:20], oa[10:20])
    assert np.all(got[20:25] == 0) and np.all(np.isneginf(l_out.cpu().numpy()[20:25]))
    assert np.max(np.abs(got - ro)) < 1e-5
    assert_lse(l_out.cpu().numpy(), rl, "merge")
    bits = bf.cpu().numpy().view(np.uint16)
    assert np.array_equal(bits, oracle.round_bf16(got.astype(np.float64)))
    # in place into the b side
    ob_d, lb_d = t(ob), t(lb)
    wsk.wsk_merge(t(oa), t(la), ob_d, lb_d, ob_d, lb_d)
    assert np.max(np.abs(ob_d.cpu().numpy() - ro)) < 1e-5
    assert_lse(lb_d.cpu().numpy(), rl, "merge in place")


# ---------------------------------------------------------------------------
# Full-size configurations
# ---------------------------------------------------------------------------

def test_c2_qwen3_full():
    w = wl.C2
    say("case c2", w.name)
    pf = wl.make_prefill(w)
    st = wl.draw_step(w, pf.gen)
    dev = torch.device("cuda", DEV)
    with DecodeSession(w, pf, DEV) as sess:
        sess.append(to_device_bf16(st.k_new, dev), to_device_bf16(st.v_new, dev))
        q = to_device_bf16(st.q, dev)
        o_g, l_g = sess.attend(q)
        o_cpu, l_cpu = _cpu_partial_dev(w, st.q, pf, pf.splits, dev)
        o_m, l_m = sess.merge(o_cpu, l_cpu, o_g, l_g)
        ranges = [sess.gpu_range(b) for b in range(sess.B)]
        _check_step(w, sess, st.q, [st.k_new], [st.v_new], pf, o_g.cpu().numpy(), l_g.cpu().numpy(),
                    o_m.cpu().numpy(), l_m.cpu().numpy(), ranges, "c2")
        model = _model_for(sess, pf, 1)
        for b in (0, 7, 15):
            for p in (0, 9829, 9830, 9831, 32767, 32768):
                assert wsk.wsk_route(sess.h, b, p) == model.route(b, p)
    # the same step as the benchmark times it: wsk_decode_step (pass 1, then
    # pass 2 scoring and storing the new row and merging the CPU partial)
    with DecodeSession(w, pf, DEV) as sess:
        o_d, l_d = sess.decode_step(q, to_device_bf16(st.k_new, dev), to_device_bf16(st.v_new, dev),
                                    o_x=o_cpu, lse_x=l_cpu)
        o_d, l_d = o_d.cpu().numpy(), l_d.cpu().numpy()
        _check_step(w, sess, st.q, [st.k_new], [st.v_new], pf, o_g.cpu().numpy(), l_g.cpu().numpy(), o_d, l_d,
                    ranges, "c2 decode step")
        assert np.abs(o_d - o_m.cpu().numpy()).max() <= 1e-5 and np.abs(l_d - l_m.cpu().numpy()).max() <= 1e-5
        for b in (0, 7, 15):
            assert wsk.wsk_route(sess.h, b, 32768) == model.route(b, 32768)


def test_c3_mixtral_sweep_without_data_movement():
    """The CPU share moves over {0, .25, .5, .75} on one cache written once with s = 0:
    only the attend range changes, and the device pool's bytes stay identical."""
    w = wl.C3
    say("case c3", w.name)
    pf = wl.make_prefill(w)
    st = wl.draw_step(w, pf.gen)
    dev = torch.device("cuda", DEV)
    with DecodeSession(w, pf, DEV, extra_tokens=0) as sess:
        _, gpu_v = wsk.wsk_views(sess.h, 0)
        nbytes = gpu_v.slot_bytes * sess.spec.device_pool_blocks
        import hashlib
        before = hashlib.blake2b(d2h(gpu_v.pool, nbytes).tobytes(), digest_size=16).hexdigest()
        q = to_device_bf16(st.q, dev)
        L = w.context
        for share in w.sweep:
            s = wl.split_point(share, L)
            o_g, l_g = sess.attend(q, [s] * sess.B, [L] * sess.B)
            o_cpu, l_cpu = _cpu_partial_dev(w, st.q, pf, [s] * sess.B, dev)
            o_m, l_m = sess.merge(o_cpu, l_cpu, o_g, l_g)
            _check_step(w, sess, st.q, [], [], pf, o_g.cpu().numpy(), l_g.cpu().numpy(), o_m.cpu().numpy(),
                        l_m.cpu().numpy(), [(s, L)] * sess.B, "c3 r=%.2f" % share)
        after = hashlib.blake2b(d2h(gpu_v.pool, nbytes).tobytes(), digest_size=16).hexdigest()
        assert before == after


def test_c5_ragged_64_steps():
    """c5 through the benchmarked call: 64 wsk_decode_step calls (append, pass 1,
    pass 2 scoring and storing the new row), routing of every appended row
    checked at every step against the oracle's model, outputs against the fp64
    oracle over the whole context at steps 0, 31 and 63 (the CPU partial of
    [0, s_b) merged in), and at step 63 also against the two-call path
    (wsk_attend over [s_b, L_b) + wsk_merge)."""
    w = wl.C5
    say("case c5", w.name)
    pf = wl.make_prefill(w)
    dev = torch.device("cuda", DEV)
    ks, vs = [], []
    with DecodeSession(w, pf, DEV) as sess:
        model = _model_for(sess, pf, 0)
        for step in range(w.steps):
            st = wl.draw_step(w, pf.gen)
            ks.append(st.k_new)
            vs.append(st.v_new)
            q = to_device_bf16(st.q, dev)
            check = step in (0, 31, 63)
            o_cpu, l_cpu = _cpu_partial_dev(w, st.q, pf, pf.splits, dev) if check else (None, None)
            o_d, l_d = sess.decode_step(q, to_device_bf16(st.k_new, dev), to_device_bf16(st.v_new, dev),
                                        o_x=o_cpu, lse_x=l_cpu)
            model.append(list(range(sess.B)))
            for b in range(sess.B):
                p = sess.lengths[b] - 1
                assert wsk.wsk_route(sess.h, b, p) == model.route(b, p), (step, b)
            if not check:
                continue
            say("c5 step %d: lengths %s" % (step, sess.lengths))
            om, lm, rm, rl = [], [], [], []
            o_d, l_d = o_d.cpu().numpy(), l_d.cpu().numpy()
            for b in range(sess.B):
                k, v = _kv_full(pf, ks, vs, b)
                o_f, l_f = _oracle_partial(w, st.q[b], k, v, 0, k.shape[0])
                om.append(o_d[b]); lm.append(l_d[b]); rm.append(o_f); rl.append(l_f)
            assert_close(np.stack(om), np.stack(rm), "c5 step %d decode step" % step)
            assert_lse(np.stack(lm), np.stack(rl), "c5 step %d decode step" % step)
            if step == 63:
                o_g, l_g = sess.attend(q)
                o_m, l_m = sess.merge(o_cpu, l_cpu, o_g, l_g)
                assert np.abs(o_m.cpu().numpy() - o_d).max() <= 1e-5
                assert np.abs(l_m.cpu().numpy() - l_d).max() <= 1e-5
        for b in range(sess.B):               # every position's route at the end
            for p in range(0, sess.lengths[b], 997):
                assert wsk.wsk_route(sess.h, b, p) == model.route(b, p)


@pytest.mark.parametrize("kind", ["gqa", "mla"])
def test_two_passes_equal_attend(kind):
    """wsk_attend_pass1 then wsk_attend_pass2 is wsk_attend, bit for bit."""
    if kind == "gqa":
        w = wl.Workload("two-pass-gqa", wl.GQA, batch=3, n_q_heads=16, n_kv_heads=2, head_dim=128,
                        context=3000, cpu_share=0.25, seed=21)
    else:
        w = wl.Workload("two-pass-mla", wl.MLA, batch=3, n_q_heads=16, n_kv_heads=1, head_dim=128,
                        latent_dim=512, rope_dim=64, nope_dim=128, context=3000, cpu_share=0.25, kv_std=0.5,
                        seed=22)
    say("case two passes", kind)
    pf = wl.make_prefill(w)
    st = wl.draw_step(w, pf.gen)
    dev = torch.device("cuda", DEV)
    with DecodeSession(w, pf, DEV, extra_tokens=0) as sess:
        q = to_device_bf16(st.q, dev)
        o1, l1 = sess.attend(q)
        o1, l1 = o1.cpu().numpy(), l1.cpu().numpy()
        sess.attend_pass1(q)
        o2, l2 = sess.attend_pass2()
        assert np.array_equal(o1, o2.cpu().numpy())
        assert np.array_equal(l1, l2.cpu().numpy())
        # pass 2 with the CPU-range partial merged in (one launch) against
        # wsk_attend + wsk_merge and against the oracle over the whole context
        H = w.n_q_heads
        dv = w.latent_dim if kind == "mla" else w.head_dim
        cpu_o, cpu_l, full_o, full_l = [], [], [], []
        for b in range(w.batch):
            s_b, L = pf.splits[b], pf.lengths[b]
            v = None if kind == "mla" else pf.v[b]
            g = w.n_q_heads if kind == "mla" else w.group
            o_c, l_c = oracle.attend(st.q[b], pf.k[b], v, 0, s_b, w.softmax_scale, g, dv=dv)
            o_f, l_f = oracle.attend(st.q[b], pf.k[b], v, 0, L, w.softmax_scale, g, dv=dv)
            cpu_o.append(o_c)
            cpu_l.append(l_c)
            full_o.append(o_f)
            full_l.append(l_f)
        o_x = torch.from_numpy(np.stack(cpu_o).astype(np.float32)).to(dev)
        l_x = torch.from_numpy(np.stack(cpu_l).astype(np.float32)).to(dev)
        sess.attend_pass1(q)
        o3, l3 = sess.attend_pass2(o_x=o_x, lse_x=l_x)
        o4, l4 = sess.merge(o_x, l_x, torch.from_numpy(o1).to(dev), torch.from_numpy(l1).to(dev))
        o3, l3 = o3.cpu().numpy(), l3.cpu().numpy()
        assert np.allclose(o3, o4.cpu().numpy(), rtol=1e-5, atol=1e-6)
        assert np.allclose(l3, l4.cpu().numpy(), rtol=0, atol=1e-5)
        assert_close(o3, np.stack(full_o), "two-pass merged %s" % kind)
        assert_lse(l3, np.stack(full_l), "two-pass merged %s" % kind)
        # an empty GPU range returns the other partial unchanged
        sess.attend_pass1(q, start=[pf.lengths[b] for b in range(w.batch)])
        o5, l5 = sess.attend_pass2(start=[pf.lengths[b] for b in range(w.batch)], o_x=o_x, lse_x=l_x)
        assert torch.equal(o5, o_x) and torch.equal(l5, l_x)


@pytest.mark.parametrize("kind", ["gqa", "mla"])
def test_cpu_engine_and_gpu_merge_to_the_whole_context(kind):
    """The method's whole step: the native CPU engine attends [0, s) in place in
    the host pool, the GPU attends [s, L), pass 2 merges both: the result is
    attention over the whole context (fp64 oracle)."""
    if kind == "gqa":
        w = wl.Workload("split-gqa", wl.GQA, batch=3, n_q_heads=16, n_kv_heads=2, head_dim=128, context=6000,
                        cpu_share=0.4, seed=41)
    else:
        w = wl.Workload("split-mla", wl.MLA, batch=2, n_q_heads=16, n_kv_heads=1, head_dim=128, latent_dim=512,
                        rope_dim=64, nope_dim=128, context=4000, cpu_share=0.4, kv_std=0.5, seed=42)
    say("case cpu+gpu merge", kind)
    pf = wl.make_prefill(w)
    st = wl.draw_step(w, pf.gen)
    dev = torch.device("cuda", DEV)
    dv = w.latent_dim if kind == "mla" else w.head_dim
    with DecodeSession(w, pf, DEV, extra_tokens=0) as sess:
        B, H = sess.B, w.n_q_heads
        q = to_device_bf16(st.q, dev)
        sess.attend_pass1(q)
        o_c = np.empty((B, H, dv), np.float32)
        l_c = np.empty((B, H), np.float32)
        wsk.wsk_cpu_attend(sess.h, sess.ids, [0] * B, [pf.splits[b] for b in range(B)], st.q, o_c, l_c, 4)
        o_m, l_m = sess.attend_pass2(o_x=torch.from_numpy(o_c).to(dev), lse_x=torch.from_numpy(l_c).to(dev))
        o_m, l_m = o_m.cpu().numpy(), l_m.cpu().numpy()
    g = w.n_q_heads if kind == "mla" else w.group
    for b in range(B):
        v = None if kind == "mla" else pf.v[b]
        o_r, l_r = oracle.attend(st.q[b], pf.k[b], v, 0, pf.lengths[b], w.softmax_scale, g, dv=dv)
        assert_close(o_m[b], o_r, "cpu+gpu %s b%d" % (kind, b))
        assert_lse(l_m[b], l_r, "cpu+gpu %s b%d" % (kind, b))
