"""The load region on the GPU (Sec. 4.2-4.4) against the fp64 oracle:
streaming of the pinned load region through the ping-pong pair
(wsk_attend_gpu), D-window eviction to the CPU and to the load region
(wsk_flush) followed by the full CPU + GPU step, and block selections whose
load-region blocks are gathered and sent as one DMA (wsk_attend_blocks)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
from tests.gpu_util import assert_close, assert_lse, say
from tests.layouts import gqa_elements, mla_elements

pytestmark = pytest.mark.gpu
DEV = 0
CPU, GPU, LOAD = wsk.PART_CPU, wsk.PART_GPU, wsk.PART_LOAD


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(DEV)
    yield
    torch.cuda.synchronize()


def _workload(kind, B, H=16, seed=0):
    if kind == "gqa":
        return wl.Workload("load-gqa", wl.GQA, batch=B, n_q_heads=H, n_kv_heads=2, head_dim=128, context=1,
                           seed=seed)
    return wl.Workload("load-mla", wl.MLA, batch=B, n_q_heads=H, n_kv_heads=1, head_dim=128, latent_dim=512,
                       rope_dim=64, nope_dim=128, context=1, kv_std=0.5, seed=seed)


def _prefill(w, lengths, splits, gen):
    if w.kind == wl.MLA:
        ks = [wl.draw_bf16(gen, (L, w.row_elems), w.kv_std) for L in lengths]
        vs = None
    else:
        ks = [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths]
        vs = [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths]
    return wl.Prefill(list(lengths), list(splits), ks, vs, gen)


def _dims(w):
    return (w.latent_dim if w.kind == wl.MLA else w.head_dim), (w.n_q_heads if w.kind == wl.MLA else w.group)


def _check(w, q_bits, k_all, v_all, positions, o, lse, what):
    """o/lse (numpy) of each sequence against the oracle over exactly `positions`."""
    dv, g = _dims(w)
    for b, pos in enumerate(positions):
        pos = np.asarray(pos, dtype=np.int64)
        if pos.size == 0:
            assert np.all(o[b] == 0) and np.all(np.isneginf(lse[b])), (what, b)
            continue
        k = k_all[b][pos]
        v = None if v_all is None else v_all[b][pos]
        o_r, l_r = oracle.attend(q_bits[b], k, v, 0, pos.size, w.softmax_scale, g, dv=dv)
        assert_close(o[b], o_r, "%s b%d" % (what, b))
        assert_lse(lse[b], l_r, "%s b%d" % (what, b))


def _cpu_partial(sess, q_bits):
    """CPU engine over every CPU position, as device tensors for the merge."""
    w = sess.w
    dv, _ = _dims(w)
    o = np.empty((sess.B, w.n_q_heads, dv), np.float32)
    lse = np.empty((sess.B, w.n_q_heads), np.float32)
    wsk.wsk_cpu_attend_all(sess.h, sess.ids, np.ascontiguousarray(q_bits), o, lse, 8)
    return torch.from_numpy(o).to(sess.dev), torch.from_numpy(lse).to(sess.dev)


@pytest.mark.parametrize("kind,bk,pp", [("gqa", 64, 3), ("gqa", 128, 5), ("mla", 64, 3), ("mla", 256, 2)])
def test_streamed_attend(kind, bk, pp):
    """Split inside a block, load_end past the prefill (a partial last load
    block), no load range (the window starts inside a block), no CPU part, a
    single-token sequence; ping-pong buffers of 2-5 blocks so that one call
    cycles through both buffers many times, arenas of 5 slots so that runs of
    slots break at arena ends."""
    lengths = [9 * bk + 5, 5 * bk + 7, 3 * bk + 20, 4 * bk, 1]
    splits = [bk + 37, 100, 2 * bk + 9, 0, 0]
    load_ends = [6 * bk, 10 * bk, 2 * bk + 9, 3 * bk, bk]
    w = _workload(kind, len(lengths), seed=bk + pp)
    gen = torch.Generator().manual_seed(w.seed + 11)
    pf = _prefill(w, lengths, splits, gen)
    q_bits = wl.draw_bf16(gen, (len(lengths), w.n_q_heads, w.row_elems))
    say("case streamed", kind, bk, pp)
    with DecodeSession(w, pf, DEV, extra_tokens=0, block_tokens=bk, load_ends=load_ends, pingpong_blocks=pp,
                       arena_blocks=5) as sess:
        q = to_device_bf16(q_bits, sess.dev)
        for b in range(sess.B):
            segs = wsk.wsk_seq_segments(sess.h, b)
            L, s, e = lengths[b], splits[b], load_ends[b]
            want = [(a, z, p) for a, z, p in ((0, min(s, L), CPU), (s, min(e, L), LOAD), (e, L, GPU)) if z > a]
            assert segs == want, (b, segs, want)
        gpu_pos = [np.arange(min(s, L), L) for s, L in zip(splits, lengths)]
        for rep in range(2):          # the second call reuses the ping-pong events
            o, lse = sess.attend_gpu(q)
            _check(w, q_bits, pf.k, pf.v, gpu_pos, o.cpu().numpy(), lse.cpu().numpy(), "gpu side %d" % rep)
        o_x, l_x = _cpu_partial(sess, q_bits)
        o, lse = sess.attend_gpu(q, o_x=o_x, lse_x=l_x)
        _check(w, q_bits, pf.k, pf.v, [np.arange(L) for L in lengths], o.cpu().numpy(), lse.cpu().numpy(),
               "whole step")
        # the two-pass form with the CPU engine running between the passes
        # (while the transfers and kernels of pass 1 are in flight)
        sess.attend_gpu_pass1(q)
        o_x2, l_x2 = _cpu_partial(sess, q_bits)
        o2, lse2 = sess.attend_gpu_pass2(o_x=o_x2, lse_x=l_x2)
        assert torch.equal(o2, o) and torch.equal(lse2, lse)
        st = wsk.wsk_load_stats(sess.h)
        load_blocks = sum(-(-min(e, L) // bk) - s // bk for s, e, L in zip(splits, load_ends, lengths) if min(e, L) > s)
        assert st.h2d_bytes == 4 * load_blocks * w.token_bytes * bk   # four calls


def test_streamed_attend_many_sequences():
    """70 sequences (two launches per chunk), every one with load blocks."""
    B = 70
    w = _workload("gqa", B, H=8, seed=3)
    gen = torch.Generator().manual_seed(5)
    lengths = [int(x) for x in torch.randint(130, 600, (B,), generator=gen)]
    splits = [L // 5 for L in lengths]
    load_ends = [max(s, (L // 2) // 64 * 64) for s, L in zip(splits, lengths)]
    pf = _prefill(w, lengths, splits, gen)
    q_bits = wl.draw_bf16(gen, (B, w.n_q_heads, w.row_elems))
    say("case streamed many")
    with DecodeSession(w, pf, DEV, extra_tokens=0, load_ends=load_ends, pingpong_blocks=16, arena_blocks=64) as sess:
        o, lse = sess.attend_gpu(to_device_bf16(q_bits, sess.dev))
        _check(w, q_bits, pf.k, pf.v, [np.arange(min(s, L), L) for s, L in zip(splits, lengths)],
               o.cpu().numpy(), lse.cpu().numpy(), "many")


@pytest.mark.parametrize("kind,bk", [("gqa", 64), ("mla", 128)])
def test_flush_then_full_step(kind, bk):
    """Decode appends fill the D-window; flushes move batches to the CPU and
    to the load region in turn; after each flush the CPU engine over every
    CPU position plus the GPU side (window in place, load region streamed)
    equals attention over the whole context.  Sequence 0 has a load range,
    sequence 1 none and a split inside a block (its first batch starts
    there), sequence 2 no CPU part."""
    D = 2 * bk
    lengths = [3 * bk + 10, 2 * bk + 50, bk + 3]
    splits = [bk + 17, bk + 50, 0]
    load_ends = [2 * bk, bk + 50, bk]
    steps = 5 * bk
    w = _workload(kind, len(lengths), H=8, seed=bk)
    gen = torch.Generator().manual_seed(w.seed + 1)
    pf = _prefill(w, lengths, splits, gen)
    hkv = 1 if kind == "mla" else w.n_kv_heads
    k_all = [k for k in pf.k]
    v_all = None if pf.v is None else [v for v in pf.v]
    say("case flush", kind, bk)
    from oracle.route import RouteModel
    with DecodeSession(w, pf, DEV, extra_tokens=steps, block_tokens=bk, load_ends=load_ends, evict_tokens=D,
                       pingpong_blocks=3, arena_blocks=4) as sess:
        # the oracle's routing model replays every operation; routes must agree bit for bit
        model = RouteModel(bk, sess.spec.host_pool_blocks, sess.spec.device_pool_blocks, sess.spec.load_pool_blocks, D)
        for b in range(sess.B):
            model.open(b, splits[b], load_ends[b])
            model.write(b, 0, lengths[b])
        parts_cycle = [LOAD, CPU, CPU, LOAD]
        flushes = 0
        for step in range(steps):
            if kind == "mla":
                kn = wl.draw_bf16(gen, (sess.B, w.row_elems), w.kv_std)
                vn = None
            else:
                kn = wl.draw_bf16(gen, (sess.B, hkv, w.head_dim))
                vn = wl.draw_bf16(gen, (sess.B, hkv, w.head_dim))
            sess.append(to_device_bf16(kn, sess.dev), None if vn is None else to_device_bf16(vn, sess.dev))
            model.append(list(range(sess.B)))
            for b in range(sess.B):
                k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                if v_all is not None:
                    v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
            if step % (bk // 2) != bk // 2 - 1:
                continue
            parts = [parts_cycle[(flushes + b) % 4] for b in range(sess.B)]
            before = [sess.gpu_range(b)[0] for b in range(sess.B)]
            moved = sess.flush(parts)
            assert moved == model.flush(list(range(sess.B)), parts)
            for b in range(sess.B):
                assert [wsk.wsk_route(sess.h, b, p) for p in range(sess.lengths[b])] == \
                    [model.route(b, p) for p in range(sess.lengths[b])], (flushes, b)
            flushes += 1
            for b in range(sess.B):
                w0, L = before[b], sess.lengths[b]
                w1 = (w0 + D) // bk * bk
                assert moved[b] == (w1 - w0 if w1 <= L else 0), (b, moved[b], w0, L)
                if moved[b]:
                    assert sess.gpu_range(b)[0] == w1
                    assert wsk.wsk_route(sess.h, b, w0)[0] == parts[b]
                    assert wsk.wsk_route(sess.h, b, w1 - 1)[0] == parts[b]
            q_bits = wl.draw_bf16(gen, (sess.B, w.n_q_heads, w.row_elems))
            q = to_device_bf16(q_bits, sess.dev)
            o_x, l_x = _cpu_partial(sess, q_bits)
            o, lse = sess.attend_gpu(q, o_x=o_x, lse_x=l_x)
            _check(w, q_bits, k_all, v_all, [np.arange(L) for L in sess.lengths], o.cpu().numpy(),
                   lse.cpu().numpy(), "after flush %d" % flushes)
        # every position's home is one of the three, the segments alternate
        # homes, and the load-region bytes follow the GPU layout
        torch.cuda.synchronize()
        for b in range(sess.B):
            segs = wsk.wsk_seq_segments(sess.h, b)
            assert segs[0][0] == 0 and segs[-1][1] == sess.lengths[b]
            assert all(x[1] == y[0] and x[2] != y[2] for x, y in zip(segs, segs[1:]))
            for a, e, part in segs:
                if part != LOAD:
                    continue
                for blk in range(a // bk, -(-e // bk)):
                    loc = wsk.wsk_route(sess.h, b, max(a, blk * bk))
                    sb = w.token_bytes * bk
                    mem = np.frombuffer((ctypes.c_uint16 * (sb // 2)).from_address(wsk.wsk_load_slot(sess.h, loc[2])),
                                        dtype=np.uint16)
                    pos = np.arange(max(a, blk * bk), min(e, (blk + 1) * bk))
                    if kind == "mla":
                        assert np.array_equal(mem[mla_elements(pos % bk, w.row_elems)], k_all[b][pos])
                    else:
                        for g in range(hkv):
                            ke, ve = gqa_elements(pos % bk, w.head_dim, bk, g)
                            assert np.array_equal(mem[ke], k_all[b][pos, g])
                            assert np.array_equal(mem[ve], v_all[b][pos, g])
        assert flushes >= 8


@pytest.mark.parametrize("kind,bk", [("gqa", 64), ("mla", 64), ("gqa", 256)])
def test_sparse_selection_with_load_blocks(kind, bk):
    """Selections mixing load-region blocks (gathered, one DMA per ping-pong
    buffer) and D-window blocks (in place): the partial block holding s, the
    partial last block, shuffled middles, load blocks only, window blocks
    only, nothing; then the refused selections."""
    lengths = [12 * bk + 9, 7 * bk + 1, 5 * bk]
    splits = [bk + 20, 0, 2 * bk]
    load_ends = [8 * bk, 5 * bk, 2 * bk]
    w = _workload(kind, len(lengths), seed=3 * bk)
    gen = torch.Generator().manual_seed(w.seed + 2)
    pf = _prefill(w, lengths, splits, gen)
    q_bits = wl.draw_bf16(gen, (len(lengths), w.n_q_heads, w.row_elems))
    rng = np.random.default_rng(bk)
    say("case sparse load", kind, bk)
    with DecodeSession(w, pf, DEV, extra_tokens=0, block_tokens=bk, load_ends=load_ends, pingpong_blocks=3,
                       arena_blocks=4) as sess:
        q = to_device_bf16(q_bits, sess.dev)
        dv, _ = _dims(w)

        def gpu_side(b, blk):
            lo = max(blk * bk, splits[b])
            return np.arange(lo, min((blk + 1) * bk, lengths[b]))

        def run(sels, o_x=None, l_x=None, extra=None):
            need = wsk.wsk_attend_blocks_workspace(sess.h, sess.ids, sels)
            ws = torch.empty(need, dtype=torch.uint8, device=sess.dev)
            o = torch.empty(sess.B, w.n_q_heads, dv, device=sess.dev)
            lse = torch.empty(sess.B, w.n_q_heads, device=sess.dev)
            wsk.wsk_attend_blocks(sess.h, sess.ids, sels, q, o, lse, ws, o_x, l_x)
            pos = [np.concatenate([gpu_side(b, x) for x in sels[b]] or [np.zeros(0, np.int64)])
                   for b in range(sess.B)]
            if extra is not None:
                pos = [np.concatenate([extra[b], p]) for b, p in enumerate(pos)]
            _check(w, q_bits, pf.k, pf.v, pos, o.cpu().numpy(), lse.cpu().numpy(), "sparse")

        blocks = [list(range(s // bk, -(-L // bk))) for s, L in zip(splits, lengths)]
        # s-block (load, partial) + shuffled load middles + window blocks incl. the partial last one
        sel0 = [blocks[0][-1]] + list(rng.permutation(blocks[0][1:-1])[:6]) + [blocks[0][0]]
        run([sel0, blocks[1][:5], []])                    # load blocks only for sequence 1
        run([blocks[0], list(rng.permutation(blocks[1])), blocks[2]])   # everything
        run([list(rng.permutation(blocks[0])[:4]), [blocks[1][-1]], [blocks[2][0]]])
        o_x, l_x = _cpu_partial(sess, q_bits)
        run([sel0, blocks[1][2:4], blocks[2]], o_x, l_x, extra=[np.arange(s) for s in splits])
        with pytest.raises(wsk.WskError) as ei:           # a CPU-only block
            wsk.wsk_attend_blocks_workspace(sess.h, [0], [[0]])
        assert ei.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_attend_blocks_workspace(sess.h, [0], [[3, 3]])
        assert ei.value.code == wsk.WSK_EINVAL
        with pytest.raises(wsk.WskError) as ei:           # past L
            wsk.wsk_attend_blocks_workspace(sess.h, [2], [[5]])
        assert ei.value.code == wsk.WSK_ERANGE


def test_policy_routed_eviction_follows_R_of_L():
    """The split policy drives eviction (Sec. 5.3 with Sec. 4.2): every D-batch
    goes where wsk_policy_route_batch sends it (the GPU side is the load region
    here), so after k batches the CPU share of the placed positions is
    R(L) = p + (R0 - p) L0 / L within D / (2L), and the full step still equals
    attention over the whole context."""
    from oracle import policy as P
    bk, D, batches = 64, 128, 12
    L0s, s0s = [1000, 700], [200, 420]
    load_ends = [896, 640]
    w = _workload("gqa", 2, H=8, seed=9)
    gen = torch.Generator().manual_seed(21)
    pf = _prefill(w, L0s, s0s, gen)
    k_all, v_all = list(pf.k), list(pf.v)
    A, Bc = 2e-9, 3e-9                      # p = 0.6
    pols = [wsk.Policy(A, Bc, 1e-5, 1e-5, 4) for _ in range(2)]
    say("case policy eviction")
    try:
        with DecodeSession(w, pf, DEV, extra_tokens=batches * D + D, load_ends=load_ends, evict_tokens=D,
                           pingpong_blocks=4, arena_blocks=8) as sess:
            placed0 = list(load_ends)
            cpu = list(s0s)
            done = [0, 0]
            while min(done) < batches:
                kn = wl.draw_bf16(gen, (2, w.n_kv_heads, w.head_dim))
                vn = wl.draw_bf16(gen, (2, w.n_kv_heads, w.head_dim))
                sess.append(to_device_bf16(kn, sess.dev), to_device_bf16(vn, sess.dev))
                for b in range(2):
                    k_all[b] = np.concatenate([k_all[b], kn[b:b + 1]])
                    v_all[b] = np.concatenate([v_all[b], vn[b:b + 1]])
                for b in range(2):
                    if done[b] >= batches or sess.gpu_range(b)[1] - sess.gpu_range(b)[0] < D:
                        continue
                    part = pols[b].route()
                    dest = CPU if part == wsk.PART_CPU else LOAD
                    moved = wsk.wsk_flush(sess.h, [b], [dest])
                    assert moved == [D]
                    done[b] += 1
                    if dest == CPU:
                        cpu[b] += D
                    L = placed0[b] + done[b] * D
                    R0 = s0s[b] / placed0[b]
                    R = P.cumulative_share(L, placed0[b], R0, P.marginal_share(A, Bc))
                    assert abs(cpu[b] / L - R) <= D / (2 * L) + 1e-12, (b, done[b], cpu[b] / L, R)
            # the library's segments agree with the count of CPU positions
            for b in range(2):
                segs = wsk.wsk_seq_segments(sess.h, b)
                w_start = sess.gpu_range(b)[0]
                assert sum(e - a for a, e, p_ in segs if p_ == CPU) == cpu[b]
                assert w_start == placed0[b] + batches * D
            q_bits = wl.draw_bf16(gen, (2, w.n_q_heads, w.row_elems))
            o_x, l_x = _cpu_partial(sess, q_bits)
            o, lse = sess.attend_gpu(to_device_bf16(q_bits, sess.dev), o_x=o_x, lse_x=l_x)
            _check(w, q_bits, k_all, v_all, [np.arange(L) for L in sess.lengths], o.cpu().numpy(),
                   lse.cpu().numpy(), "policy-routed")
    finally:
        for p_ in pols:
            p_.close()
