"""Block-sparse attention (wsk_attend_blocks, Sec. 4.4) against the fp64
oracle over exactly the selected positions, GQA and MLA: partial first and
last blocks, any order, single blocks, empty selections, more sequences than
one launch carries, an optional merged partial, and the refused selections."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
from tests.gpu_util import assert_close, assert_lse, say

pytestmark = pytest.mark.gpu
DEV = 0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(DEV)
    yield
    torch.cuda.synchronize()


def _positions(blocks, bk, s, L):
    pos = []
    for b in blocks:
        pos.extend(range(max(b * bk, s), min((b + 1) * bk, L)))
    return np.array(pos, dtype=np.int64)


def _run(sess, w, pf, q_bits, sels, o_x=None, lse_x=None, ref_extra=None):
    dev = torch.device("cuda", DEV)
    B, H = sess.B, w.n_q_heads
    dv = w.latent_dim if w.kind == wl.MLA else w.head_dim
    ids = list(range(B))
    need = wsk.wsk_attend_blocks_workspace(sess.h, ids, sels)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    o = torch.empty(B, H, dv, device=dev)
    lse = torch.empty(B, H, device=dev)
    wsk.wsk_attend_blocks(sess.h, ids, sels, to_device_bf16(q_bits, dev), o, lse, ws, o_x, lse_x)
    o, lse = o.cpu().numpy(), lse.cpu().numpy()
    bk = sess.spec.block_tokens
    g = w.n_q_heads if w.kind == wl.MLA else w.group
    for b in range(B):
        pos = _positions(sels[b], bk, pf.splits[b], pf.lengths[b])
        if ref_extra is not None:
            pos = np.concatenate([ref_extra[b], pos])
        if pos.size == 0:
            assert np.all(o[b] == 0) and np.all(np.isneginf(lse[b]))
            continue
        k = pf.k[b][pos]
        v = None if w.kind == wl.MLA else pf.v[b][pos]
        o_r, l_r = oracle.attend(q_bits[b], k, v, 0, pos.size, w.softmax_scale, g, dv=dv)
        assert_close(o[b], o_r, "sparse b%d (%d blocks)" % (b, len(sels[b])))
        assert_lse(lse[b], l_r, "sparse b%d" % b)


@pytest.mark.parametrize("kind,bk", [("gqa", 64), ("gqa", 128), ("mla", 64), ("mla", 256)])
def test_block_selections(kind, bk):
    lengths = [3000, 700, 1100, 64, 257]
    splits = [1000, 70, 0, 0, 200]
    if kind == "gqa":
        w = wl.Workload("sparse-gqa", wl.GQA, batch=5, n_q_heads=16, n_kv_heads=2, head_dim=128, context=3000,
                        seed=51)
    else:
        w = wl.Workload("sparse-mla", wl.MLA, batch=5, n_q_heads=16, n_kv_heads=1, head_dim=128, latent_dim=512,
                        rope_dim=64, nope_dim=128, context=3000, kv_std=0.5, seed=52)
    gen = torch.Generator().manual_seed(w.seed)
    if kind == "gqa":
        ks = [wl.draw_bf16(gen, (L, 2, 128)) for L in lengths]
        vs = [wl.draw_bf16(gen, (L, 2, 128)) for L in lengths]
    else:
        ks = [wl.draw_bf16(gen, (L, w.row_elems), w.kv_std) for L in lengths]
        vs = None
    pf = wl.Prefill(lengths, splits, ks, vs, gen)
    q_bits = wl.draw_bf16(gen, (5, w.n_q_heads, w.row_elems))
    rng = np.random.default_rng(bk)
    say("case sparse", kind, bk)
    with DecodeSession(w, pf, DEV, extra_tokens=0, block_tokens=bk) as sess:
        def gpu_blocks(b):
            return list(range(splits[b] // bk, (lengths[b] - 1) // bk + 1))
        # 1: the partial first and last blocks with a shuffled middle, one block,
        #    nothing, every GPU block, the last block only
        sels = []
        for b in range(5):
            gb = gpu_blocks(b)
            if b == 0:
                mid = list(rng.permutation(gb[1:-1])[: max(1, len(gb) // 3)])
                sels.append([gb[-1]] + mid + [gb[0]])
            elif b == 1:
                sels.append([gb[len(gb) // 2]])
            elif b == 2:
                sels.append([])
            elif b == 3:
                sels.append(gb)
            else:
                sels.append([gb[-1]])
        _run(sess, w, pf, q_bits, sels)
        # 2: random top-k-like selections
        sels = [list(rng.permutation(gpu_blocks(b))[: rng.integers(0, len(gpu_blocks(b)) + 1)]) for b in range(5)]
        _run(sess, w, pf, q_bits, sels)
        # 3: merged with the CPU-range partial of [0, s)
        dv = w.latent_dim if kind == "mla" else w.head_dim
        g = w.n_q_heads if kind == "mla" else w.group
        o_c, l_c = [], []
        for b in range(5):
            o_, l_ = oracle.attend(q_bits[b], ks[b], None if vs is None else vs[b], 0, splits[b], w.softmax_scale,
                                   g, dv=dv)
            o_c.append(o_)
            l_c.append(l_)
        dev = torch.device("cuda", DEV)
        o_x = torch.from_numpy(np.stack(o_c).astype(np.float32)).to(dev)
        l_x = torch.from_numpy(np.stack(l_c).astype(np.float32)).to(dev)
        _run(sess, w, pf, q_bits, sels, o_x, l_x, ref_extra=[np.arange(splits[b]) for b in range(5)])


def test_many_sequences_and_refused_selections():
    w = wl.Workload("sparse-many", wl.GQA, batch=70, n_q_heads=8, n_kv_heads=2, head_dim=128, context=300,
                    cpu_share=0.25, seed=53)
    pf = wl.make_prefill(w)
    q_bits = wl.draw_bf16(pf.gen, (70, 8, 128))
    say("case sparse many")
    with DecodeSession(w, pf, DEV, extra_tokens=0) as sess:
        first, last = 75 // 64, 299 // 64
        sels = [[last, first + (b % (last - first))] if b % 3 else [first] for b in range(70)]
        _run(sess, w, pf, q_bits, sels)
        ids = [0]
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_attend_blocks_workspace(sess.h, ids, [[first, first]])
        assert ei.value.code == wsk.WSK_EINVAL
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_attend_blocks_workspace(sess.h, ids, [[first - 1]])   # a CPU block
        assert ei.value.code == wsk.WSK_ERANGE
        with pytest.raises(wsk.WskError) as ei:
            wsk.wsk_attend_blocks_workspace(sess.h, ids, [[last + 1]])
        assert ei.value.code == wsk.WSK_ERANGE
