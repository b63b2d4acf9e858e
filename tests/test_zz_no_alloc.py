"""wsk_decode_step_noalloc (the decode step whose chunk partials live in the
library's own device scratch, for callers that cannot allocate) against
wsk_decode_step with a caller workspace: two caches built from the same
prefill take the same steps, one through each entry point, and must agree bit
for bit (outputs, LSE, every pool byte), two calls in a row, the second with
a smaller input; both also against the fp64 oracle.  Also its refusal of a
step whose partials exceed the scratch, which changes nothing."""
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


def _workload(kind):
    if kind == "gqa":
        return wl.Workload("noalloc-gqa", wl.GQA, batch=6, n_q_heads=32, n_kv_heads=4, head_dim=128, context=1,
                           seed=61)
    return wl.Workload("noalloc-mla", wl.MLA, batch=6, n_q_heads=16, n_kv_heads=1, head_dim=128, latent_dim=512,
                       rope_dim=64, nope_dim=128, context=1, kv_std=0.5, seed=62)


def _pool(sess):
    _, gv = wsk.wsk_views(sess.h, 0)
    return d2h(gv.pool, gv.slot_bytes * sess.spec.device_pool_blocks)


@pytest.mark.parametrize("kind", ["gqa", "mla"])
def test_noalloc_step_equals_workspace_step(kind):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(DEV)
    dev = torch.device("cuda", DEV)
    w = _workload(kind)
    lengths = [9000, 4100, 700, 64, 1, 12345]
    splits = [2000, 0, 650, 64, 0, 7000]
    gen = torch.Generator().manual_seed(w.seed)
    if kind == "mla":
        ks = [wl.draw_bf16(gen, (L, w.row_elems), w.kv_std) for L in lengths]
        vs = None
    else:
        ks = [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths]
        vs = [wl.draw_bf16(gen, (L, w.n_kv_heads, w.head_dim)) for L in lengths]
    pf = wl.Prefill(lengths, splits, ks, vs, gen)
    H, dv = w.n_q_heads, (w.latent_dim if kind == "mla" else w.head_dim)
    g = H if kind == "mla" else w.group
    say("case noalloc", kind)
    with DecodeSession(w, pf, DEV, extra_tokens=4) as a, DecodeSession(w, pf, DEV, extra_tokens=4) as b:
        for call, ids in enumerate(([0, 1, 2, 3, 4, 5], [5, 2, 4])):     # the second call is smaller
            n = len(ids)
            q_bits = wl.draw_bf16(gen, (n, H, w.row_elems))
            if kind == "mla":
                kn, vn = wl.draw_bf16(gen, (n, w.row_elems), w.kv_std), None
            else:
                kn = wl.draw_bf16(gen, (n, w.n_kv_heads, w.head_dim))
                vn = wl.draw_bf16(gen, (n, w.n_kv_heads, w.head_dim))
            # CPU partial of [0, s_b) from the oracle, merged by both calls
            o_x, l_x = [], []
            for i, sq in enumerate(ids):
                v = None if vs is None else np.asarray(vs[sq])
                o_c, l_c = oracle.attend(q_bits[i], ks[sq], v, 0, splits[sq], w.softmax_scale, g, dv=dv)
                o_x.append(o_c)
                l_x.append(l_c)
            o_xd = torch.from_numpy(np.stack(o_x).astype(np.float32)).to(dev)
            l_xd = torch.from_numpy(np.stack(l_x).astype(np.float32)).to(dev)
            q, knd = to_device_bf16(q_bits, dev), to_device_bf16(kn, dev)
            vnd = None if vn is None else to_device_bf16(vn, dev)
            o_a, l_a = a.decode_step(q, knd, vnd, o_x=o_xd, lse_x=l_xd, ids=ids)
            o_b = torch.empty(n, H, dv, device=dev)
            l_b = torch.empty(n, H, device=dev)
            wsk.wsk_decode_step_noalloc(b.h, ids, q, knd, vnd, o_b, l_b, o_x=o_xd, lse_x=l_xd)
            for sq in ids:
                b.lengths[sq] += 1
            torch.cuda.synchronize()
            o_a, l_a, o_b, l_b = o_a.cpu().numpy(), l_a.cpu().numpy(), o_b.cpu().numpy(), l_b.cpu().numpy()
            assert np.array_equal(o_a, o_b) and np.array_equal(l_a, l_b), "call %d: outputs differ" % call
            assert np.array_equal(_pool(a), _pool(b)), "call %d: pools differ" % call
            for sq in ids:
                assert wsk.wsk_seq_info(a.h, sq) == wsk.wsk_seq_info(b.h, sq)
            for i, sq in enumerate(ids):
                ks[sq] = np.concatenate([ks[sq], kn[i:i + 1]])
                if vs is not None:
                    vs[sq] = np.concatenate([vs[sq], vn[i:i + 1]])
            ref_o, ref_l = [], []
            for i, sq in enumerate(ids):
                v = None if vs is None else vs[sq]
                o_r, l_r = oracle.attend(q_bits[i], ks[sq], v, 0, ks[sq].shape[0], w.softmax_scale, g, dv=dv)
                ref_o.append(o_r)
                ref_l.append(l_r)
            assert_close(o_b, np.stack(ref_o), "noalloc %s call %d" % (kind, call))
            assert_lse(l_b, np.stack(ref_l), "noalloc %s call %d" % (kind, call))


def test_noalloc_refuses_a_step_beyond_its_scratch():
    """600 sequences of 64 query heads each need one chunk partial of
    64 x 129 floats (about 19.8 MB in all, beyond the 16 MiB scratch): the
    call is refused before any launch and every length stays as it was."""
    torch.cuda.set_device(DEV)
    dev = torch.device("cuda", DEV)
    n = 600
    spec = wsk.make_spec(wsk.KIND_GQA, 64, 1, 128, 64, n, 256, 2 * n, 0, 0.088)
    h = wsk.wsk_init(spec, DEV)
    try:
        for sq in range(n):
            wsk.wsk_seq_open(h, sq, 0)
            wsk.wsk_reserve(h, sq, 70)
        ids = list(range(n))
        need = wsk.wsk_decode_step_workspace(h, ids)
        say("  %d sequences need %d bytes of partials (scratch %d)" % (n, need, 16 << 20))
        assert need > (16 << 20)
        q = torch.zeros(n, 64, 128, dtype=torch.bfloat16, device=dev)
        kn = torch.zeros(n, 1, 128, dtype=torch.bfloat16, device=dev)
        o = torch.empty(n, 64, 128, device=dev)
        lse = torch.empty(n, 64, device=dev)
        with pytest.raises(wsk.WskError) as ex:
            wsk.wsk_decode_step_noalloc(h, ids, q, kn, kn, o, lse)
        assert ex.value.name == "ERANGE", str(ex.value)
        assert all(wsk.wsk_seq_info(h, sq)[0] == 70 for sq in ids)
    finally:
        torch.cuda.synchronize()
        wsk.wsk_destroy(h)
