"""The hand-derived eviction fixture (tests/golden/route_flush.json) replayed
through the library on the GPU: evictions of several sequences listed out of
order to the CPU partition and the load region (wsk_flush), with every route
bit-exact against the hand-derived slots (Sec. 4.1-4.2: block-granular
routing; evicted batches never move again), and then the whole CPU + GPU
attention of every sequence against the fp64 oracle, which checks that each
batch's bytes landed in the slots the routes name."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_14507_amd import workloads as wl
from paper_2609_14507_amd import wsk
from tests.gpu_util import assert_close, assert_lse, say
from tests.test_oracle import expand_runs

pytestmark = pytest.mark.gpu
DEV = 0
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _scaled_ops(g, scale):
    """Positions, lengths and batch sizes times `scale` (the library's smallest
    block is 64 tokens, the fixture's 4); one appended position becomes `scale`."""
    out = []
    for op in g["ops"]:
        op = dict(op)
        for key in ("split", "pos0", "n", "length"):
            if key in op:
                op[key] *= scale
        if "moved" in op:
            op["moved"] = [m * scale for m in op["moved"]]
        if op["op"] == "expect_runs":
            op["runs"] = [[a * scale, e * scale, part, slot] for a, e, part, slot in op["runs"]]
        out.extend([op] * scale if op["op"] == "append" else [op])
    return out


def test_flush_fixture_routes_and_bytes():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(DEV)
    dev = torch.device("cuda", DEV)
    with open(os.path.join(GOLDEN, "route_flush.json")) as f:
        g = json.load(f)
    bk = 64
    scale = bk // g["block_tokens"]
    Hq, Hkv, D = 8, 2, 128
    max_len = 40 * scale
    spec = wsk.make_spec(wsk.KIND_GQA, Hq, Hkv, D, bk, 4, max_len, g["device_blocks"], g["host_blocks"],
                         1.0 / np.sqrt(D), evict_tokens=g["evict_tokens"] * scale,
                         load_pool_blocks=g["load_blocks"], load_arena_blocks=4, pingpong_blocks=2)
    gen = torch.Generator().manual_seed(41)
    K = [wl.draw_bf16(gen, (max_len, Hkv, D)) for _ in range(4)]
    V = [wl.draw_bf16(gen, (max_len, Hkv, D)) for _ in range(4)]
    length = {}
    h = wsk.wsk_init(spec, DEV)

    def check_attention(when):
        """Every open sequence: the CPU engine over its CPU segments, the GPU
        side (load region streamed, D-window in place), one LSE join, against
        attention over [0, L)."""
        ids = sorted(length)
        q = wl.draw_bf16(gen, (len(ids), Hq, D))
        o_c = np.empty((len(ids), Hq, D), np.float32)
        l_c = np.empty((len(ids), Hq), np.float32)
        wsk.wsk_cpu_attend_all(h, ids, q, o_c, l_c, 4)
        qd = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).to(dev)
        o = torch.empty(len(ids), Hq, D, device=dev)
        lse = torch.empty(len(ids), Hq, device=dev)
        ws = torch.empty(wsk.wsk_attend_gpu_workspace(h, ids), dtype=torch.uint8, device=dev)
        wsk.wsk_attend_gpu(h, ids, qd, o, lse, ws, torch.from_numpy(o_c).to(dev), torch.from_numpy(l_c).to(dev))
        torch.cuda.synchronize()
        o, lse = o.cpu().numpy(), lse.cpu().numpy()
        for i, sq in enumerate(ids):
            L = length[sq]
            o_r, l_r = oracle.attend(q[i], K[sq][:L], V[sq][:L], 0, L, 1.0 / np.sqrt(D), Hq // Hkv)
            assert_close(o[i], o_r, "seq %d %s" % (sq, when))
            assert_lse(lse[i], l_r, "seq %d %s" % (sq, when))

    say("flush fixture: Bk %d, D %d, %d ops" % (bk, g["evict_tokens"] * scale, len(g["ops"])))
    try:
        for op in _scaled_ops(g, scale):
            kind, err = op["op"], op.get("error")
            try:
                if kind == "open":
                    wsk.wsk_seq_open(h, op["seq"], op["split"])
                    length[op["seq"]] = 0
                elif kind == "write":
                    sq, a, n = op["seq"], op["pos0"], op["n"]
                    wsk.wsk_write(h, sq, a, K[sq][a:a + n], V[sq][a:a + n])
                    length[sq] += n
                elif kind == "append":
                    ids = op["seqs"]
                    kn = np.stack([K[sq][length[sq]] for sq in ids])
                    vn = np.stack([V[sq][length[sq]] for sq in ids])
                    to_dev = lambda x: torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
                    wsk.wsk_append(h, ids, to_dev(kn), to_dev(vn))
                    torch.cuda.synchronize()
                    for sq in ids:
                        length[sq] += 1
                elif kind == "flush":
                    moved = wsk.wsk_flush(h, op["seqs"], op["parts"])
                    torch.cuda.synchronize()
                    assert list(moved) == op["moved"], (op, moved)
                elif kind == "close":
                    check_attention("before closing sequence %d" % op["seq"])
                    wsk.wsk_seq_close(h, op["seq"])
                    del length[op["seq"]]
                elif kind == "expect_runs":
                    want = expand_runs(op["runs"], bk)
                    assert wsk.wsk_seq_info(h, op["seq"])[0] == len(want), op
                    got = [list(wsk.wsk_route(h, op["seq"], p)) for p in range(len(want))]
                    assert got == want, ("routes differ", op["seq"],
                                         next(i for i in range(len(want)) if got[i] != want[i]))
                elif kind == "expect_length":
                    assert wsk.wsk_seq_info(h, op["seq"])[0] == op["length"], op
            except wsk.WskError as ex:
                assert err == ex.name, (op, str(ex))
                continue
            assert err is None, ("expected failure", op)
        check_attention("at the end")
    finally:
        torch.cuda.synchronize()
        wsk.wsk_destroy(h)
