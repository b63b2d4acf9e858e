"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: an
independent library routine (torch's fp64 SDPA, logsumexp, scipy's softmax,
torch's bf16 rounding), a closed form, an invariant the paper states (exact
LSE merge of disjoint ranges, Sec. 5.1), brute force, or values the paper
prints (tests/golden/).  A dropped term, a wrong sign, index or scale, or a
transposed operand in the oracle fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle.route import CPU, GPU, LOAD, RouteError, RouteModel
from paper_2609_14507_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16(rng, shape, std=1.0):
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * std)
    return wl.bf16_bits(x.to(torch.bfloat16))


def _f64(bits):
    return torch.from_numpy(oracle.bf16_to_f64(bits))


def _case(rng, H, G, T, dk=128, dv=128, std=1.0):
    Hkv = H // G
    q = _bf16(rng, (H, dk))
    k = _bf16(rng, (T, Hkv, dk), std)
    v = _bf16(rng, (T, Hkv, dv), std)
    return q, k, v


def _sdpa_ref(q, k, v, a, e, scale, G):
    """torch fp64 SDPA over [a, e) with KV heads repeated to query heads (HF repeat_kv)."""
    qq = _f64(q)[None, :, None, :]                                    # [1, H, 1, dk]
    kk = _f64(k[a:e]).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]  # [1, H, T, dk]
    vv = _f64(v[a:e]).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=scale)[0, :, 0]
    lse = torch.logsumexp(scale * (qq @ kk.transpose(-1, -2))[0, :, 0], dim=-1)
    return o.numpy(), lse.numpy()


def _rel(x, y):
    return float(np.max(np.abs(x - y)) / max(np.max(np.abs(y)), 1e-300))


@pytest.mark.parametrize("H,G,T,a,e", [
    (8, 4, 200, 0, 200),      # GQA
    (8, 4, 200, 37, 161),     # GQA, interior range
    (4, 1, 64, 3, 64),        # G = 1: plain multi-head attention
    (6, 6, 90, 10, 80),       # G = H: multi-query attention
    (8, 2, 33, 5, 6),         # a single key
])
def test_attend_matches_torch_sdpa(H, G, T, a, e):
    rng = np.random.default_rng(100 + H * T + a)
    q, k, v = _case(rng, H, G, T)
    scale = 1 / math.sqrt(128)
    o, lse = oracle.attend(q, k, v, a, e, scale, G)
    o_ref, lse_ref = _sdpa_ref(q, k, v, a, e, scale, G)
    assert _rel(o, o_ref) < 1e-12
    assert np.max(np.abs(lse - lse_ref)) < 1e-12


def test_head_to_kv_mapping_is_contiguous_groups():
    """Query head h reads KV head floor(h/G): changing KV head g moves exactly heads gG..gG+G-1."""
    rng = np.random.default_rng(7)
    q, k, v = _case(rng, 8, 4, 40)
    o1, _ = oracle.attend(q, k, v, 0, 40, 0.1, 4)
    v2 = v.copy()
    v2[:, 1, :] = _bf16(rng, (40, 128))
    o2, _ = oracle.attend(q, k, v2, 0, 40, 0.1, 4)
    changed = np.any(o1 != o2, axis=1)
    assert changed.tolist() == [False] * 4 + [True] * 4


def test_split_invariance_every_split_point():
    """Sec. 5.1: partial outputs over [0, s) and [s, L) merge exactly to the unsplit result."""
    rng = np.random.default_rng(11)
    H, G, L = 4, 2, 48
    q, k, v = _case(rng, H, G, L, dk=32, dv=24)
    scale = 0.3
    o_full, lse_full = oracle.attend(q, k, v, 0, L, scale, G)
    for s in range(L + 1):
        o_c, l_c = oracle.attend(q, k, v, 0, s, scale, G)
        o_g, l_g = oracle.attend(q, k, v, s, L, scale, G)
        o_m, l_m = oracle.merge(o_c, l_c, o_g, l_g)
        assert _rel(o_m, o_full) < 1e-12, s
        assert np.max(np.abs(l_m - lse_full)) < 1e-12, s
        # LSE of the whole range is the logaddexp of the two sides
        assert np.max(np.abs(np.logaddexp(l_c, l_g) - lse_full)) < 1e-12


def test_empty_range_and_empty_side_merge():
    """s = 0 and s = L: an empty side is O = 0, LSE = -inf and merges to the other side bitwise."""
    rng = np.random.default_rng(12)
    q, k, v = _case(rng, 4, 2, 20)
    o_e, l_e = oracle.attend(q, k, v, 7, 7, 0.2, 2)
    assert np.all(o_e == 0) and np.all(l_e == -np.inf)
    o, l = oracle.attend(q, k, v, 0, 20, 0.2, 2)
    for a_side, b_side in (((o_e, l_e), (o, l)), ((o, l), (o_e, l_e))):
        o_m, l_m = oracle.merge(*a_side, *b_side)
        assert np.array_equal(o_m, o) and np.array_equal(l_m, l)
    o_m, l_m = oracle.merge(o_e, l_e, o_e, l_e)
    assert np.all(o_m == 0) and np.all(l_m == -np.inf)


def test_softmax_rows_sum_to_one():
    """With one-hot values, O is the probability row: it sums to 1 and equals scipy's softmax."""
    rng = np.random.default_rng(13)
    H, T, dk = 4, 16, 32
    q = _bf16(rng, (H, dk))
    k = _bf16(rng, (T, 1, dk), 2.0)
    v = np.zeros((T, 1, T), np.uint16)
    for j in range(T):
        v[j, 0, j] = 0x3F80                    # bf16 1.0
    scale = 0.5
    o, lse = oracle.attend(q, k, v, 0, T, scale, H)
    assert np.max(np.abs(o.sum(axis=1) - 1.0)) < 1e-12
    s = scale * (oracle.bf16_to_f64(q) @ oracle.bf16_to_f64(k[:, 0, :]).T)
    assert np.max(np.abs(o - scipy.special.softmax(s, axis=1))) < 1e-13
    assert np.max(np.abs(lse - scipy.special.logsumexp(s, axis=1))) < 1e-12


def test_single_token_returns_value_exactly():
    rng = np.random.default_rng(14)
    q, k, v = _case(rng, 8, 4, 5)
    o, lse = oracle.attend(q, k, v, 3, 4, 0.125, 4)
    for h in range(8):
        assert np.array_equal(o[h], oracle.bf16_to_f64(v[3, h // 4]))
        s0 = math.fsum(oracle.bf16_to_f64(q[h]) * oracle.bf16_to_f64(k[3, h // 4])) * 0.125
        assert abs(lse[h] - s0) <= 1e-13 * max(1.0, abs(s0))


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(15)
    _, k, v = _case(rng, 4, 4, 30)
    q = np.zeros((4, 128), np.float64)
    o, lse = oracle.attend(q, k, v, 4, 29, 1.0, 4)
    mean = oracle.bf16_to_f64(v[4:29, 0]).mean(axis=0)
    assert np.max(np.abs(o - mean[None])) < 1e-14
    assert np.max(np.abs(lse - math.log(25))) < 1e-14


def test_key_permutation_invariance():
    rng = np.random.default_rng(16)
    q, k, v = _case(rng, 4, 2, 64)
    perm = rng.permutation(64)
    o1, l1 = oracle.attend(q, k, v, 0, 64, 0.09, 2)
    o2, l2 = oracle.attend(q, k[perm], v[perm], 0, 64, 0.09, 2)
    assert _rel(o1, o2) < 1e-13 and np.max(np.abs(l1 - l2)) < 1e-13


def test_merge_commutative_associative_and_doubling():
    rng = np.random.default_rng(17)
    parts = [(rng.standard_normal((5, 16)), rng.standard_normal(5) * 3) for _ in range(3)]
    (oa, la), (ob, lb), (oc, lc) = parts
    m1 = oracle.merge(oa, la, ob, lb)
    m2 = oracle.merge(ob, lb, oa, la)
    assert np.array_equal(m1[0], m2[0]) and np.array_equal(m1[1], m2[1])
    left = oracle.merge(*oracle.merge(oa, la, ob, lb), oc, lc)
    right = oracle.merge(oa, la, *oracle.merge(ob, lb, oc, lc))
    assert np.max(np.abs(left[0] - right[0])) < 1e-14
    assert np.max(np.abs(left[1] - right[1])) < 1e-14
    od, ld = oracle.merge(oa, la, oa, la)
    assert np.array_equal(od, oa)
    assert np.max(np.abs(ld - (la + math.log(2)))) < 1e-15


def test_merge_weights_follow_lse():
    """A side whose LSE is ln(w) larger carries w times the weight of the other."""
    oa = np.full((1, 4), 2.0)
    ob = np.full((1, 4), -1.0)
    o, l = oracle.merge(oa, np.array([math.log(3.0)]), ob, np.array([0.0]))
    assert np.max(np.abs(o - (3 * 2.0 + 1 * -1.0) / 4)) < 1e-15
    assert abs(l[0] - math.log(4.0)) < 1e-15


def test_mla_absorbed_equals_explicit_multihead():
    """Sec. 6.1: absorbing W_UK into the query and expanding with W_UV after attention over
    the shared latent equals multi-head attention with per-head keys [W_UK c; r] and
    values W_UV^T c (fp64 identity, checked against torch SDPA)."""
    rng = np.random.default_rng(18)
    H, dn, dl, dr, dv, T = 4, 16, 32, 8, 12, 50
    c_rows = _bf16(rng, (T, dl + dr), 0.5)           # latent | rope per token
    q_nope = _bf16(rng, (H, dn))
    q_rope = _bf16(rng, (H, dr))
    w_uk = _bf16(rng, (H, dn, dl), 0.25)
    w_uv = _bf16(rng, (H, dl, dv), 0.2)
    scale = 1 / math.sqrt(dn + dr)
    q_lat = oracle.mla_absorb(q_nope, w_uk)
    q_full = np.concatenate([q_lat, oracle.bf16_to_f64(q_rope)], axis=1)
    o_lat, lse = oracle.attend(q_full, c_rows, None, 5, 45, scale, H, dv=dl)
    o = oracle.mla_expand(o_lat, w_uv)

    C = _f64(c_rows[:, :dl])
    R = _f64(c_rows[:, dl:])
    Wk, Wv = _f64(w_uk), _f64(w_uv)
    keys = torch.cat([torch.einsum("hil,tl->hti", Wk, C), R[None].expand(H, T, dr)], dim=2)
    vals = torch.einsum("hlj,tl->htj", Wv, C)
    qq = torch.cat([_f64(q_nope), _f64(q_rope)], dim=1)
    ref = torch.nn.functional.scaled_dot_product_attention(
        qq[None, :, None], keys[None, :, 5:45], vals[None, :, 5:45], scale=scale)[0, :, 0]
    ref_lse = torch.logsumexp(scale * torch.einsum("hi,hti->ht", qq, keys[:, 5:45]), dim=1)
    assert _rel(o, ref.numpy()) < 1e-10
    assert np.max(np.abs(lse - ref_lse.numpy())) < 1e-10


def test_mla_absorb_expand_match_matmul():
    rng = np.random.default_rng(19)
    q_nope = _bf16(rng, (3, 8))
    w = _bf16(rng, (3, 8, 10))
    ref = np.einsum("hi,hil->hl", oracle.bf16_to_f64(q_nope), oracle.bf16_to_f64(w))
    assert np.max(np.abs(oracle.mla_absorb(q_nope, w) - ref)) < 1e-13
    o_lat = rng.standard_normal((3, 10))
    w2 = _bf16(rng, (3, 10, 6))
    ref2 = np.einsum("hl,hlj->hj", o_lat, oracle.bf16_to_f64(w2))
    assert np.max(np.abs(oracle.mla_expand(o_lat, w2) - ref2)) < 1e-13


def test_bf16_rounding_matches_torch_and_edge_cases():
    rng = np.random.default_rng(20)
    x32 = (rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))).astype(np.float32)
    ref = wl.bf16_bits(torch.from_numpy(x32).to(torch.bfloat16))
    assert np.array_equal(oracle.round_bf16(x32.astype(np.float64)), ref)
    one = 1.0
    ulp = 2.0 ** -7
    cases = {
        one + ulp / 2: 0x3F80,               # tie -> even (1.0)
        one + 3 * ulp / 2: 0x3F82,           # tie -> even (1 + 2 ulp)
        one + ulp / 2 + 1e-12: 0x3F81,       # just above the tie
        -0.0: 0x8000,
        3.4e38: 0x7F80,                      # rounds past the largest finite bf16
        2.0 ** -133: 0x0001,                 # smallest bf16 subnormal
        -(2.0 ** -126): 0x8080,
    }
    for val, bits in cases.items():
        assert int(oracle.round_bf16(np.array([val]))[0]) == bits, val


# ---------------------------------------------------------------------------
# Routing oracle
# ---------------------------------------------------------------------------

def _replay(model, ops):
    for op in ops:
        kind = op["op"]
        err = op.get("error")
        try:
            if kind == "open":
                model.open(op["seq"], op["split"])
            elif kind == "write":
                model.write(op["seq"], op["pos0"], op["n"])
            elif kind == "append":
                model.append(op["seqs"])
            elif kind == "close":
                model.close(op["seq"])
            elif kind == "flush":
                moved = model.flush(op["seqs"], op["parts"])
                assert moved == op["moved"], (op, moved)
            elif kind == "expect_route":
                got = [list(model.route(op["seq"], p)) for p in range(len(op["routes"]))]
                assert got == op["routes"], (op, got)
            elif kind == "expect_runs":
                want = expand_runs(op["runs"], model.bk)
                got = [list(model.route(op["seq"], p)) for p in range(len(want))]
                assert model.length[op["seq"]] == len(want), op
                assert got == want, (op, got)
            elif kind == "expect_length":
                assert model.length[op["seq"]] == op["length"]
        except RouteError as ex:
            assert err == ex.code, (op, ex)
            continue
        assert err is None, ("expected failure", op)


def expand_runs(runs, bk):
    """[a, e, part, slot] runs -> one (part, logical block, slot, offset) per position."""
    return [[part, p // bk, slot, p % bk] for a, e, part, slot in runs for p in range(a, e)]


def test_route_golden_hand_derived():
    with open(os.path.join(GOLDEN, "route_small.json")) as f:
        g = json.load(f)
    _replay(RouteModel(g["block_tokens"], g["host_blocks"], g["device_blocks"]), g["ops"])


def test_route_flush_golden_hand_derived():
    """Evictions of several sequences listed out of order, both destinations, a
    straddling block keeping its CPU slot, a batch that is not whole, an
    exhausted load region that changes nothing, and slot reuse afterwards."""
    with open(os.path.join(GOLDEN, "route_flush.json")) as f:
        g = json.load(f)
    model = RouteModel(g["block_tokens"], g["host_blocks"], g["device_blocks"], g["load_blocks"],
                       g["evict_tokens"])
    _replay(model, g["ops"])


def test_route_flush_golden_discriminates_slot_order():
    """The fixture decides the slot order: a model that takes slots in listed
    order (a planted mistake) fails it at the first out-of-order flush."""
    import heapq

    class ListedOrder(RouteModel):
        def flush(self, seqs, parts):
            batches, pending = [], {}
            for sq, part in zip(seqs, parts):
                w = self.window[sq]
                w1 = (w + self.evict) // self.bk * self.bk
                if w1 > self.length[sq]:
                    batches.append(None)
                    continue
                batches.append((w, w1))
                for blk in range(w // self.bk, w1 // self.bk):
                    if (part, sq, blk) not in self.slot and (part, sq, blk) not in pending:
                        if not self.free[part]:
                            self._undo(pending)
                            raise RouteError("ENOMEM", "pool exhausted")
                        pending[(part, sq, blk)] = heapq.heappop(self.free[part])
            self._commit(pending)
            moved = []
            for sq, part, b in zip(seqs, parts, batches):
                if b is None:
                    moved.append(0)
                    continue
                for blk in range(b[0] // self.bk, b[1] // self.bk):
                    heapq.heappush(self.free[GPU], self.slot.pop((GPU, sq, blk)))
                for p in range(*b):
                    self.homes[sq][p] = part
                self.window[sq] = b[1]
                moved.append(b[1] - b[0])
            return moved

    with open(os.path.join(GOLDEN, "route_flush.json")) as f:
        g = json.load(f)
    model = ListedOrder(g["block_tokens"], g["host_blocks"], g["device_blocks"], g["load_blocks"],
                        g["evict_tokens"])
    with pytest.raises(AssertionError):
        _replay(model, g["ops"])


@pytest.mark.parametrize("bk,L,s", [(4, 13, 6), (4, 16, 0), (4, 9, 9), (8, 30, 17), (2, 7, 3), (4, 12, 8)])
def test_route_brute_force_invariants(bk, L, s):
    """Every written position has one home; the side is fixed by s; a block straddling s
    has a slot on each side; homes never move as later positions are written."""
    m = RouteModel(bk, 64, 64)
    m.open(0, s)
    m.open(1, 0)
    m.write(1, 0, 5)
    homes = {}
    m.write(0, 0, L // 2)
    for step in range(L - L // 2):
        m.append([0, 1] if step % 2 else [1, 0])
        for p in range(m.length[0]):
            r = m.route(0, p)
            assert r[0] == (CPU if p < s else GPU)
            assert r[1] == p // bk and r[3] == p % bk
            homes.setdefault(p, r)
            assert homes[p] == r
    addrs = [(m.route(sq, p)[0], m.route(sq, p)[2], m.route(sq, p)[3])
             for sq in (0, 1) for p in range(m.length[sq])]
    assert len(addrs) == len(set(addrs))
    kstar = s // bk
    if s % bk and s < L:
        assert m.slot.get((CPU, 0, kstar)) is not None and m.slot.get((GPU, 0, kstar)) is not None


def test_route_exhaustion_changes_nothing_and_close_reclaims():
    m = RouteModel(4, 2, 3)
    m.open(0, 4)
    m.write(0, 0, 8)                     # host slot 0, device slot 0
    m.open(1, 0)
    with pytest.raises(RouteError) as ex:
        m.write(1, 0, 9)                 # needs 3 device slots, 2 free
    assert ex.value.code == "ENOMEM"
    assert m.length[1] == 0 and sorted(m.free[GPU]) == [1, 2]
    m.write(1, 0, 8)
    assert m.table(GPU, 1, 2) == [1, 2]
    m.close(0)
    m.append([1])                        # position 8 opens block 2 in the freed slot 0
    m.write(1, 9, 3)
    assert m.table(GPU, 1, 4) == [1, 2, 0, -1]
    with pytest.raises(RouteError):
        m.write(1, 12, 1)                # block 3 would need a fourth device slot


@pytest.mark.parametrize("bk,D,s,e,L0", [(4, 8, 5, 12, 14), (4, 4, 3, 3, 9), (2, 4, 0, 6, 7), (4, 8, 0, 0, 2),
                                          (8, 16, 20, 24, 30)])
def test_route_load_region_and_eviction_invariants(bk, D, s, e, L0):
    """Brute force over appends and every choice of flush destinations: homes at
    write time follow [0, s) CPU, [s, load_end) load region, then the D-window;
    a flush moves exactly the batch [w, floor((w + D)/Bk)*Bk) when it is whole,
    to its destination, once: a position that left the window never moves again;
    slots stay unique per pool and none is lost; a batch that is not whole
    changes nothing."""
    import itertools
    for dests in itertools.product((CPU, LOAD), repeat=4):
        m = RouteModel(bk, 64, 64, 64, D)
        m.open(0, s, e)
        m.write(0, 0, L0)
        for p in range(L0):
            assert m.route(0, p)[0] == (CPU if p < s else LOAD if p < e else GPU)
        placed, k = {}, 0
        for step in range(4 * D):
            m.append([0])
            w = m.window[0]
            w1 = (w + D) // bk * bk
            before = (dict(m.slot), list(m.homes[0]), m.window[0])
            moved = m.flush([0], [dests[k % 4]])[0]
            if w1 > m.length[0]:
                assert moved == 0 and (dict(m.slot), list(m.homes[0]), m.window[0]) == before
                continue
            assert moved == w1 - w and m.window[0] == w1
            for p in range(w, w1):
                assert m.route(0, p)[0] == dests[k % 4]
                assert p not in placed
            k += 1
            for p in range(m.length[0]):
                r = m.route(0, p)
                if p < m.window[0]:
                    assert r[0] != GPU
                    placed.setdefault(p, r)
                    assert placed[p] == r            # placed data never moves again
                else:
                    assert r[0] == GPU
            for part in (CPU, GPU, LOAD):            # slots unique per pool, none lost
                used = [v for (pp, _, _), v in m.slot.items() if pp == part]
                assert len(used) == len(set(used)) and len(used) + len(m.free[part]) == 64
            addrs = [(m.route(0, p)[0], m.route(0, p)[2], m.route(0, p)[3]) for p in range(m.length[0])]
            assert len(addrs) == len(set(addrs))


def test_route_eviction_exhaustion_changes_nothing():
    m = RouteModel(4, 1, 8, 1, 8)
    m.open(0, 0, 0)
    m.write(0, 0, 8)                     # GPU blocks 0, 1
    with pytest.raises(RouteError) as ex:
        m.flush([0], [LOAD])             # two load slots needed, one exists
    assert ex.value.code == "ENOMEM"
    assert m.window[0] == 0 and sorted(m.free[LOAD]) == [0] and len(m.free[GPU]) == 6
    with pytest.raises(RouteError) as ex:
        m.flush([0, 0], [CPU, CPU])
    assert ex.value.code == "EINVAL"


# ---------------------------------------------------------------------------
# Workload shapes against the paper's printed byte counts (Tables 1 and 2)
# ---------------------------------------------------------------------------

def test_token_bytes_reproduce_paper_tables():
    with open(os.path.join(GOLDEN, "paper_tables.json")) as f:
        g = json.load(f)
    per_token = {
        "qwen3-30b-a3b": wl.C2.token_bytes,
        "mixtral-8x7b": wl.C3.token_bytes,
        "deepseek-v2-lite": wl.C4.token_bytes,
    }
    assert per_token == {"qwen3-30b-a3b": 2048, "mixtral-8x7b": 4096, "deepseek-v2-lite": 1152}
    for model, tb in per_token.items():
        layers = g["layers"][model]
        kv_bs4 = tb * layers * 4 * 32768 / 1e9
        assert round(kv_bs4, 1) == g["table1_kv_gb_bs4_seq32k"][model]
        t3 = g["table2_seq32k_bs32"][model]
        full = tb * layers * 32 * 32768 / 1e9
        assert abs((t3["unpinned_gb"] + t3["pinned_gb"]) - full) < 0.011
        dwin = g["dwindow_tokens"] * 32 * tb * layers / 1e6
        assert abs(dwin - t3["dwindow_mb"]) < 0.5
        pp = g["pingpong_tokens"] * 32 * tb / 1e6
        # DS2: 1024 * 32 * 1152 B = 37.75 MB, printed as 37.8
        assert abs(pp - t3["pingpong_mb"]) <= 0.06
