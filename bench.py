"""Benchmark of the GPU-partition decode step on one MI355X.

One step = the whole hot path over one batch (wsk_decode_step): the new
token's K/V of every sequence is routed to its GPU partition, split-KV
attention covers the GPU range written so far (pass 1), then one pass 2
scores and merges the new token, stores it into the pool, and merges the
chunk partials and the CPU-range partial by their LSE (MLA: the query
absorption runs before, and wsk_decode_step_mla's pass 2 also expands the
merged latent output by W_UV).  Inputs are seeded synthetic tensors already
resident in HBM; the CPU-range partial fed to the merge is a seeded
synthetic (O, LSE) pair (the merge's cost does not depend on its values).

Timing: W untimed warmup steps, then K timed steps.  Before each step a
512 MB buffer is rewritten so the 256 MB Infinity Cache holds no KV.  One
pair of HIP events on the stream the kernels run on brackets the K
(flush + step) pairs, and others the same K flushes alone, run right before
and right after; a step's time is the difference (from the flushes' mean)
over K.  Events are not recorded between
the steps: each record leaves the GPU idle for ~5 us, which a per-step pair
would count as step time.  The pass-1 kernel alone (the roofline's kernel)
is timed the same way, K (flush + pass 1) pairs less K flushes.  K more
steps, each between its own pair of events, give the per-step median, p10
and p90 (each with one event's idle time in it); K more diagnostic steps
run the pieces as separate calls with events between them, for the
breakdown.  The algorithmic bytes of a step are the bf16 K
and V rows (MLA: latent rows) of every attended position, read once.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GPU-partition decode attention effective KV GB/s and % of HBM peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def cpu_baseline(w, pf, steps_inputs, budget_s: float):
    """The fp64 oracle, as it stands, over the same GPU ranges as the timed
    decode steps (step k attends [s_b, L_b + k + 1) with the appended rows), on
    the host's cores: steps are taken in order, sequence by sequence, until the
    time budget is spent."""
    import oracle
    B = len(pf.lengths)
    S = len(steps_inputs)
    ks, vs = [], []
    for b in range(B):   # cache rows plus every step's appended row, in place
        L = pf.lengths[b]
        k = np.empty((L + S,) + pf.k[b].shape[1:], dtype=pf.k[b].dtype)
        k[:L] = pf.k[b]
        for j, st in enumerate(steps_inputs):
            k[L + j] = st.k_new[b]
        ks.append(k)
        if pf.v is not None:
            v = np.empty((L + S,) + pf.v[b].shape[1:], dtype=pf.v[b].dtype)
            v[:L] = pf.v[b]
            for j, st in enumerate(steps_inputs):
                v[L + j] = st.v_new[b]
            vs.append(v)
    t_total, nbytes, done = 0.0, 0, 0
    for j, st in enumerate(steps_inputs):
        for b in range(B):
            L = pf.lengths[b] + j + 1
            s = min(pf.splits[b], L)
            t0 = time.perf_counter()
            if pf.v is None:   # MLA: one latent row per token, values = its latent part
                oracle.attend(st.q[b], ks[b][:L], None, s, L, w.softmax_scale, w.n_q_heads, dv=w.latent_dim)
            else:
                oracle.attend(st.q[b], ks[b][:L], vs[b][:L], s, L, w.softmax_scale, w.group)
            t_total += time.perf_counter() - t0
            nbytes += (L - s) * w.token_bytes
            done += 1
            if t_total >= budget_s:
                break
        if t_total >= budget_s:
            break
    return {
        "value": nbytes / t_total / 1e9,
        "unit": "GB/s",
        "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": "fp64 oracle over the GPU ranges of the decode steps in order, %d (sequence, step) ranges "
                  "of %d sequences x %d steps (%.2f GB of KV, %.1f s); CPU: %s"
                  % (done, B, S, nbytes / 1e9, t_total, cpu_model()),
    }


# HBM bytes per launch of the pass-1 kernel, from two rocprofv3 --pmc runs of
# this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled by
# what the same counter reads for the plain 256 MiB copy of --copy-calibration
# (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0).  Keyed by workload; valid only for the
# kernel source they were taken on (sha256), null otherwise.
TRAFFIC = {
    "qwen3-30b-a3b-b16-L32768": {
        "source": "paper_2609_14507_amd/csrc/attend_gqa.hip",
        "sha256": "3c5725ebbdfd995009107330266a6eea2eec21b5d5791d7493b3e17112d7b199",
        "fetch_bytes": 368787.1 * 1024 * 2.0,
        "write_bytes": 774.0 * 1024 * 1.0,
        "kv_bytes": 751714304,
    },
    "deepseek-v2-lite-mla-b8-L65536": {
        "source": "paper_2609_14507_amd/csrc/attend_mla.hip",
        "sha256": "4df8a57ec4065ad10e72b3e174e71bce14707792ab7dea83e03b7889f82faa92",
        "fetch_bytes": 177688.0 * 1024 * 2.0,
        "write_bytes": 7951.5 * 1024 * 1.0,
        "kv_bytes": 362414592,
    },
}


def roofline(w, kind, achieved_gbs, kv_bytes):
    """Roofline entry of the pass-1 kernel (the one that streams the KV)."""
    import hashlib
    traffic = None
    t = TRAFFIC.get(w.name)
    if t is not None:
        with open(os.path.join(ROOT, t["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() == t["sha256"]:
                traffic = t["fetch_bytes"] + t["write_bytes"]
    out = {
        "bound": "hbm",
        "kernel": "%s_attend_kernel (wsk_attend pass 1)" % kind,
        "achieved": round(achieved_gbs, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
        "traffic": None if traffic is None else int(traffic),
    }
    if traffic is not None:
        out["traffic_per_kv_byte"] = round(traffic / t["kv_bytes"], 4)
    return out


def wsk_mod():
    from paper_2609_14507_amd import wsk
    return wsk


def cpu_gpu_steps(w, sess, wsk, steps_in, i0, F, splits, qs, kn, vn, o_m, l_m, flush, dev, absorb, expand,
                  gpu_ns_per_token, gpu_fixed_us):
    """The paper's whole decode step on this machine: the GPU appends and runs pass 1
    over [s_b, L_b + 1) while the native CPU engine (wsk_cpu_attend) attends
    [0, s_b) in place in the host pool on every available core; the CPU partial
    is copied to the device and pass 2 merges it with the GPU chunks.  Timed on
    the host clock from the first launch to the end of pass 2.  Also fits the
    roofline split policy (Eq. 2) to the measured per-token costs."""
    import torch
    B, H = sess.B, w.n_q_heads
    D = sess.out_width
    threads = len(os.sched_getaffinity(0))
    ids = sess.ids
    o_c = np.empty((B, H, D), np.float32)
    l_c = np.empty((B, H), np.float32)
    o_pin = torch.empty(B, H, D, pin_memory=True)
    l_pin = torch.empty(B, H, pin_memory=True)
    o_cd = torch.empty(B, H, D, device=dev)
    l_cd = torch.empty(B, H, device=dev)
    cpu_s, full_s, cpu_tok = [], [], []
    for f in range(F):
        i = i0 + f
        ce = [min(splits[b], sess.lengths[b]) for b in range(B)]
        flush.add_(1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if absorb:
            absorb(i)
        sess.append(kn[i], vn[i])
        sess.attend_pass1(qs[i])                         # the GPU works from here on ...
        t1 = time.perf_counter()
        wsk.wsk_cpu_attend(sess.h, ids, [0] * B, ce, steps_in[i].q, o_c, l_c, threads)   # ... while the CPU does
        t2 = time.perf_counter()
        o_pin.numpy()[:] = o_c
        l_pin.numpy()[:] = l_c
        o_cd.copy_(o_pin, non_blocking=True)
        l_cd.copy_(l_pin, non_blocking=True)
        sess.attend_pass2(o=o_m, lse=l_m, o_x=o_cd, lse_x=l_cd)
        if expand:
            expand()
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        cpu_s.append(t2 - t1)
        full_s.append(t3 - t0)
        cpu_tok.append(sum(ce))
    tok = float(np.mean(cpu_tok))
    if tok == 0:
        return None, {"ms": round(float(np.median(full_s)) * 1e3, 3), "cpu_ms": 0.0,
                      "note": "no CPU range in this workload"}, None
    # fixed cost of a CPU engine call: one 16-token range per sequence
    small = []
    for _ in range(5):
        t = time.perf_counter()
        wsk.wsk_cpu_attend(sess.h, ids, [0] * B, [min(16, c) for c in ce], steps_in[i0].q, o_c, l_c, threads)
        small.append(time.perf_counter() - t)
    c_cpu = min(small)
    t_cpu = float(np.median(cpu_s))
    A = max(t_cpu - c_cpu, 1e-12) / tok
    Bc = gpu_ns_per_token * 1e-9
    # A and B are per token of the whole batch and the fixed costs are per
    # call, so Eq. 2 takes the step's token count
    L = float(np.sum(sess.lengths))
    r = wsk.wsk_roofline_share(A, Bc, c_cpu, gpu_fixed_us * 1e-6, int(L))
    # the plain host read rate on the same threads: the CPU engine's ceiling
    probe = np.ones((1 << 30) // 8, dtype=np.uint64)
    wsk.wsk_host_read(probe, threads)
    rd = []
    for _ in range(3):
        t = time.perf_counter()
        wsk.wsk_host_read(probe, threads)
        rd.append(time.perf_counter() - t)
    host_gbs = probe.nbytes / float(np.median(rd)) / 1e9
    del probe
    engine_gbs = tok * w.token_bytes / t_cpu / 1e9
    cpu_engine = {"value": round(engine_gbs, 2), "unit": "GB/s", "cores": threads,
                  "kind": "native (wsk_cpu_attend)",
                  "host_read_gbs": round(host_gbs, 2), "frac_of_host_read": round(engine_gbs / host_gbs, 4),
                  "sample": "the workload's CPU ranges [0, s_b) of %d sequences, %.0f tokens per call, median of %d; "
                            "host_read_gbs: wsk_host_read of 1 GiB on the same threads, median of 3"
                            % (B, tok, F)}
    full = {"ms": round(float(np.median(full_s)) * 1e3, 3), "cpu_ms": round(t_cpu * 1e3, 3),
            "what": "append + GPU pass 1 over [s_b, L_b] while the CPU engine attends [0, s_b), then pass 2 "
                    "merging both partials (the workload's split)"}
    policy = {"A_ns_per_token": round(A * 1e9, 4), "B_ns_per_token": round(Bc * 1e9, 4),
              "c_cpu_us": round(c_cpu * 1e6, 1), "c_gpu_us": round(gpu_fixed_us, 1), "step_tokens": int(L),
              "balanced_cpu_share": round(r, 5),
              "what": "Eq. 2 with A from the CPU engine and B from GPU pass 1 measured above"}
    log("bench: CPU engine %.1f GB/s on %d cores (plain host read %.1f GB/s); full CPU+GPU step %.2f ms; "
        "balanced CPU share %.4f" % (cpu_engine["value"], threads, host_gbs, full["ms"], r))
    return cpu_engine, full, policy


PCIE_PEAK_GBS = 63.0   # PCIe 5.0 x16, one direction: 32 GT/s x 16 lanes x 128/130 / 8


def load_region_section(w, pf, steps_in, dev, flush, n_steps=5):
    """The paper's GPU side with the GPU share in the pinned load region
    (Sec. 4.2): the prefill's GPU positions below the last 256 go to the load
    region, the rest is the D-window in HBM; a step streams the load region
    through the ping-pong pair (wsk_attend_gpu) and merges a CPU partial.
    Also the block-sparse variant (gather + one DMA per buffer), D-window
    eviction to both homes, the pinning cost, and plain host<->device copies
    (pinned vs pageable, transfer size, one DMA vs one per block) as the
    ceilings the streamed rate is compared with.  Timed on the host clock."""
    import torch
    from paper_2609_14507_amd import wsk
    from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
    from paper_2609_14507_amd import workloads as wl
    D, bk = 256, 64
    B, H = len(pf.lengths), w.n_q_heads
    load_ends = [max(s, (L - D) // bk * bk) for s, L in zip(pf.splits, pf.lengths)]
    log("load region: routing the prefill (GPU share below the last %d positions pinned)" % D)
    sess = DecodeSession(w, pf, 0, extra_tokens=D + 2, load_ends=load_ends, evict_tokens=D, pingpong_blocks=512,
                         arena_blocks=1024)
    info0 = wsk.wsk_load_stats(sess.h)
    q = to_device_bf16(steps_in[0].q, dev)
    width = sess.out_width
    o = torch.empty(B, H, width, device=dev)
    lse = torch.empty(B, H, device=dev)
    o_c, l_c = wl.draw_cpu_partial(pf.gen, B * H, width)
    o_x = torch.from_numpy(o_c).to(dev).view(B, H, width)
    l_x = torch.from_numpy(l_c).to(dev).view(B, H)

    def timed(fn, reps):
        ts = []
        for _ in range(reps):
            flush.add_(1)
            torch.cuda.synchronize()
            t = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t)
        return float(np.median(ts))

    # dense streamed step
    sess.attend_gpu(q, o_x=o_x, lse_x=l_x, o=o, lse=lse)
    torch.cuda.synchronize()
    h0 = wsk.wsk_load_stats(sess.h).h2d_bytes
    t_step = timed(lambda: sess.attend_gpu(q, o_x=o_x, lse_x=l_x, o=o, lse=lse), n_steps)
    h2d = (wsk.wsk_load_stats(sess.h).h2d_bytes - h0) / n_steps
    win = sum(L - e for L, e in zip(sess.lengths, load_ends)) * w.token_bytes
    # block-sparse: every 4th load-region block of each sequence plus its D-window blocks
    sels = []
    for b in range(B):
        segs = wsk.wsk_seq_segments(sess.h, b)
        lb = [blk for a, e, part in segs if part == wsk.PART_LOAD for blk in range(a // bk, -(-e // bk))]
        gb = [blk for a, e, part in segs if part == wsk.PART_GPU for blk in range(a // bk, -(-e // bk))]
        sels.append(lb[::4] + gb)
    need = wsk.wsk_attend_blocks_workspace(sess.h, sess.ids, sels)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    run_sparse = lambda: wsk.wsk_attend_blocks(sess.h, sess.ids, sels, q, o, lse, ws, o_x, l_x)
    run_sparse()
    torch.cuda.synchronize()
    h0 = wsk.wsk_load_stats(sess.h).h2d_bytes
    t_sparse = timed(run_sparse, n_steps)
    h2d_sparse = (wsk.wsk_load_stats(sess.h).h2d_bytes - h0) / n_steps
    # D-window eviction: one batch of D per sequence to the load region, then
    # (after D more appends) one to the CPU partition
    d0 = wsk.wsk_load_stats(sess.h).d2h_bytes
    t_fl = timed(lambda: sess.flush([wsk.PART_LOAD] * B), 1)
    d_fl = wsk.wsk_load_stats(sess.h).d2h_bytes - d0
    if w.kind == wl.MLA:
        kn, vn = torch.zeros(B, w.row_elems, dtype=torch.bfloat16, device=dev), None
    else:
        kn = torch.zeros(B, w.n_kv_heads, w.head_dim, dtype=torch.bfloat16, device=dev)
        vn = torch.zeros_like(kn)
    for _ in range(D):
        sess.append(kn, vn)
    d0 = wsk.wsk_load_stats(sess.h).d2h_bytes
    t_fc = timed(lambda: sess.flush([wsk.PART_CPU] * B), 1)
    d_fc = wsk.wsk_load_stats(sess.h).d2h_bytes - d0
    info = wsk.wsk_load_stats(sess.h)
    sess.close()

    # plain copies through the same link
    def h2d_gbs(nbytes, pinned=True, reps=3):
        src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=pinned)
        src.fill_(1)
        dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        dst.copy_(src, non_blocking=pinned)
        torch.cuda.synchronize()
        t = timed(lambda: dst.copy_(src, non_blocking=pinned), reps)
        return nbytes / t / 1e9
    ceiling = h2d_gbs(256 << 20)
    micro = {"pinned_256MiB": round(ceiling, 2), "pageable_256MiB": round(h2d_gbs(256 << 20, pinned=False), 2)}
    for label, n in (("192KiB", 192 << 10), ("1MiB", 1 << 20), ("8MiB", 8 << 20), ("64MiB", 64 << 20)):
        micro["pinned_" + label] = round(h2d_gbs(n, reps=5), 2)
    # 64 MiB as one DMA versus one DMA per 128 KiB block from scattered offsets
    blk = 128 << 10
    src = torch.empty(128 << 20, dtype=torch.uint8, pin_memory=True)
    src.fill_(2)
    dst = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    order = np.random.default_rng(0).permutation(1024)[:512]
    def per_block():
        for j, k in enumerate(order):
            dst[j * blk:(j + 1) * blk].copy_(src[int(k) * blk:(int(k) + 1) * blk], non_blocking=True)
    per_block()
    torch.cuda.synchronize()
    micro["per_block_dmas_64MiB"] = round((64 << 20) / timed(per_block, 3) / 1e9, 2)
    sect = {
        "workload": w.name,
        "what": "GPU side of a step with the GPU share in the pinned load region: load-region blocks streamed "
                "host->device through two HBM ping-pong buffers of 512 blocks while pass 1 attends the other "
                "buffer, the D-window attended in place, all merged with a CPU partial (wsk_attend_gpu); host "
                "clock, median of %d, Infinity Cache flushed before each" % n_steps,
        "bound": "pcie",
        "streamed_step_ms": round(t_step * 1e3, 3),
        "h2d_bytes_per_step": int(h2d),
        "window_bytes_per_step": int(win),
        "achieved": round(h2d / t_step / 1e9, 2),
        "peak": PCIE_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(h2d / t_step / 1e9 / PCIE_PEAK_GBS, 4),
        "copy_ceiling_gbs": round(ceiling, 2),
        "frac_of_copy_ceiling": round(h2d / t_step / 1e9 / ceiling, 4),
        "sparse_gather": {"ms": round(t_sparse * 1e3, 3), "h2d_bytes": int(h2d_sparse),
                          "gbs": round(h2d_sparse / t_sparse / 1e9, 2),
                          "what": "wsk_attend_blocks: every 4th load-region block (gathered by the host, one memcpy "
                                  "per block, one DMA per buffer) plus the D-window blocks in place"},
        "flush": {"to_load": {"ms": round(t_fl * 1e3, 3), "bytes": int(d_fl), "gbs": round(d_fl / t_fl / 1e9, 2)},
                  "to_cpu": {"ms": round(t_fc * 1e3, 3), "bytes": int(d_fc), "gbs": round(d_fc / t_fc / 1e9, 2)},
                  "what": "wsk_flush of one D = %d batch of every sequence; to the CPU includes the host's "
                          "token-major rewrite" % D},
        "pinning": {"pinned_bytes": int(info0.pinned_bytes), "arenas": int(info0.arenas),
                    "ms_per_MiB": round(info0.pin_seconds * 1e3 / max(info0.pinned_bytes / 2 ** 20, 1e-9), 4)},
        "transfer_micro_gbs": micro,
    }
    log("load region: streamed step %.2f ms, %.1f GB/s host->device (copy ceiling %.1f, pageable %.1f); sparse %.2f "
        "ms; flush to load %.2f ms, to CPU %.2f ms; pinning %.3f ms/MiB"
        % (t_step * 1e3, sect["achieved"], ceiling, micro["pageable_256MiB"], t_sparse * 1e3, t_fl * 1e3, t_fc * 1e3,
           sect["pinning"]["ms_per_MiB"]))
    return sect


def offload_section(w, pf, steps_in, dev, flush, A_s, c_cpu_s, B_s, n_steps=3):
    """The paper's step when the KV does not stay in HBM (Sec. 4.2, 5.1): each
    sequence's CPU share [0, s) is attended in place by the CPU engine while
    the GPU streams its share from the pinned load region (plus the D-window)
    and attends it; one LSE join.  Timed on the host clock at the all-GPU
    split (s = 0) and at CPU shares around the one Eq. 2 gives with A (CPU
    engine) and B (streamed GPU side) measured on this machine, next to Eq. 1's
    prediction max(r A L, (1 - r) B L) + C for each share (the paper's Fig. 7
    comparison of the model with measured optima)."""
    import torch
    from paper_2609_14507_amd import wsk
    from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
    from paper_2609_14507_amd import workloads as wl
    D, bk = 256, 64
    B, H = len(pf.lengths), w.n_q_heads
    threads = len(os.sched_getaffinity(0))
    tokens = float(sum(pf.lengths))
    # A and B are per token of the whole batch and the CPU engine's fixed cost
    # is per call, so Eq. 2 takes the step's token count
    r_star = wsk.wsk_roofline_share(A_s, B_s, c_cpu_s, 0.0, int(tokens))
    shares = sorted({0.0} | {round(min(1.0, max(0.0, r_star + d)), 4)
                             for d in (-0.2, -0.1, -0.05, 0.0, 0.05, 0.1, 0.2)})
    q_bits = np.ascontiguousarray(steps_in[0].q)
    q = to_device_bf16(q_bits, dev)
    rows = []
    for r in shares:
        splits = [wl.split_point(r, L) for L in pf.lengths]
        load_ends = [max(s, (L - D) // bk * bk) for s, L in zip(splits, pf.lengths)]
        p2 = wl.Prefill(pf.lengths, splits, pf.k, pf.v, pf.gen)
        log("offload: routing the prefill with CPU share %.3f" % r)
        sess = DecodeSession(w, p2, 0, extra_tokens=0, load_ends=load_ends, evict_tokens=D, pingpong_blocks=512,
                             arena_blocks=1024)
        width = sess.out_width
        o_c = np.empty((B, H, width), np.float32)
        l_c = np.empty((B, H), np.float32)
        o_pin = torch.empty(B, H, width, pin_memory=True)
        l_pin = torch.empty(B, H, pin_memory=True)
        o_x = torch.empty(B, H, width, device=dev)
        l_x = torch.empty(B, H, device=dev)
        o = torch.empty(B, H, width, device=dev)
        lse = torch.empty(B, H, device=dev)

        def full_step():
            sess.attend_gpu_pass1(q)                              # transfers + kernels in flight ...
            wsk.wsk_cpu_attend_all(sess.h, sess.ids, q_bits, o_c, l_c, threads)   # ... while the CPU attends
            o_pin.numpy()[:] = o_c
            l_pin.numpy()[:] = l_c
            o_x.copy_(o_pin, non_blocking=True)
            l_x.copy_(l_pin, non_blocking=True)
            sess.attend_gpu_pass2(o_x=o_x, lse_x=l_x, o=o, lse=lse)

        ts = []
        for it in range(n_steps + 1):
            flush.add_(1)
            torch.cuda.synchronize()
            t = time.perf_counter()
            full_step()
            torch.cuda.synchronize()
            if it:
                ts.append(time.perf_counter() - t)
        cpu_tok = sum(min(s, L) for s, L in zip(splits, pf.lengths))
        rr = cpu_tok / tokens
        model = max(rr * A_s * tokens + c_cpu_s, (1 - rr) * B_s * tokens)
        rows.append((r, float(np.median(ts)), cpu_tok, model))
        sess.close()
    base = rows[0][1]
    best = min(rows, key=lambda x: x[1])
    at_star = [x for x in rows if x[0] == round(r_star, 4)][0]
    out = {"what": "full decode step with the GPU share offloaded: GPU side streamed from the pinned load region "
                   "(wsk_attend_gpu_pass1) while the CPU engine attends [0, s) in place (wsk_cpu_attend_all, %d "
                   "threads), CPU partial copied over, one LSE join (wsk_attend_gpu_pass2); host clock, median of "
                   "%d, at CPU shares around Eq. 2's, with Eq. 1's prediction" % (threads, n_steps),
           "A_ns_per_token": round(A_s * 1e9, 3), "B_ns_per_token": round(B_s * 1e9, 3),
           "c_cpu_us": round(c_cpu_s * 1e6, 1), "eq2_share": round(r_star, 4),
           "sweep": [{"cpu_share": r, "ms": round(t * 1e3, 3), "model_ms": round(mdl * 1e3, 3)}
                     for r, t, _, mdl in rows],
           "measured_best_share": best[0],
           "all_gpu": {"cpu_share": 0.0, "ms": round(base * 1e3, 3)},
           "balanced": {"cpu_share": at_star[0], "ms": round(at_star[1] * 1e3, 3), "cpu_tokens": int(at_star[2]),
                        "speedup_vs_all_gpu": round(base / at_star[1], 3)}}
    log("offload: all-GPU streamed step %.2f ms; Eq. 2 share %.3f step %.2f ms (%.2fx); measured best share %.3f "
        "(%.2f ms); sweep %s" % (base * 1e3, r_star, at_star[1] * 1e3, base / at_star[1], best[0], best[1] * 1e3,
                                 [(r, round(t * 1e3, 2)) for r, t, _, _ in rows]))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c2", help="workload: c2 (default, the metric's), c1, c3, c4, c5")
    ap.add_argument("--share", type=float, default=None, help="override the CPU share (sweep configs)")
    ap.add_argument("--no-flush", action="store_true", help="skip the Infinity Cache flush between steps")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cpu-engine", action="store_true",
                    help="skip the native CPU engine and the full CPU + GPU steps")
    ap.add_argument("--no-load-region", action="store_true",
                    help="skip the streamed load-region step, eviction and transfer measurements")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run a plain 256 MiB device copy three times (the reference "
                         "dispatch that scales HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_14507_amd import workloads as wl
    from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16

    w = wl.CONFIGS[args.config]
    mla = w.kind == wl.MLA
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    K, W = args.steps, args.warmup

    log("bench: drawing %s" % w.name)
    pf = wl.make_prefill(w)
    splits = pf.splits
    if args.share is not None:
        splits = [wl.split_point(args.share, L) for L in pf.lengths]
        pf = wl.Prefill(pf.lengths, splits, pf.k, pf.v, pf.gen)
    F = 5                                    # full CPU + GPU steps after the GPU-only ones
    steps_in = [wl.draw_step(w, pf.gen) for _ in range(W + 3 * K + F)]
    log("bench: routing the prefill into the cache")
    sess = DecodeSession(w, pf, 0, extra_tokens=W + 3 * K + F)
    B, H = sess.B, w.n_q_heads
    D = sess.out_width                      # attend output width (MLA: the latent)
    qs = [to_device_bf16(s.q, dev) for s in steps_in]
    kn = [to_device_bf16(s.k_new, dev) for s in steps_in]
    vn = [None if mla else to_device_bf16(s.v_new, dev) for s in steps_in]
    if mla:
        from paper_2609_14507_amd import wsk
        w_uk, w_uv = wl.draw_mla_weights(w, pf.gen)
        w_uk_d, w_uv_d = to_device_bf16(w_uk, dev), to_device_bf16(w_uv, dev)
        qn = [to_device_bf16(s.q_nope, dev) for s in steps_in]
        o_out = torch.empty(B, H, w.head_dim, device=dev)
    o_c, l_c = wl.draw_cpu_partial(pf.gen, B * H, D)
    o_cpu = torch.from_numpy(o_c).to(dev).view(B, H, D)
    l_cpu = torch.from_numpy(l_c).to(dev).view(B, H)
    o_m = torch.empty(B, H, D, device=dev)
    l_m = torch.empty(B, H, device=dev)
    sess.workspace(sess.ids, [min(s, L) for s, L in zip(splits, pf.lengths)], list(pf.lengths))
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step(i, ev=None, parts=None):
        """One decode step.  ev = (start, end) events around the step: the timed
        steps run it as wsk_decode_step (pass 1 over the positions written so
        far, then one pass 2 that folds in the appended row, stores it and
        merges the CPU partial; MLA: wsk_decode_step_mla, whose pass 2 also
        expands the merged latent output by W_UV).  parts = 5 events around its pieces
        (diagnostic steps only, every event record costs GPU time of its own):
        those run the same work as separate calls -- append, pass 1 over
        [s, L + 1), pass 2 -- so that pass 1 is timed on its own."""
        if not args.no_flush:
            flush.add_(1)
        mark = (lambda k: parts[k].record(stream)) if parts else (lambda k: None)
        if ev:
            ev[0].record(stream)
        mark(0)
        if mla:   # query-side projection into the latent space, in place
            wsk.wsk_mla_absorb(qn[i], w_uk_d, qs[i], w.row_elems)
        if parts:
            sess.append(kn[i], vn[i])
            mark(1)
            sess.attend_pass1(qs[i])
            mark(2)
            sess.attend_pass2(o=o_m, lse=l_m, o_x=o_cpu, lse_x=l_cpu)
            mark(3)
        elif mla:
            sess.decode_step_mla(qs[i], kn[i], w_uv_d, o=o_out, lse=l_m, o_x=o_cpu, lse_x=l_cpu)
        else:
            sess.decode_step(qs[i], kn[i], vn[i], o_x=o_cpu, lse_x=l_cpu, o=o_m, lse=l_m)
        if mla and parts:   # output-side expansion of the merged latent output
            wsk.wsk_mla_expand(o_m, w_uv_d, o_out)
            mark(4)
        if ev:
            ev[1].record(stream)

    def kv_bytes():   # algorithmic bytes of the next step: [s_b, L_b + 1) of every sequence
        return sum((sess.lengths[b] + 1 - min(splits[b], sess.lengths[b])) * w.token_bytes for b in range(B))

    def bracket(fn):   # ms of fn() on the stream, one event pair around it
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        for _ in range(3):   # a GPU backlog ahead of the bracket: the host then runs ahead of
            flush.add_(1)    # the timed launches, and a host stall cannot idle the GPU inside it
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def flushes():
        if not args.no_flush:
            for _ in range(K):
                flush.add_(1)

    ev_part = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K)]
    log("bench: %d warmup + %d timed steps (+ %d diagnostic steps with per-part events)" % (W, K, K))
    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    nbytes = []

    def timed_steps():
        for k in range(K):
            nbytes.append(kv_bytes())
            step(W + k)
    t_flush_a = bracket(flushes)
    t0 = time.perf_counter()
    t_steps = bracket(timed_steps)
    wall = time.perf_counter() - t0
    t_flush = 0.5 * (t_flush_a + bracket(flushes))   # flushes timed before and after: drift cancels
    step_ms = (t_steps - t_flush) / K

    # the pass-1 kernel alone, K launches over the current GPU ranges
    p1_bytes = float(sum((sess.lengths[b] - min(splits[b], sess.lengths[b])) * w.token_bytes for b in range(B)))

    def pass1s():
        for k in range(K):
            if not args.no_flush:
                flush.add_(1)
            sess.attend_pass1(qs[W + k])
    t_p1 = bracket(pass1s)
    t_flush2 = 0.5 * (t_flush + bracket(flushes))
    p1_kernel_ms = (t_p1 - t_flush2) / K

    # the per-step distribution: K more steps, each between its own pair of
    # events (each pair counts one event's idle time, ~5.5 us, as step time)
    ev_step = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    for k in range(K):
        step(W + K + k, ev=ev_step[k])
    torch.cuda.synchronize()
    ev_us = np.array([e[0].elapsed_time(e[1]) for e in ev_step]) * 1e3

    d_bytes = []
    for k in range(K):
        d_bytes.append(kv_bytes())
        step(W + 2 * K + k, parts=ev_part[k])
    torch.cuda.synchronize()
    el = lambda a, b: np.array([e[a].elapsed_time(e[b]) for e in ev_part])
    app_ms, p1_ms, p2_ms = el(0, 1), el(1, 2), el(2, 3)
    exp_ms = el(3, 4) if mla else np.zeros(K)
    nbytes = np.array(nbytes, dtype=np.float64)
    d_bytes = np.array(d_bytes, dtype=np.float64)
    value = float(nbytes.mean() / (step_ms * 1e-3) / 1e9)
    att_gbs = float(d_bytes.sum() / ((p1_ms + p2_ms).sum() * 1e-3) / 1e9)
    p1_gbs = float(p1_bytes / (p1_kernel_ms * 1e-3) / 1e9)
    log("bench: step %.1f us (%.1f us per flush + step less %.1f us per flush); pass 1 alone %.1f us, %.0f GB/s; "
        "diagnostic steps (events between parts): absorb+append %.1f, attend pass 1 %.1f, pass 2 with merge %.1f, "
        "expand %.1f us; wall %.1f ms/step"
        % (step_ms * 1e3, t_steps / K * 1e3, t_flush / K * 1e3, p1_kernel_ms * 1e3, p1_gbs, app_ms.mean() * 1e3,
           p1_ms.mean() * 1e3, p2_ms.mean() * 1e3, exp_ms.mean() * 1e3, wall / K * 1e3))
    cpu_engine, full_step, policy = None, None, None
    if not args.no_cpu_engine:
        cpu_engine, full_step, policy = cpu_gpu_steps(
            w, sess, wsk_mod(), steps_in, W + 3 * K, F, splits, qs, kn, vn, o_m, l_m, flush, dev,
            None,   # MLA: the drawn absorbed query feeds both engines (no absorb launch)
            (lambda: wsk_mod().wsk_mla_expand(o_m, w_uv_d, o_out)) if mla else None,
            gpu_ns_per_token=float(p1_kernel_ms * 1e6 / (p1_bytes / w.token_bytes)),
            gpu_fixed_us=float((step_ms - p1_kernel_ms) * 1e3))
    sess.close()
    load_region = None if args.no_load_region else load_region_section(w, pf, steps_in, dev, flush)
    offload = None
    if load_region is not None and policy is not None:
        offload = offload_section(w, pf, steps_in, dev, flush, policy["A_ns_per_token"] * 1e-9,
                                  policy["c_cpu_us"] * 1e-6, w.token_bytes / (load_region["achieved"] * 1e9))
    # plain streaming read of 2 GiB with the attention kernels' load pattern:
    # the practical HBM read ceiling the pass-1 rate is compared with
    from paper_2609_14507_amd import wsk as _wsk
    probe = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    probe.fill_(3)
    fold = torch.zeros(1, dtype=torch.int32, device=dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count

    def read_gbs(workgroups):
        ms = []
        for it in range(6):
            flush.add_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            _wsk.wsk_stream_read(probe, fold, workgroups)
            e1.record(stream)
            torch.cuda.synchronize()
            if it:
                ms.append(e0.elapsed_time(e1))
        return float(probe.numel() / (np.median(ms) * 1e-3) / 1e9)
    probe_gbs = read_gbs(0)
    probe_sweep = {str(n): round(read_gbs(n), 1) for n in (cus // 2, cus * 3 // 4, cus, 2 * cus, 4 * cus)}
    del probe
    log("bench: streaming-read probe %.0f GB/s; by workgroups %s" % (probe_gbs, probe_sweep))
    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        for _ in range(3):
            flush.add_(1)
            dst.copy_(src)
        torch.cuda.synchronize()
        log("bench: copy calibration: 3 x %d bytes read + written" % src.numel())

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(float(step_ms), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": B,
            "q_heads": w.n_q_heads,
            "kv_heads": w.n_kv_heads,
            "head_dim": w.head_dim,
            **({"latent_dim": w.latent_dim, "rope_dim": w.rope_dim, "nope_dim": w.nope_dim} if mla else {}),
            "context": w.context if w.context else [w.ragged_lo, w.ragged_hi],
            "cpu_share": args.share if args.share is not None else (w.cpu_share or [w.share_lo, w.share_hi]),
            "gpu_tokens_per_step": int(nbytes.mean() / w.token_bytes),
            "kv_bytes_per_step": int(nbytes.mean()),
            "step": ("absorb + wsk_decode_step_mla (attend pass 1 over [s, L), then one pass 2: the appended row "
                     "scored, merged and stored, chunk combine, LSE merge with the CPU partial, expansion by W_UV)"
                     if mla else "wsk_decode_step: attend pass 1 over [s, L), then one pass 2: the appended row "
                     "scored, merged and stored, chunk combine, LSE merge with the CPU partial"),
            "cache_flush_between_steps": not args.no_flush,
        },
        "breakdown_us": {
            "step": round(step_ms * 1e3, 2),
            "flush_plus_step": round(t_steps / K * 1e3, 2),
            "flush": round(t_flush / K * 1e3, 2),
            "pass1_kernel": round(p1_kernel_ms * 1e3, 2),
            "step_event_pairs": {"median": round(float(np.median(ev_us)), 2),
                                 "p10": round(float(np.percentile(ev_us, 10)), 2),
                                 "p90": round(float(np.percentile(ev_us, 90)), 2),
                                 "what": "K more steps, each between its own pair of events: the per-step "
                                         "spread; each includes one event record's idle time (~5.5 us)"},
            "wall_per_step_incl_flush": round(wall / K * 1e6, 1),
            "diagnostic_steps": "K more steps with events between the parts (each record adds ~5 us of GPU "
                                "idle time to the part it closes)",
            ("absorb_append" if mla else "append"): round(float(app_ms.mean() * 1e3), 2),
            "attend_pass1": round(float(p1_ms.mean() * 1e3), 2),
            "attend_pass2_combine_merge": round(float(p2_ms.mean() * 1e3), 2),
            **({"expand": round(float(exp_ms.mean() * 1e3), 2)} if mla else {}),
            "attend_gbs": round(att_gbs, 1),
        },
        "roofline": roofline(w, "mla" if mla else "gqa", p1_gbs, p1_bytes),
        "stream_read_probe": {"value": round(probe_gbs, 1), "unit": "GB/s", "bytes": 2 << 30,
                              "by_workgroups": probe_sweep,
                              "what": "wsk_stream_read: one plain read of 2 GiB with the attention kernels' "
                                      "loads by 4-wavefront workgroups (value: 3/4 of the CUs, the GQA grid's "
                                      "aim), median of 5, cache flushed before each"},
    }
    if load_region is not None:
        out["load_region"] = load_region
    if offload is not None:
        out["offload_step"] = offload
    if cpu_engine is not None:
        out["cpu_engine"] = cpu_engine
        out["full_step"] = full_step
        out["split_policy"] = policy
    if not args.no_cpu_baseline:
        log("bench: timing the oracle on the host (%.0f s budget)" % args.cpu_budget)
        out["cpu_baseline"] = cpu_baseline(w, pf, steps_in, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
