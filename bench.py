"""Benchmark of the GPU-partition decode step on one MI355X.

The headline workload is the largest single-GPU configuration: the ragged
1M-token aggregate (Qwen3-30B-A3B attention shape, 8 sequences of 98K-164K
tokens, per-sequence CPU shares of 10-60 %), run as its 64 decode steps.  One
step = the whole hot path over one batch (wsk_decode_step, one kernel launch
for GQA): the new token's K/V of every sequence is routed to its GPU
partition, split-KV attention covers the GPU range written so far (pass 1),
and the last workgroup of each (sequence, KV head, head group) scores and
merges the new token, stores it into the pool, and merges the chunk partials
and the CPU-range partial by their LSE (pass 2).  The W warmup steps append the last W
rows of the drawn context, so the K timed steps start exactly at the drawn
lengths.  Inputs are seeded synthetic tensors already resident in HBM; the
CPU-range partial fed to the merge is a seeded synthetic (O, LSE) pair (the
merge's cost does not depend on its values).

The same JSON line carries the other model shapes ("configs"): the
Mixtral-8x7B shape swept over CPU shares {0, .25, .5, .75} on ONE cache
written with s = 0 (only the attend range changes between sweep points: pass
1 over [s', L) and pass 2 merging the CPU partial), the DeepSeek-V2-Lite MLA
shape (query absorption + wsk_decode_step_mla, whose pass 2 also expands by
W_UV), the Qwen3 shape at batch 16 x 32K (with the native CPU engine, the
pinned load region, eviction and the offloaded step measured after it), and
the tiny single-sequence case.

Timing of every decode workload: before each step a 512 MB buffer is read
through the caches so that neither L2 nor the 256 MB Infinity Cache holds
any KV (a read, not a rewrite, so that no dirty lines are left to be written
back during the step).  One pair of HIP events on
the stream the kernels run on brackets the K (flush + step) pairs, and others
the same K flushes alone, run right before and right after; a step's time is
the difference (from the flushes' mean) over K.  Events are not recorded
between the steps: each record leaves the GPU idle for ~5 us, which a
per-step pair would count as step time.  The pass-1 kernel alone (the
roofline's kernel) is timed the same way, K (flush + pass 1) pairs less K
flushes; for GQA the step itself is one launch of the step kernel, which is
then the roofline's kernel.  More steps, each between its own pair of events, give the per-step
median, p10 and p90 (each with one event's idle time in it); more diagnostic
steps run the pieces as separate calls with events between them.  The
algorithmic bytes of a step are the bf16 K and V rows (MLA: latent rows) of
every attended position, read once.

Every KV-streaming kernel dispatch this process issues is counted per kernel, in
order ("dispatch_windows"), so that a rocprofv3 trace of the same command can
be split by section: `python bench.py --trace-summary DIR --bench-json FILE`
prints, per section, the profiler's mean kernel time (and HBM counters, for a
--pmc run) over exactly that section's dispatches.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GPU-partition decode attention effective KV GB/s and % of HBM peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
EXTRA_STEPS = 20               # timed steps of each non-headline decode workload
EXTRA_WARMUP = 3
EVENT_STEPS = 20               # steps between their own event pairs
DIAG_STEPS = 20                # steps run as separate calls with events between the parts


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


def gqa_heads_per_workgroup(group: int) -> int:
    """Query heads one GQA pass-1 workgroup serves (its template argument)."""
    h = 1
    while h < min(group, 16):
        h *= 2
    return h


class Dispatches:
    """Dispatches of the KV-streaming kernels issued so far, per kernel, in
    order.  Every call of the decode workloads here covers at most 64
    sequences, i.e. exactly one dispatch: a GQA decode step (no load region)
    is one gqa_step_kernel launch (pass 1 with pass 2 in its last
    workgroups); pass 1 alone, and every MLA pass 1, one attend-kernel
    launch."""

    def __init__(self):
        self.n = {}

    @staticmethod
    def key(w, step: bool = False) -> str:
        from paper_2609_14507_amd import workloads as wl
        if w.kind == wl.MLA:
            return "mla_attend_kernel"
        return "gqa_%s_kernel<%d>" % ("step" if step else "attend", gqa_heads_per_workgroup(w.group))

    def at(self, w, step: bool = False) -> int:
        return self.n.get(self.key(w, step), 0)

    def add(self, w, k: int, step: bool = False):
        self.n[self.key(w, step)] = self.at(w, step) + k

    def part(self, w, first: int, step: bool = False):
        """[first, count, kernel] of the dispatches of w's kernel since `first`."""
        return [first, self.at(w, step) - first, self.key(w, step)]


def wsk_mod():
    from paper_2609_14507_amd import wsk
    return wsk


# HBM bytes per launch of each section's roofline kernel, from two rocprofv3
# --pmc runs of this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch,
# averaged over the section's dispatches), each scaled by what the same counter reads for
# the plain 256 MiB copy of --copy-calibration (FETCH_SIZE x 2.0,
# WRITE_SIZE x 1.0).  Keyed by section; valid only for the kernel source they
# were taken on (sha256), null otherwise.
TRAFFIC = {
    # the decode steps' roofline kernel: gqa_step_kernel (timed steps)
    "c5": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 622065.4 * 1024 * 2.0, "write_bytes": 1151.9 * 1024 * 1.0, "kv_bytes": 1270605824},
    "c2": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 369623.6 * 1024 * 2.0, "write_bytes": 1242.0 * 1024 * 1.0, "kv_bytes": 751976448},
    "c1": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 647.4 * 1024 * 2.0, "write_bytes": 30.5 * 1024 * 1.0, "kv_bytes": 1059328},
    # the sweep's and the MLA step's roofline kernel: pass 1 (launches alone)
    "c3 r=0.00": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 1048909.0 * 1024 * 2.0, "write_bytes": 390.0 * 1024 * 1.0, "kv_bytes": 2147483648},
    "c3 r=0.25": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 786701.0 * 1024 * 2.0, "write_bytes": 390.0 * 1024 * 1.0, "kv_bytes": 1610612736},
    "c3 r=0.50": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 524493.0 * 1024 * 2.0, "write_bytes": 390.0 * 1024 * 1.0, "kv_bytes": 1073741824},
    "c3 r=0.75": {"source": "paper_2609_14507_amd/csrc/attend_gqa.hip", "sha256": "dd13240b9482a9c2d0850924fc7ec9e9ae79171c2f848167129493327e6cfac1",
           "fetch_bytes": 262285.0 * 1024 * 2.0, "write_bytes": 390.0 * 1024 * 1.0, "kv_bytes": 536870912},
    "c4": {"source": "paper_2609_14507_amd/csrc/attend_mla.hip", "sha256": "fc7de28eef1c19d2054c21535bb9ce8b390632da3c964280ae047638d62b3edb",
           "fetch_bytes": 177748.1 * 1024 * 2.0, "write_bytes": 8208.0 * 1024 * 1.0, "kv_bytes": 362575872},
}


def roofline(section, kernel, achieved_gbs, kv_bytes, what="pass 1"):
    """Roofline entry of the kernel that streams the KV."""
    traffic = None
    t = TRAFFIC.get(section)
    if t is not None:
        with open(os.path.join(ROOT, t["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() == t["sha256"]:
                traffic = t["fetch_bytes"] + t["write_bytes"]
    out = {
        "bound": "hbm",
        "kernel": "%s (%s)" % (kernel, what),
        "achieved": round(achieved_gbs, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
        "traffic": None if traffic is None else int(traffic),
        "kv_bytes_per_launch": int(kv_bytes),
    }
    if traffic is not None:
        out["traffic_per_kv_byte"] = round(traffic / t["kv_bytes"], 4)
    return out


def evict(buf):
    """Read a 512 MiB buffer through the caches (its maximum, as int32), so
    that neither L2 nor the 256 MB Infinity Cache holds any KV when the next
    launch starts.  A read leaves the caches clean: a buffer rewrite would
    also leave up to 256 MB of dirty lines whose write-back lands in the next
    timed launch, which is the flush's cost, not the step's."""
    import torch
    return buf.view(torch.int32).amax()


class Timer:
    """Stream-ordered timing with one event pair around a whole bracket."""

    def __init__(self, flush, stream, no_flush):
        self.flush, self.stream, self.no_flush = flush, stream, no_flush

    def flush_once(self):
        if not self.no_flush:
            evict(self.flush)

    def bracket(self, fn):
        """ms of fn() on the stream, one event pair around it."""
        import torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        for _ in range(3):   # a GPU backlog ahead of the bracket: the host then runs ahead of
            evict(self.flush)    # the timed launches, and a host stall cannot idle the GPU inside it
        e0.record(self.stream)
        fn()
        e1.record(self.stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def flushes_ms(self, K):
        def run():
            for _ in range(K):
                self.flush_once()
        return self.bracket(run)


def decode_section(w, K, W, timer, disp, dev, tag, with_cpu_engine=False, keep=False):
    """K timed decode steps of workload w (after W warmup steps that append the
    last W rows of the drawn context), then pass 1 alone K times, EVENT_STEPS
    event-paired steps and DIAG_STEPS diagnostic steps."""
    import torch
    from paper_2609_14507_amd import workloads as wl
    from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
    wsk = wsk_mod()
    mla = w.kind == wl.MLA
    log("%s: drawing %s" % (tag, w.name))
    pf = wl.make_prefill(w)
    splits = pf.splits
    B, H = len(pf.lengths), w.n_q_heads
    assert all(L - W >= s for L, s in zip(pf.lengths, splits)), "warmup rows must lie on the GPU side"
    F = 5 if with_cpu_engine else 0
    n_steps = K + EVENT_STEPS + DIAG_STEPS + F
    steps_in = [wl.draw_step(w, pf.gen) for _ in range(W + n_steps)]
    for i in range(W):   # warmup steps append the context's last W rows
        steps_in[i].k_new = np.stack([pf.k[b][pf.lengths[b] - W + i] for b in range(B)])
        if not mla:
            steps_in[i].v_new = np.stack([pf.v[b][pf.lengths[b] - W + i] for b in range(B)])
    short = wl.Prefill([L - W for L in pf.lengths], splits, [k[:L - W] for k, L in zip(pf.k, pf.lengths)],
                       None if mla else [v[:L - W] for v, L in zip(pf.v, pf.lengths)], pf.gen)
    log("%s: routing the prefill into the cache" % tag)
    sess = DecodeSession(w, short, 0, extra_tokens=W + n_steps)
    D = sess.out_width                      # attend output width (MLA: the latent)
    qs = [to_device_bf16(s.q, dev) for s in steps_in]
    kn = [to_device_bf16(s.k_new, dev) for s in steps_in]
    vn = [None if mla else to_device_bf16(s.v_new, dev) for s in steps_in]
    if mla:
        w_uk, w_uv = wl.draw_mla_weights(w, pf.gen)
        w_uk_d, w_uv_d = to_device_bf16(w_uk, dev), to_device_bf16(w_uv, dev)
        qn = [to_device_bf16(s.q_nope, dev) for s in steps_in]
        o_out = torch.empty(B, H, w.head_dim, device=dev)
    o_c, l_c = wl.draw_cpu_partial(pf.gen, B * H, D)
    o_cpu = torch.from_numpy(o_c).to(dev).view(B, H, D)
    l_cpu = torch.from_numpy(l_c).to(dev).view(B, H)
    o_m = torch.empty(B, H, D, device=dev)
    l_m = torch.empty(B, H, device=dev)
    sess.workspace(sess.ids, [min(s, L) for s, L in zip(splits, sess.lengths)], list(sess.lengths))
    stream = timer.stream

    def step(i, ev=None, parts=None):
        """One decode step.  ev = (start, end) events around the step: the timed
        steps run it as wsk_decode_step (GQA: one launch, pass 1 over the
        positions written so far with pass 2 -- the appended row scored,
        merged and stored, the CPU partial merged -- in its last workgroups;
        MLA: wsk_decode_step_mla, pass 1 then a pass 2 that also expands the
        merged latent output by W_UV).  parts = 5 events around its
        pieces (diagnostic steps only, every event record costs GPU time of its
        own): those run the same work as separate calls -- append, pass 1 over
        [s, L + 1), pass 2 -- so that pass 1 is timed on its own."""
        timer.flush_once()
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
        disp.add(w, 1, step=fused and not parts)

    def kv_bytes():   # algorithmic bytes of the next step: [s_b, L_b + 1) of every sequence
        return sum((sess.lengths[b] + 1 - min(splits[b], sess.lengths[b])) * w.token_bytes for b in range(B))

    # a GQA step is one launch of the step kernel, the roofline's kernel;
    # an MLA step's KV-streaming kernel is its pass 1
    fused = not mla
    win = {"kernel": disp.key(w, fused)}
    log("%s: %d warmup + %d timed steps" % (tag, W, K))
    d0 = disp.at(w, fused)
    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    win["warmup"] = disp.part(w, d0, fused)
    assert list(sess.lengths) == list(pf.lengths)
    contexts = list(sess.lengths)
    nbytes = []

    def timed_steps():
        for k in range(K):
            nbytes.append(kv_bytes())
            step(W + k)
    t_flush_a = timer.flushes_ms(K)
    t0 = time.perf_counter()
    d0 = disp.at(w, fused)
    t_steps = timer.bracket(timed_steps)
    win["timed_steps"] = disp.part(w, d0, fused)
    wall = time.perf_counter() - t0
    t_flush = 0.5 * (t_flush_a + timer.flushes_ms(K))   # flushes timed before and after: drift cancels
    step_ms = (t_steps - t_flush) / K

    # the pass-1 kernel alone, K launches over the current GPU ranges
    p1_bytes = float(sum((sess.lengths[b] - min(splits[b], sess.lengths[b])) * w.token_bytes for b in range(B)))

    def pass1s():
        for k in range(K):
            timer.flush_once()
            sess.attend_pass1(qs[W + k])
            disp.add(w, 1)
    d0 = disp.at(w)
    t_p1 = timer.bracket(pass1s)
    win["pass1_alone"] = disp.part(w, d0)
    t_flush2 = 0.5 * (t_flush + timer.flushes_ms(K))
    p1_kernel_ms = (t_p1 - t_flush2) / K

    # the per-step distribution: steps each between their own pair of events
    # (each pair counts one event's idle time, ~5.5 us, as step time)
    ev_step = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(EVENT_STEPS)]
    d0 = disp.at(w, fused)
    for k in range(EVENT_STEPS):
        step(W + K + k, ev=ev_step[k])
    torch.cuda.synchronize()
    win["event_pairs"] = disp.part(w, d0, fused)
    ev_us = np.array([e[0].elapsed_time(e[1]) for e in ev_step]) * 1e3

    ev_part = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(DIAG_STEPS)]
    d_bytes = []
    d0 = disp.at(w)
    for k in range(DIAG_STEPS):
        d_bytes.append(kv_bytes())
        step(W + K + EVENT_STEPS + k, parts=ev_part[k])
    torch.cuda.synchronize()
    win["diagnostic"] = disp.part(w, d0)
    el = lambda a, b: np.array([e[a].elapsed_time(e[b]) for e in ev_part])
    app_ms, p1_ms, p2_ms = el(0, 1), el(1, 2), el(2, 3)
    exp_ms = el(3, 4) if mla else np.zeros(DIAG_STEPS)
    nbytes = np.array(nbytes, dtype=np.float64)
    d_bytes = np.array(d_bytes, dtype=np.float64)
    value = float(nbytes.mean() / (step_ms * 1e-3) / 1e9)
    att_gbs = float(d_bytes.sum() / ((p1_ms + p2_ms).sum() * 1e-3) / 1e9)
    p1_gbs = float(p1_bytes / (p1_kernel_ms * 1e-3) / 1e9)
    log("%s: step %.1f us (%.1f GB/s); pass 1 alone %.1f us, %.0f GB/s; diagnostic parts: absorb+append %.1f, "
        "pass 1 %.1f, pass 2 %.1f, expand %.1f us"
        % (tag, step_ms * 1e3, value, p1_kernel_ms * 1e3, p1_gbs, app_ms.mean() * 1e3, p1_ms.mean() * 1e3,
           p2_ms.mean() * 1e3, exp_ms.mean() * 1e3))
    out = {
        "workload": w.name,
        "config": {
            "batch": B, "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
            **({"latent_dim": w.latent_dim, "rope_dim": w.rope_dim, "nope_dim": w.nope_dim} if mla else {}),
            "context": contexts if w.ragged_hi else w.context,
            "cpu_split": list(splits) if w.ragged_hi else splits[0],
            "cpu_share": [w.share_lo, w.share_hi] if w.ragged_hi else w.cpu_share,
            "gpu_tokens_per_step": int(nbytes.mean() / w.token_bytes),
            "kv_bytes_per_step": int(nbytes.mean()),
            "step": ("absorb + wsk_decode_step_mla (attend pass 1 over [s, L), then one pass 2: the appended row "
                     "scored, merged and stored, chunk combine, LSE merge with the CPU partial, expansion by W_UV)"
                     if mla else "wsk_decode_step, one launch: attend pass 1 over [s, L); the last workgroup of "
                     "each (sequence, KV head, head group) scores, merges and stores the appended row, combines "
                     "the chunks and merges the CPU partial by LSE"),
            "cache_flush_between_steps": not timer.no_flush,
        },
        "steps": K, "warmup": W,
        "step_us": round(step_ms * 1e3, 2),
        "step_gbs": round(value, 1),
        "step_frac_of_peak": round(value / HBM_PEAK_GBS, 4),
        "breakdown_us": {
            "step": round(step_ms * 1e3, 2),
            "flush_plus_step": round(t_steps / K * 1e3, 2),
            "flush": round(t_flush / K * 1e3, 2),
            "pass1_kernel": round(p1_kernel_ms * 1e3, 2),
            "pass1_kv_bytes": int(p1_bytes),
            "step_event_pairs": {"median": round(float(np.median(ev_us)), 2),
                                 "p10": round(float(np.percentile(ev_us, 10)), 2),
                                 "p90": round(float(np.percentile(ev_us, 90)), 2),
                                 "what": "steps each between their own pair of events: the per-step spread; each "
                                         "includes one event record's idle time (~5.5 us)"},
            "wall_per_step_incl_flush": round(wall / K * 1e6, 1),
            "diagnostic_steps": "steps with events between the parts (each record adds ~5 us of GPU idle time to "
                                "the part it closes)",
            ("absorb_append" if mla else "append"): round(float(app_ms.mean() * 1e3), 2),
            "attend_pass1": round(float(p1_ms.mean() * 1e3), 2),
            "attend_pass2_combine_merge": round(float(p2_ms.mean() * 1e3), 2),
            **({"expand": round(float(exp_ms.mean() * 1e3), 2)} if mla else {}),
            "attend_gbs": round(att_gbs, 1),
        },
        "roofline": (roofline(tag, disp.key(w), p1_gbs, p1_bytes) if mla else
                     roofline(tag, disp.key(w, True), value, float(nbytes.mean()), "the whole step")),
        "dispatch_window": win,
        "_ms_per_step": float(step_ms),
    }
    state = None
    if with_cpu_engine or keep:
        state = dict(pf=pf, sess=sess if with_cpu_engine else None, steps_in=steps_in,
                     i0=W + K + EVENT_STEPS + DIAG_STEPS, F=F, splits=splits, qs=qs, kn=kn, vn=vn, o_m=o_m,
                     l_m=l_m, p1_kernel_ms=p1_kernel_ms, p1_bytes=p1_bytes, step_ms=step_ms, K=K, W=W)
    if not with_cpu_engine:
        sess.close()
    return out, state


def sweep_section(w, K, W, timer, disp, dev, tag="c3"):
    """The CPU share swept over w.sweep on ONE cache written once with s = 0:
    between sweep points only the attend range [s', L) changes (no data is
    written or moved).  A point's step is pass 1 over [s', L) plus pass 2
    merging the CPU partial of [0, s') (a synthetic stand-in here), timed as
    K (flush + step) pairs less K flushes; pass 1 alone the same way."""
    import torch
    from paper_2609_14507_amd import workloads as wl
    from paper_2609_14507_amd.runner import DecodeSession, to_device_bf16
    log("%s: drawing %s" % (tag, w.name))
    pf = wl.make_prefill(w)
    assert all(s == 0 for s in pf.splits), "the sweep cache is written with s = 0"
    B, H, L = len(pf.lengths), w.n_q_heads, w.context
    st = wl.draw_step(w, pf.gen)
    log("%s: routing the prefill into the cache (s = 0, once)" % tag)
    sess = DecodeSession(w, pf, 0, extra_tokens=0)
    q = to_device_bf16(st.q, dev)
    o_c, l_c = wl.draw_cpu_partial(pf.gen, B * H, w.head_dim)
    o_x = torch.from_numpy(o_c).to(dev).view(B, H, w.head_dim)
    l_x = torch.from_numpy(l_c).to(dev).view(B, H)
    o = torch.empty(B, H, w.head_dim, device=dev)
    lse = torch.empty(B, H, device=dev)
    points = []
    win = {"kernel": disp.key(w)}
    for share in w.sweep:
        s = wl.split_point(share, L)
        start, end = [s] * B, [L] * B
        sess.workspace(sess.ids, start, end)

        def one_step():
            timer.flush_once()
            sess.attend_pass1(q, start, end)
            sess.attend_pass2(start, end, o=o, lse=lse, o_x=o_x, lse_x=l_x)
            disp.add(w, 1)
        d0 = disp.at(w)
        for _ in range(W):
            one_step()
        torch.cuda.synchronize()
        fa = timer.flushes_ms(K)
        d1 = disp.at(w)
        t_steps = timer.bracket(lambda: [one_step() for _ in range(K)])
        d2 = disp.at(w)
        t_flush = 0.5 * (fa + timer.flushes_ms(K))

        def p1():
            for _ in range(K):
                timer.flush_once()
                sess.attend_pass1(q, start, end)
                disp.add(w, 1)
        t_p1 = timer.bracket(p1)
        t_flush2 = 0.5 * (t_flush + timer.flushes_ms(K))
        step_ms = (t_steps - t_flush) / K
        p1_ms = (t_p1 - t_flush2) / K
        kvb = float(B * (L - s) * w.token_bytes)
        key = "%s r=%.2f" % (tag, share)
        points.append({
            "cpu_share": share, "split": s, "kv_bytes_per_step": int(kvb),
            "step_us": round(step_ms * 1e3, 2), "step_gbs": round(kvb / (step_ms * 1e-3) / 1e9, 1),
            "step_frac_of_peak": round(kvb / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "pass1_us": round(p1_ms * 1e3, 2),
            "roofline": roofline(key, disp.key(w), kvb / (p1_ms * 1e-3) / 1e9, kvb),
        })
        win["r=%.2f" % share] = {"warmup": [d0, d1 - d0], "timed_steps": [d1, d2 - d1], "pass1_alone": [d2, K]}
        log("%s: r = %.2f (s' = %d): step %.1f us (%.0f GB/s), pass 1 %.1f us (%.0f GB/s)"
            % (tag, share, s, step_ms * 1e3, kvb / (step_ms * 1e-3) / 1e9, p1_ms * 1e3, kvb / (p1_ms * 1e-3) / 1e9))
    sess.close()
    return {
        "workload": w.name,
        "config": {"batch": B, "q_heads": H, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "context": L,
                   "written_with_split": 0, "sweep": list(w.sweep),
                   "step": "wsk_attend_pass1 over [s', L) + wsk_attend_pass2 (chunk combine and LSE merge of the "
                           "CPU partial of [0, s')); one cache, written once, no data moved between points",
                   "cache_flush_between_steps": not timer.no_flush},
        "steps": K, "warmup": W,
        "sweep": points,
        "dispatch_window": win,
    }


def cpu_baseline(w5, pf5, steps5, W, K, w1, budget_s: float):
    """The fp64 oracle, as it stands, on the host's cores: the headline's GPU
    ranges [s_b, L_b + k + 1) of all sequences at timed decode steps 0, 31 and
    63 first (and their CPU ranges [0, s_b), which feed the merge), then
    further steps in order until the time budget is spent; also the tiny
    single-sequence case on one thread and on all of them."""
    import oracle
    B = len(pf5.lengths)
    timed = steps5[W:W + K]
    ks, vs = [], []
    for b in range(B):   # cache rows plus every timed step's appended row, in place
        L = pf5.lengths[b]
        k = np.empty((L + K,) + pf5.k[b].shape[1:], dtype=pf5.k[b].dtype)
        v = np.empty_like(k)
        k[:L], v[:L] = pf5.k[b], pf5.v[b]
        for j, st in enumerate(timed):
            k[L + j], v[L + j] = st.k_new[b], st.v_new[b]
        ks.append(k)
        vs.append(v)
    threads = oracle.max_threads()
    order = [j for j in (0, 31, 63) if j < K] + [j for j in range(K) if j not in (0, 31, 63)]
    t_total, nbytes, done, first = 0.0, 0, 0, []
    for j in order:
        st = timed[j]
        tg, bg, tc, bc = 0.0, 0, 0.0, 0
        for b in range(B):
            L = pf5.lengths[b] + j + 1
            s = pf5.splits[b]
            t0 = time.perf_counter()
            oracle.attend(st.q[b], ks[b][:L], vs[b][:L], s, L, w5.softmax_scale, w5.group)
            t1 = time.perf_counter()
            tg += t1 - t0
            bg += (L - s) * w5.token_bytes
            if j in (0, 31, 63):
                oracle.attend(st.q[b], ks[b][:L], vs[b][:L], 0, s, w5.softmax_scale, w5.group)
                tc += time.perf_counter() - t1
                bc += s * w5.token_bytes
        t_total += tg
        nbytes += bg
        done += 1
        if j in (0, 31, 63):
            first.append({"step": j, "gpu_range_s": round(tg, 3), "gpu_range_gbs": round(bg / tg / 1e9, 3),
                          "cpu_range_s": round(tc, 3), "cpu_range_gbs": round(bc / tc / 1e9, 3)})
        elif t_total >= budget_s:
            break
    # the tiny case: one sequence, [s, L + 1) after its append, single thread and all threads
    from paper_2609_14507_amd import workloads as wl
    pf1 = wl.make_prefill(w1)
    st1 = wl.draw_step(w1, pf1.gen)
    k1 = np.concatenate([pf1.k[0], st1.k_new[0][None]])
    v1 = np.concatenate([pf1.v[0], st1.v_new[0][None]])
    s1, L1 = pf1.splits[0], k1.shape[0]
    c1 = {}
    for label, n in (("threads_1", 1), ("threads_all", threads)):
        oracle.set_threads(n)
        reps, t = 0, 0.0
        while t < 1.0:
            t0 = time.perf_counter()
            oracle.attend(st1.q[0], k1, v1, s1, L1, w1.softmax_scale, w1.group)
            t += time.perf_counter() - t0
            reps += 1
        c1[label] = {"threads": n, "ms": round(t / reps * 1e3, 3),
                     "gbs": round((L1 - s1) * w1.token_bytes * reps / t / 1e9, 3)}
    oracle.set_threads(threads)
    return {
        "value": nbytes / t_total / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "fp64 oracle over the GPU ranges [s_b, L_b + k + 1) of all %d sequences of the headline "
                  "workload at timed decode steps 0, 31, 63, then further steps in order until %.0f s were spent: "
                  "%d steps, %.2f GB of KV in %.1f s; CPU: %s"
                  % (B, budget_s, done, nbytes / 1e9, t_total, cpu_model()),
        "steps_0_31_63": first,
        "tiny_c1": dict(c1, what="one sequence, L 2048 + 1 appended, GPU range [1024, 2049), fp64 oracle"),
    }


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
        evict(flush)
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
    sess = DecodeSession(w, pf, 0, extra_tokens=5 * D + 2, load_ends=load_ends, evict_tokens=D, pingpong_blocks=512,
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
            evict(flush)
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
    # (three of each; D more rows are appended to every sequence before each)
    if w.kind == wl.MLA:
        kn, vn = torch.zeros(B, w.row_elems, dtype=torch.bfloat16, device=dev), None
    else:
        kn = torch.zeros(B, w.n_kv_heads, w.head_dim, dtype=torch.bfloat16, device=dev)
        vn = torch.zeros_like(kn)
    fl_t, fl_b = {wsk.PART_LOAD: [], wsk.PART_CPU: []}, {wsk.PART_LOAD: [], wsk.PART_CPU: []}
    for k, dest in enumerate([wsk.PART_LOAD, wsk.PART_CPU] * 3):
        if k:
            for _ in range(D):
                sess.append(kn, vn)
        d0 = wsk.wsk_load_stats(sess.h).d2h_bytes
        fl_t[dest].append(timed(lambda: sess.flush([dest] * B), 1))
        fl_b[dest].append(wsk.wsk_load_stats(sess.h).d2h_bytes - d0)
    t_fl, d_fl = float(np.median(fl_t[wsk.PART_LOAD])), int(np.median(fl_b[wsk.PART_LOAD]))
    t_fc, d_fc = float(np.median(fl_t[wsk.PART_CPU])), int(np.median(fl_b[wsk.PART_CPU]))
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

    def d2h_gbs(nbytes, reps=5):   # device -> pinned host: the eviction direction
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        return nbytes / timed(lambda: dst.copy_(src, non_blocking=True), reps) / 1e9
    for label, n in (("8MiB", 8 << 20), ("256MiB", 256 << 20)):
        micro["d2h_pinned_" + label] = round(d2h_gbs(n), 2)
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
                  "what": "wsk_flush of one D = %d batch of every sequence (median of 3 each, alternating); to "
                          "the CPU includes the token-major rewrite (on the GPU) and the host's copy into the "
                          "slots" % D},
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
            evict(flush)
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




def _read_rows(pattern):
    paths = sorted(glob.glob(pattern, recursive=True))
    rows = []
    for p in paths:
        with open(p, newline="") as f:
            rows.extend(csv.DictReader(f))
    return rows


def trace_summary(trace_dir, bench_json):
    """Markdown summary of a rocprofv3 run of this script: for every section
    of the JSON line the same run printed, the profiler's mean duration (kernel
    trace) or counter value (--pmc, KiB per dispatch) over exactly that
    section's pass-1 dispatches, matched by kernel name in dispatch order."""
    with open(bench_json) as f:
        line = [ln for ln in f if ln.startswith("{")][-1]
    out = json.loads(line)
    trace = _read_rows(os.path.join(trace_dir, "**", "*kernel_trace.csv"))
    counters = _read_rows(os.path.join(trace_dir, "**", "*counter_collection.csv"))

    def per_kernel(rows, key):
        # the GQA kernels come as a per-sequence-chunk and a flat-split
        # instantiation ("<8, false>", "<8, true>"): one key, dispatch order
        sel = [r for r in rows if (key + "(") in re.sub(r", (true|false)>", ">", r["Kernel_Name"])]
        return sorted(sel, key=lambda r: int(r["Dispatch_Id"]))

    # per section: its windows, and per part the algorithmic KV bytes of one
    # dispatch and bench.py's own time of it (event-timed parts only)
    sections = []
    for name, sec in [("headline", out)] + sorted(out.get("configs", {}).items()):
        win = sec.get("dispatch_window")
        if not win:
            continue
        if "timed_steps" in win:
            bd = sec["breakdown_us"]
            kv_step = sec["config"]["kv_bytes_per_step"]
            kv_p1 = bd.get("pass1_kv_bytes", sec["roofline"]["kv_bytes_per_launch"])
            kv = {"timed_steps": kv_step, "event_pairs": kv_step, "diagnostic": kv_step, "pass1_alone": kv_p1}
            us = {"pass1_alone": bd["pass1_kernel"]}
            if "step" in win["kernel"]:
                us["timed_steps"] = bd["step"]
            sections.append((name, win["kernel"], win, kv, us))
        for label, sub in sorted(win.items()):
            if isinstance(sub, dict):
                pt = [p for p in sec["sweep"] if "r=%.2f" % p["cpu_share"] == label][0]
                kvp = pt["roofline"]["kv_bytes_per_launch"]
                sections.append(("%s %s" % (name, label), win["kernel"], sub, {"timed_steps": kvp, "pass1_alone": kvp},
                                 {"pass1_alone": pt["pass1_us"]}))
    lines = []
    if trace:
        lines += ["| section | kernel | part | dispatches | mean us | min us | max us | KV MB per launch | "
                  "TB/s at mean | % of 8 TB/s | bench.py us |", "|---|---|---|---|---|---|---|---|---|---|---|"]
        cache = {}
        for name, kernel, win, kv, bench_us in sections:
            for part in ("timed_steps", "pass1_alone", "event_pairs", "diagnostic"):
                if part not in win:
                    continue
                a, n = win[part][:2]
                key = win[part][2] if len(win[part]) > 2 else kernel
                kvb = kv[part]
                d = cache.setdefault(key, per_kernel(trace, key))
                us = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in d[a:a + n]]
                if len(us) != n:
                    lines.append("| %s | %s | %s | %d of %d found | | | | | | | |" % (name, key, part, len(us), n))
                    continue
                m = float(np.mean(us))
                lines.append("| %s | %s | %s | %d | %.2f | %.2f | %.2f | %.1f | %.2f | %.1f | %s |"
                             % (name, key, part, n, m, min(us), max(us), kvb / 1e6, kvb / (m * 1e-6) / 1e12,
                                100 * kvb / (m * 1e-6) / 8e12, bench_us.get(part, "")))
    if counters:
        names = sorted({r["Counter_Name"] for r in counters})
        copies = [r for r in counters if "__amd_rocclr_copyBuffer" in r["Kernel_Name"]]
        lines += ["", "Counters (KiB per dispatch); copy calibration (%d dispatches of __amd_rocclr_copyBuffer, "
                  "the last three are the 256 MiB copies): %s" % (len(copies), ", ".join(
                      "%s %s" % (c, [round(float(r["Counter_Value"]), 1) for r in copies if r["Counter_Name"] == c][-3:])
                      for c in names)), "",
                  "| section | kernel | part | dispatches | " + " | ".join(names) + " | KV MB per launch |",
                  "|---|---|---|---|" + "---|" * len(names) + "---|"]
        for name, kernel, win, kv, _ in sections:
            for part in ("timed_steps", "pass1_alone"):
                if part not in win:
                    continue
                a, n = win[part][:2]
                key = win[part][2] if len(win[part]) > 2 else kernel
                kvb = kv[part]
                vals = []
                for c in names:
                    d = per_kernel([r for r in counters if r["Counter_Name"] == c], key)[a:a + n]
                    vals.append("%.1f" % np.mean([float(r["Counter_Value"]) for r in d]) if len(d) == n else "-")
                lines.append("| %s | %s | %s | %d | %s | %.1f |" % (name, key, part, n, " | ".join(vals), kvb / 1e6))
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64, help="timed decode steps of the headline workload")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c5", help="headline workload: c5 (default), c2, c4 or c1")
    ap.add_argument("--headline-only", action="store_true", help="skip the other configurations")
    ap.add_argument("--no-flush", action="store_true", help="skip the Infinity Cache flush between steps")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cpu-engine", action="store_true",
                    help="skip the native CPU engine and the full CPU + GPU steps")
    ap.add_argument("--no-load-region", action="store_true",
                    help="skip the streamed load-region step, eviction and transfer measurements")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="at the end, run a plain 256 MiB device copy three times (the reference dispatch that "
                         "scales HBM byte counters)")
    ap.add_argument("--trace-summary", default=None, help="summarise a rocprofv3 output directory of this script "
                    "(needs --bench-json) and exit; uses no GPU")
    ap.add_argument("--bench-json", default=None, help="file holding the JSON line of the profiled run")
    args = ap.parse_args()

    if args.trace_summary:
        trace_summary(args.trace_summary, args.bench_json)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_14507_amd import workloads as wl

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    timer = Timer(flush, torch.cuda.current_stream(), args.no_flush)
    disp = Dispatches()
    K, W = args.steps, args.warmup
    w = wl.CONFIGS[args.config]
    if w.sweep:
        raise SystemExit("the swept configuration is reported under 'configs'; pick c5, c2, c4 or c1")

    # headline: K timed decode steps
    cpu_c2 = not args.no_cpu_engine
    head, head_state = decode_section(w, K, W, timer, disp, dev, args.config,
                                      with_cpu_engine=(args.config == "c2" and cpu_c2), keep=True)
    configs, c2_state = {}, (head_state if args.config == "c2" else None)
    if not args.headline_only:
        configs["c3"] = sweep_section(wl.C3, EXTRA_STEPS, EXTRA_WARMUP, timer, disp, dev)
        for tag in ("c4", "c2", "c1"):
            if tag == args.config:
                continue
            res, st = decode_section(wl.CONFIGS[tag], EXTRA_STEPS, EXTRA_WARMUP, timer, disp, dev, tag,
                                     with_cpu_engine=(tag == "c2" and cpu_c2), keep=(tag == "c2"))
            configs[tag] = res
            if tag == "c2":
                c2_state = st
    # the native CPU engine and the full CPU + GPU step (the Qwen3 shape at
    # batch 16), on that workload's decode session
    cpu_engine = full_step = policy = None
    wc = wl.C2
    if c2_state is not None and c2_state["sess"] is not None:
        st = c2_state
        d0 = disp.at(wc)
        cpu_engine, full_step, policy = cpu_gpu_steps(
            wc, st["sess"], wsk_mod(), st["steps_in"], st["i0"], st["F"], st["splits"], st["qs"], st["kn"],
            st["vn"], st["o_m"], st["l_m"], flush, dev, None, None,
            gpu_ns_per_token=float(st["p1_kernel_ms"] * 1e6 / (st["p1_bytes"] / wc.token_bytes)),
            gpu_fixed_us=float((st["step_ms"] - st["p1_kernel_ms"]) * 1e3))
        disp.add(wc, st["F"])
        (configs.get("c2") or head)["dispatch_window"]["cpu_gpu_steps"] = disp.part(wc, d0)
        st["sess"].close()
        st["sess"] = None
    # after every counted dispatch: the pinned load region, eviction, the
    # offloaded step (their streamed pass-1 launches are not counted)
    load_region = offload = None
    if not args.no_load_region and c2_state is not None:
        load_region = load_region_section(wc, c2_state["pf"], c2_state["steps_in"], dev, flush)
        if policy is not None:
            offload = offload_section(wc, c2_state["pf"], c2_state["steps_in"], dev, flush,
                                      policy["A_ns_per_token"] * 1e-9, policy["c_cpu_us"] * 1e-6,
                                      wc.token_bytes / (load_region["achieved"] * 1e9))
    c2_state = None
    # plain streaming read of 2 GiB with the attention kernels' load pattern:
    # the practical HBM read ceiling the pass-1 rate is compared with
    from paper_2609_14507_amd import wsk as _wsk
    probe = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    probe.fill_(3)
    fold = torch.zeros(1, dtype=torch.int32, device=dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    stream = timer.stream

    def read_gbs(workgroups):
        ms = []
        for it in range(6):
            evict(flush)
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
            evict(flush)
            dst.copy_(src)
        torch.cuda.synchronize()
        log("bench: copy calibration: 3 x %d bytes read + written" % src.numel())

    step_ms = head.pop("_ms_per_step")
    for c in configs.values():
        c.pop("_ms_per_step", None)
    out = {
        "metric": METRIC,
        "value": head["step_gbs"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": dict(workload=head["workload"], decode_steps=K, **head["config"]),
        "frac_of_peak": head["step_frac_of_peak"],
        "breakdown_us": head["breakdown_us"],
        "roofline": head["roofline"],
        "workload": head["workload"],
        "dispatch_window": head["dispatch_window"],
        "configs": configs,
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
    if head_state is not None:
        if not args.no_cpu_baseline:
            if w is wl.C5:
                log("bench: timing the oracle on the host (%.0f s budget)" % args.cpu_budget)
                out["cpu_baseline"] = cpu_baseline(w, head_state["pf"], head_state["steps_in"], W, K, wl.C1,
                                                   args.cpu_budget)
            else:
                log("bench: cpu_baseline is taken on the ragged 1M-token workload only")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
