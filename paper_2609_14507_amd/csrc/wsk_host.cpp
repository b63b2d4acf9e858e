// Host side of the partitioned KV cache: spec validation, block pools, the
// deterministic slot allocator (write-time routing), views, and the launch
// plumbing of the decode-path kernels.  Implements include/wsk.h.

#include <hip/hip_runtime.h>
#include <sys/mman.h>

#include <algorithm>
#include <queue>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "cache.h"

using namespace wsk;

namespace {
thread_local std::string g_err;
}  // namespace

int wsk::fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int wsk::hip_fail(hipError_t e, const char *what) {
    return fail(WSK_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// Error reporting for the policy functions (policy.cpp).
int wsk::policy_fail(int code, const char *msg) { return fail(code, "%s", msg); }

namespace {

int validate_spec(const wsk_partition_spec *s) {
    if (!s) return fail(WSK_EINVAL, "spec is NULL");
    if (s->reserved != 0) return fail(WSK_EINVAL, "spec.reserved must be 0");
    if (s->kind != WSK_KIND_GQA && s->kind != WSK_KIND_MLA) return fail(WSK_EINVAL, "spec.kind %d", s->kind);
    if (s->n_q_heads <= 0 || s->n_kv_heads <= 0) return fail(WSK_EINVAL, "head counts must be positive");
    if (s->block_tokens != 64 && s->block_tokens != 128 && s->block_tokens != 256)
        return fail(WSK_EINVAL, "block_tokens must be 64, 128 or 256 (got %d)", s->block_tokens);
    if (s->max_seqs <= 0 || s->max_seq_len <= 0) return fail(WSK_EINVAL, "max_seqs and max_seq_len must be positive");
    if (s->device_pool_blocks < 0 || s->host_pool_blocks < 0 || s->device_pool_blocks > INT32_MAX ||
        s->host_pool_blocks > INT32_MAX)
        return fail(WSK_EINVAL, "pool sizes must be in [0, 2^31)");
    if (!(std::isfinite(s->softmax_scale) && s->softmax_scale > 0.f))
        return fail(WSK_EINVAL, "softmax_scale must be finite and positive");
    if ((int64_t)s->max_seqs * ((s->max_seq_len + s->block_tokens - 1) / s->block_tokens) > INT32_MAX)
        return fail(WSK_EINVAL, "block table too large");
    if (s->evict_tokens < 0 || s->evict_tokens % s->block_tokens)
        return fail(WSK_EINVAL, "evict_tokens must be a non-negative multiple of block_tokens");
    if (s->load_pool_blocks < 0 || s->load_pool_blocks > INT32_MAX)
        return fail(WSK_EINVAL, "load_pool_blocks must be in [0, 2^31)");
    if (s->load_pool_blocks > 0 && (s->load_arena_blocks <= 0 || s->pingpong_blocks <= 0))
        return fail(WSK_EINVAL, "a load region needs load_arena_blocks > 0 and pingpong_blocks > 0");
    if (s->load_pool_blocks == 0 && (s->load_arena_blocks != 0 || s->pingpong_blocks != 0))
        return fail(WSK_EINVAL, "load_arena_blocks and pingpong_blocks must be 0 without a load region");
    if (s->pingpong_blocks < 0 || s->load_arena_blocks < 0) return fail(WSK_EINVAL, "negative load-region size");
    if (s->kind == WSK_KIND_GQA) {
        if (s->n_q_heads % s->n_kv_heads) return fail(WSK_EINVAL, "n_q_heads must be a multiple of n_kv_heads");
        if (s->n_q_heads / s->n_kv_heads > WSK_MAX_GROUP) return fail(WSK_EINVAL, "group size above %d", WSK_MAX_GROUP);
        if (s->head_dim != kHeadDim) return fail(WSK_EINVAL, "GQA head_dim must be %d", kHeadDim);
        if (s->latent_dim != 0 || s->rope_dim != 0) return fail(WSK_EINVAL, "GQA latent_dim/rope_dim must be 0");
    } else {
        if (s->n_kv_heads != 1) return fail(WSK_EINVAL, "MLA n_kv_heads must be 1");
        if (s->latent_dim != kLatent || s->rope_dim != kRope)
            return fail(WSK_EINVAL, "MLA latent_dim/rope_dim must be %d/%d", kLatent, kRope);
        if (s->n_q_heads > 16) return fail(WSK_EINVAL, "MLA supports at most 16 heads");
    }
    return WSK_OK;
}

}  // namespace

int wsk::check_seq(const wsk_cache *c, int32_t seq) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    if (seq < 0 || seq >= c->spec.max_seqs) return fail(WSK_EINVAL, "sequence id %d out of range", seq);
    if (!c->is_open[seq]) return fail(WSK_ESTATE, "sequence %d is not open", seq);
    return WSK_OK;
}

void wsk::undo(wsk_cache *c, const std::vector<Pending> &pend) {
    for (const Pending &p : pend) c->free_slots[p.part].push(p.slot);
}

namespace {
const char *const kPartName[3] = {"CPU", "GPU", "load"};
}

// Routing decision for positions [pos0, pos0+n) of seq (Sec. 4.2): position
// p goes to the CPU pool if p < s, to the load region if s <= p < load_end,
// else to the GPU pool.  Every (pool, logical block) touched for the first
// time takes the lowest free slot of its pool, blocks in ascending order and,
// within a block, pools in the order CPU, GPU, load.
int wsk::plan(wsk_cache *c, int32_t seq, int32_t pos0, int32_t n, std::vector<Pending> &pend) {
    if (n <= 0) return WSK_OK;
    const int bk = c->spec.block_tokens;
    const int32_t s = c->split[seq], w0 = std::max(c->load_end[seq], s);
    const int32_t end = pos0 + n;
    for (int32_t blk = pos0 / bk; blk <= (end - 1) / bk; ++blk) {
        const int32_t lo = std::max(pos0, blk * bk), hi = std::min(end, (blk + 1) * bk);
        for (int part : {WSK_PART_CPU, WSK_PART_GPU, WSK_PART_LOAD}) {
            const bool touched = part == WSK_PART_CPU   ? lo < s
                                 : part == WSK_PART_GPU ? hi > w0
                                                        : std::max(lo, s) < std::min(hi, w0);
            if (!touched || tab(c, part, seq, blk) >= 0) continue;
            bool pending_already = false;
            for (const Pending &p : pend)
                if (p.part == part && p.seq == seq && p.blk == blk) pending_already = true;
            if (pending_already) continue;
            if (c->free_slots[part].empty()) {
                undo(c, pend);
                pend.clear();
                return fail(WSK_ENOMEM, "%s pool exhausted", kPartName[part]);
            }
            pend.push_back({part, seq, blk, c->free_slots[part].top()});
            c->free_slots[part].pop();
        }
    }
    return WSK_OK;
}

int wsk::home_of(const wsk_cache *c, int32_t seq, int32_t pos) {
    if (pos >= c->window[seq]) return WSK_PART_GPU;
    for (const Seg &g : c->segs[seq])
        if (pos >= g.a && pos < g.e) return g.part;
    return WSK_PART_CPU;   // not reached: the segments cover [0, window)
}

bool wsk::range_in(const wsk_cache *c, int32_t seq, int32_t a, int32_t e, int part) {
    const int32_t L = c->length[seq];
    if (a < 0 || a > e || e > L) return false;
    if (a == e) return true;
    const int32_t w = std::min(c->window[seq], L);
    if (part == WSK_PART_GPU) return a >= w;
    int32_t p = a;   // walk the segments in order, extending the covered prefix [a, p)
    for (const Seg &g : c->segs[seq])
        if (g.part == part && g.a <= p && g.e > p) p = std::min(g.e, w);
    return p >= e;
}

void wsk::commit(wsk_cache *c, const std::vector<Pending> &pend) {
    for (const Pending &p : pend) tab(c, p.part, p.seq, p.blk) = p.slot;
}

namespace {

// Validates ranges of the GPU pool (the D-window [window, L) of each
// sequence) and plans their chunking.
int make_plan(const wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
              AttendPlan &pl) {
    if (n < 0) return fail(WSK_EINVAL, "n < 0");
    if (n > 0 && (!ids || !start || !end)) return fail(WSK_EINVAL, "seq_ids/start/end must not be NULL");
    for (int32_t i = 0; i < n; ++i) {
        int rc = check_seq(c, ids[i]);
        if (rc) return rc;
        const int32_t L = c->length[ids[i]], w = std::min(c->window[ids[i]], L);
        if (!(w <= start[i] && start[i] <= end[i] && end[i] <= L))
            return fail(WSK_ERANGE, "range [%d, %d) of sequence %d outside its GPU partition [%d, %d)", start[i],
                        end[i], ids[i], w, L);
    }
    plan_chunks(c, n, start, end, pl);
    return WSK_OK;
}

}  // namespace

namespace {

// Per-sequence chunks of ranges [i0, i0 + m), min-max: every non-empty range
// starts with one chunk, and each further chunk of the budget goes to the
// range whose chunks are currently the largest (never below 4 tiles, one per
// wavefront, per chunk).  A launch lasts as long as its largest chunk, so on
// ragged batches this beats counts in proportion to the ranges' tiles.  Sets
// nchunks and tpc of those ranges; returns the largest chunk's tiles.
int64_t chunks_per_range(const int32_t *start, const int32_t *end, int32_t i0, int32_t m, int64_t budget,
                         bool min_one, AttendPlan &pl) {
    std::vector<int64_t> T(m);
    std::priority_queue<std::pair<int64_t, int32_t>> big;   // (tiles per chunk now, range)
    int64_t spent = 0;
    for (int32_t r = 0; r < m; ++r) {
        T[r] = n_tiles(start[i0 + r], end[i0 + r]);
        pl.nchunks[i0 + r] = 0;
        pl.tpc[i0 + r] = 1;
        if (T[r] == 0) continue;
        pl.nchunks[i0 + r] = 1;
        ++spent;
        big.push({T[r], r});
    }
    while (spent < budget && !big.empty()) {
        const int32_t r = big.top().second;
        big.pop();
        int32_t &nc = pl.nchunks[i0 + r];
        if (nc + 1 > (T[r] + 3) / 4) continue;
        ++nc;
        ++spent;
        big.push({(T[r] + nc - 1) / nc, r});
    }
    int64_t worst = 0;
    for (int32_t r = 0; r < m; ++r) {
        int32_t &nc = pl.nchunks[i0 + r];
        if (T[r] == 0) {
            nc = min_one ? 1 : 0;
            continue;
        }
        const int64_t tpc = (T[r] + nc - 1) / nc;
        pl.tpc[i0 + r] = (int32_t)tpc;
        nc = (int32_t)((T[r] + tpc - 1) / tpc);
        worst = std::max(worst, tpc);
    }
    return worst;
}

}  // namespace

// Chunking of valid ranges (positions on the tile grid of the table the
// kernels will read: the cache's, or a compacted one for block selections),
// per launch of up to kMaxLaunchSeqs ranges, each launch aiming at the whole
// GPU.
void wsk::plan_chunks(const wsk_cache *c, int32_t n, const int32_t *start, const int32_t *end, AttendPlan &pl,
                      bool min_one) {
    const wsk_partition_spec &sp = c->spec;
    const bool gqa = sp.kind == WSK_KIND_GQA;
    int units = 1;
    if (gqa) {
        const int G = sp.n_q_heads / sp.n_kv_heads;
        pl.heads_per_wg = gqa_heads_per_wg(G);
        pl.head_groups = G / pl.heads_per_wg;
        units = sp.n_kv_heads * pl.head_groups;
    }
    // workgroups a launch aims at (GQA: 3/4 per CU; MLA, whose workgroups
    // are twice as wide: 1 per CU); the budget per (KV head, head group)
    // unit follows from it
    const int64_t slots = gqa ? gqa_resident_slots(c->cu_count) : (int64_t)c->cu_count;
    const int64_t budget = std::max<int64_t>(1, slots / units);
    pl.tpc.assign(n, 1);
    pl.nchunks.assign(n, 0);
    pl.flat_first.assign(n, 0);
    pl.wfirst.assign(n, 0);
    pl.launch_tiles.clear();
    pl.launch_wgs.clear();
    for (int32_t i0 = 0; i0 < n; i0 += kMaxLaunchSeqs) {
        const int32_t m = std::min(kMaxLaunchSeqs, n - i0);
        const int64_t worst = chunks_per_range(start, end, i0, m, budget, min_one, pl);
        pl.launch_tiles.push_back(0);
        pl.launch_wgs.push_back(0);   // 0: per-range chunks
        if (!gqa) continue;
        // GQA, the flat split: the launch's tiles in range order, a gap of
        // kSegmentTiles before each non-empty range, cut into equal runs, one
        // per workgroup of each unit, whatever the ranges' lengths.  A run
        // that crosses into a range pays for the restart with the gap.  Taken
        // when its runs are shorter than the largest per-range chunk.
        int64_t total = 0, tiles = 0;
        for (int32_t r = 0; r < m; ++r) {
            const int64_t t = n_tiles(start[i0 + r], end[i0 + r]);
            if (t > 0) total += kSegmentTiles;
            pl.flat_first[i0 + r] = (int32_t)total;
            total += t;
            tiles += t;
        }
        if (tiles == 0) continue;
        const int64_t nw = std::max<int64_t>(1, std::min<int64_t>(budget, (tiles + 3) / 4));
        if ((total + nw - 1) / nw >= worst) continue;
        pl.launch_tiles.back() = (int32_t)total;
        pl.launch_wgs.back() = (int32_t)nw;
        // the run holding flat position x: the last w with w * total / nw <= x
        auto owner = [&](int64_t x) { return (int32_t)(((x + 1) * nw + total - 1) / total - 1); };
        for (int32_t r = 0; r < m; ++r) {
            const int32_t i = i0 + r;
            const int64_t f = pl.flat_first[i], t = n_tiles(start[i], end[i]);
            if (t > 0) {
                pl.wfirst[i] = owner(f);
                pl.nchunks[i] = owner(f + t - 1) - pl.wfirst[i] + 1;
            } else {   // an empty range: its one empty partial (min_one) comes from the run at f
                pl.wfirst[i] = f < total ? owner(f) : (int32_t)nw - 1;
                pl.nchunks[i] = min_one ? 1 : 0;
            }
        }
    }
    pl.partials = 0;
    for (int32_t i = 0; i < n; ++i) pl.partials += pl.nchunks[i];
    const int width = gqa ? kHeadDim : kLatent;
    pl.part_o_bytes = ((size_t)pl.partials * sp.n_q_heads * width * sizeof(float) + 255) / 256 * 256;
    pl.bytes = pl.part_o_bytes + ((size_t)pl.partials * sp.n_q_heads * sizeof(float) + 255) / 256 * 256;
}

extern "C" {

const char *wsk_last_error(void) { return g_err.c_str(); }

int wsk_init(const wsk_partition_spec *spec, int device, wsk_cache **out) {
    if (!out) return fail(WSK_EINVAL, "out is NULL");
    *out = nullptr;
    int rc = validate_spec(spec);
    if (rc) return rc;
    if (device < -1) return fail(WSK_EINVAL, "device %d", device);
    wsk_cache *c = new (std::nothrow) wsk_cache();
    if (!c) return fail(WSK_ENOMEM, "host allocation failed");
    c->spec = *spec;
    c->device = device;
    c->max_blocks = (spec->max_seq_len + spec->block_tokens - 1) / spec->block_tokens;
    if (spec->kind == WSK_KIND_GQA) {
        c->row_elems = spec->head_dim;
        c->rows_per_pos = 2 * spec->n_kv_heads;
    } else {
        c->row_elems = spec->latent_dim + spec->rope_dim;
        c->rows_per_pos = 1;
    }
    c->slot_elems = (int64_t)c->rows_per_pos * spec->block_tokens * c->row_elems;
    try {
        const size_t tab_n = (size_t)spec->max_seqs * c->max_blocks;
        c->htab[0].assign(tab_n, -1);
        c->htab[1].assign(tab_n, -1);
        if (spec->load_pool_blocks > 0) c->htab[2].assign(tab_n, -1);
        c->is_open.assign(spec->max_seqs, 0);
        c->split.assign(spec->max_seqs, 0);
        c->load_end.assign(spec->max_seqs, 0);
        c->window.assign(spec->max_seqs, 0);
        c->length.assign(spec->max_seqs, 0);
        c->segs.resize(spec->max_seqs);
        const int64_t sizes[3] = {spec->host_pool_blocks, spec->device_pool_blocks, spec->load_pool_blocks};
        for (int part = 0; part < 3; ++part) {
            std::vector<int32_t> v(sizes[part]);
            for (int32_t i = 0; i < (int32_t)v.size(); ++i) v[i] = i;
            c->free_slots[part] = MinHeap(std::greater<int32_t>(), std::move(v));
        }
    } catch (const std::bad_alloc &) {
        delete c;
        return fail(WSK_ENOMEM, "host allocation failed");
    }
    const size_t slot_bytes = (size_t)c->slot_elems * 2;
    if (spec->host_pool_blocks > 0) {
        // 2 MB aligned and, where the OS allows, backed by 2 MB pages: the CPU
        // engine reads each KV head's rows in one-block runs a slot apart, and
        // fewer page boundaries mean fewer TLB misses and prefetcher restarts
        // (a hint only; without it the pool is ordinary 4 KB pages)
        const size_t huge = 2u << 20;
        const size_t bytes = ((size_t)spec->host_pool_blocks * slot_bytes + huge - 1) / huge * huge;
        c->hpool = (uint16_t *)aligned_alloc(huge, bytes);
        if (!c->hpool) {
            delete c;
            return fail(WSK_ENOMEM, "host pool of %zu bytes", bytes);
        }
        (void)madvise(c->hpool, bytes, MADV_HUGEPAGE);
        memset(c->hpool, 0, bytes);
    }
    if (device >= 0) {
        DeviceGuard guard(device);
        if (guard.err != hipSuccess) {
            wsk_destroy(c);
            return hip_fail(guard.err, "hipSetDevice");
        }
        hipError_t e = hipDeviceGetAttribute(&c->cu_count, hipDeviceAttributeMultiprocessorCount, device);
        if (e == hipSuccess && c->cu_count <= 0) c->cu_count = 256;
        const size_t pool_bytes = (size_t)spec->device_pool_blocks * slot_bytes;
        if (pool_bytes) e = hipMalloc((void **)&c->dpool, pool_bytes);
        if (e == hipSuccess && pool_bytes) e = hipMemset(c->dpool, 0, pool_bytes);
        const size_t tab_bytes = c->htab[1].size() * sizeof(int32_t);
        if (e == hipSuccess) e = hipMalloc((void **)&c->dtab, tab_bytes);
        if (e == hipSuccess) e = hipMemset(c->dtab, 0xff, tab_bytes);
        if (e == hipSuccess) e = hipMalloc((void **)&c->dstage, kStageBytes);
        const size_t done_bytes = (size_t)kMaxLaunchSeqs * spec->n_q_heads * sizeof(uint32_t);
        if (e == hipSuccess && spec->kind == WSK_KIND_GQA) e = hipMalloc((void **)&c->dstep_done, done_bytes);
        if (e == hipSuccess && c->dstep_done) e = hipMemset(c->dstep_done, 0, done_bytes);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        if (e != hipSuccess) {
            const int r = hip_fail(e, "device allocation");
            wsk_destroy(c);
            return r;
        }
        // the device address of wsk_decode_step_noalloc's scratch array on
        // this device, resolved here once so the step itself only looks it up
        void *scratch = nullptr;
        rc = noalloc_scratch(device, &scratch);
        if (rc) {
            const std::string msg = g_err;
            wsk_destroy(c);
            g_err = msg;
            return rc;
        }
    }
    if (device >= 0 && spec->evict_tokens > 0) {
        rc = evict_init(c);
        if (rc) {
            const std::string msg = g_err;
            wsk_destroy(c);
            g_err = msg;
            return rc;
        }
    }
    if (spec->load_pool_blocks > 0) {
        rc = load_init(c);
        if (rc) {
            const std::string msg = g_err;
            wsk_destroy(c);
            g_err = msg;
            return rc;
        }
    }
    *out = c;
    return WSK_OK;
}

int wsk_destroy(wsk_cache *c) {
    if (!c) return WSK_OK;
    if (c->device >= 0) {
        DeviceGuard guard(c->device);
        if (c->dpool) (void)hipFree(c->dpool);
        if (c->dtab) (void)hipFree(c->dtab);
        if (c->dstage) (void)hipFree(c->dstage);
        if (c->dstep_done) (void)hipFree(c->dstep_done);
        if (c->hsel_ev) (void)hipEventSynchronize(c->hsel_ev);
        if (c->hsel) (void)hipHostFree(c->hsel);
        if (c->hsel_ev) (void)hipEventDestroy(c->hsel_ev);
    }
    load_destroy(c);
    free(c->hpool);
    delete c;
    return WSK_OK;
}

int wsk_get_spec(const wsk_cache *c, wsk_partition_spec *out) {
    if (!c || !out) return fail(WSK_EINVAL, "NULL argument");
    *out = c->spec;
    return WSK_OK;
}

int wsk_seq_open_window(wsk_cache *c, int32_t seq, int32_t split, int32_t load_end) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    if (seq < 0 || seq >= c->spec.max_seqs) return fail(WSK_EINVAL, "sequence id %d out of range", seq);
    if (split < 0) return fail(WSK_EINVAL, "split %d < 0", split);
    if (load_end < split) return fail(WSK_EINVAL, "load_end %d below split %d", load_end, split);
    if (load_end > c->spec.max_seq_len) return fail(WSK_EINVAL, "load_end %d past max_seq_len", load_end);
    if (load_end > split) {
        if (!has_load_region(c)) return fail(WSK_ESTATE, "the cache has no load region");
        if (load_end % c->spec.block_tokens)
            return fail(WSK_EINVAL, "load_end %d must be a multiple of block_tokens", load_end);
    }
    if (c->is_open[seq]) return fail(WSK_ESTATE, "sequence %d already open", seq);
    std::vector<Seg> segs;
    if (split > 0) segs.push_back({0, split, WSK_PART_CPU});
    if (load_end > split) segs.push_back({split, load_end, WSK_PART_LOAD});
    c->segs[seq].swap(segs);
    c->is_open[seq] = 1;
    c->split[seq] = split;
    c->load_end[seq] = load_end;
    c->window[seq] = load_end;
    c->length[seq] = 0;
    return WSK_OK;
}

int wsk_seq_open(wsk_cache *c, int32_t seq, int32_t split) { return wsk_seq_open_window(c, seq, split, split); }

int wsk_seq_close(wsk_cache *c, int32_t seq) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    bool load_freed = false;
    for (int part = 0; part < 3; ++part) {
        if (c->htab[part].empty()) continue;
        for (int32_t k = 0; k < c->max_blocks; ++k) {
            int32_t &t = tab(c, part, seq, k);
            if (t >= 0) {
                c->free_slots[part].push(t);
                t = -1;
                load_freed |= part == WSK_PART_LOAD;
            }
        }
    }
    // a freed load slot may be rewritten by the host as soon as it is reused:
    // transfers still reading or writing it must end first
    if (load_freed && c->device >= 0) {
        DeviceGuard guard(c->device);
        if (c->copy_stream) (void)hipStreamSynchronize(c->copy_stream);
        if (c->flush_ev) (void)hipEventSynchronize(c->flush_ev);
    }
    c->segs[seq].clear();
    c->is_open[seq] = 0;
    c->length[seq] = 0;
    c->split[seq] = 0;
    c->load_end[seq] = 0;
    c->window[seq] = 0;
    return WSK_OK;
}

int wsk_seq_info(const wsk_cache *c, int32_t seq, int32_t *length, int32_t *split) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    if (length) *length = c->length[seq];
    if (split) *split = c->split[seq];
    return WSK_OK;
}

int wsk_reserve(wsk_cache *c, int32_t seq, int32_t n) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    if (n < 0 || (int64_t)c->length[seq] + n > c->spec.max_seq_len)
        return fail(WSK_EINVAL, "reserve of %d positions past max_seq_len", n);
    std::vector<Pending> pend;
    rc = plan(c, seq, c->length[seq], n, pend);
    if (rc) return rc;
    rc = load_ensure(c, pend);
    if (rc) {
        undo(c, pend);
        return rc;
    }
    // the device table must follow for GPU blocks
    if (c->device >= 0) {
        bool any_gpu = false;
        for (const Pending &p : pend) any_gpu |= p.part == WSK_PART_GPU;
        if (any_gpu) {
            DeviceGuard guard(c->device);
            hipError_t e = guard.err;
            for (const Pending &p : pend) {
                if (p.part != WSK_PART_GPU || e != hipSuccess) continue;
                e = hipMemcpy(c->dtab + (size_t)p.seq * c->max_blocks + p.blk, &p.slot, sizeof(int32_t),
                              hipMemcpyHostToDevice);
            }
            if (e != hipSuccess) {
                undo(c, pend);
                return hip_fail(e, "block table update");
            }
        }
    }
    commit(c, pend);
    c->length[seq] += n;
    return WSK_OK;
}

int wsk_write(wsk_cache *c, int32_t seq, int32_t pos0, int32_t n, const void *k, const void *v, void *stream) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    const wsk_partition_spec &sp = c->spec;
    if (n < 0) return fail(WSK_EINVAL, "n < 0");
    if (pos0 != c->length[seq]) return fail(WSK_ERANGE, "write at %d, sequence %d has length %d", pos0, seq, c->length[seq]);
    if ((int64_t)pos0 + n > sp.max_seq_len) return fail(WSK_EINVAL, "write past max_seq_len");
    if (n == 0) return WSK_OK;
    if (!k) return fail(WSK_EINVAL, "k is NULL");
    if (sp.kind == WSK_KIND_GQA && !v) return fail(WSK_EINVAL, "v is NULL");
    if (sp.kind == WSK_KIND_MLA && v) return fail(WSK_EINVAL, "MLA caches take no v");
    const int32_t s = c->split[seq], w0 = std::max(c->load_end[seq], s);
    const int32_t end = pos0 + n;
    const bool has_gpu = end > w0;
    if (has_gpu && c->device < 0) return fail(WSK_ESTATE, "host-only cache cannot hold GPU-partition rows");

    std::vector<Pending> pend;
    rc = plan(c, seq, pos0, n, pend);
    if (rc) return rc;
    rc = load_ensure(c, pend);
    if (rc) {
        undo(c, pend);
        return rc;
    }
    commit(c, pend);

    const int hkv = sp.kind == WSK_KIND_GQA ? sp.n_kv_heads : 1;
    const int nsrc = sp.kind == WSK_KIND_GQA ? 2 : 1;
    const size_t row_bytes = (size_t)c->row_elems * 2;
    const size_t pos_bytes = (size_t)hkv * row_bytes;   // one source position of K (or V)
    const uint16_t *src[2] = {(const uint16_t *)k, (const uint16_t *)v};

    // CPU partition rows: memcpy into the host pool
    for (int32_t p = pos0; p < std::min(end, s); ++p) {
        const int32_t slot = tab(c, WSK_PART_CPU, seq, p / sp.block_tokens);
        uint16_t *base = c->hpool + (int64_t)slot * c->slot_elems;
        for (int w = 0; w < nsrc; ++w)
            for (int g = 0; g < hkv; ++g)
                memcpy(base + row_offset(c, p, g, w), src[w] + ((int64_t)(p - pos0) * hkv + g) * c->row_elems,
                       row_bytes);
    }
    // load-region rows: placed by the host in the GPU slot layout
    if (pos0 < w0 && end > s)
        load_write_rows(c, seq, pos0, std::max(pos0, s), std::min(end, w0), (const uint16_t *)k, (const uint16_t *)v);
    if (!has_gpu) {
        c->length[seq] = end;
        return WSK_OK;
    }

    // GPU partition rows: table update, then H2D through staging + scatter
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    hipStream_t st = (hipStream_t)stream;
    const int32_t g0 = std::max(pos0, w0);
    const int32_t b0 = g0 / sp.block_tokens, b1 = (end - 1) / sp.block_tokens;
    hipError_t e = hipMemcpyAsync(c->dtab + (size_t)seq * c->max_blocks + b0, &tab(c, WSK_PART_GPU, seq, b0),
                                  (size_t)(b1 - b0 + 1) * sizeof(int32_t), hipMemcpyHostToDevice, st);
    const size_t per_piece = kStageBytes / (nsrc * pos_bytes);
    uint16_t *stage[2] = {c->dstage, c->dstage + (kStageBytes / 2) / 2};
    for (int32_t p = g0; p < end && e == hipSuccess; p += (int32_t)per_piece) {
        const int32_t m = (int32_t)std::min<int64_t>(per_piece, end - p);
        for (int w = 0; w < nsrc && e == hipSuccess; ++w)
            e = hipMemcpyAsync(stage[w], src[w] + (int64_t)(p - pos0) * hkv * c->row_elems, (size_t)m * pos_bytes,
                               hipMemcpyHostToDevice, st);
        if (e != hipSuccess) break;
        ScatterParams sc{};
        sc.src_k = stage[0];
        sc.src_v = stage[1];
        sc.pool = c->dpool;
        sc.table_row = c->dtab + (size_t)seq * c->max_blocks;
        sc.slot_elems = c->slot_elems;
        sc.p0 = p;
        sc.m = m;
        sc.kind = sp.kind;
        sc.n_kv_heads = hkv;
        sc.block_tokens = sp.block_tokens;
        sc.row_elems = c->row_elems;
        e = launch_scatter(sc, st);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    c->length[seq] = end;
    if (e != hipSuccess) return hip_fail(e, "wsk_write");
    return WSK_OK;
}

int wsk_append(wsk_cache *c, int32_t n, const int32_t *ids, const void *k_new, const void *v_new, void *stream) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    const wsk_partition_spec &sp = c->spec;
    if (n <= 0 || !ids) return fail(WSK_EINVAL, "n must be positive and seq_ids non-NULL");
    if (!k_new) return fail(WSK_EINVAL, "k_new is NULL");
    if (sp.kind == WSK_KIND_GQA && !v_new) return fail(WSK_EINVAL, "v_new is NULL");
    if (sp.kind == WSK_KIND_MLA && v_new) return fail(WSK_EINVAL, "MLA caches take no v_new");
    if (!aligned16(k_new) || !aligned16(v_new)) return fail(WSK_EINVAL, "k_new/v_new must be 16-byte aligned");
    if (c->device < 0) return fail(WSK_ESTATE, "host-only cache");
    std::vector<int32_t> order(n);
    for (int32_t i = 0; i < n; ++i) {
        int rc = check_seq(c, ids[i]);
        if (rc) return rc;
        order[i] = i;
    }
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return ids[a] < ids[b]; });
    for (int32_t j = 1; j < n; ++j)
        if (ids[order[j]] == ids[order[j - 1]]) return fail(WSK_EINVAL, "sequence %d listed twice", ids[order[j]]);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t sq = ids[i];
        if (c->length[sq] >= sp.max_seq_len) return fail(WSK_ERANGE, "sequence %d is full", sq);
        const int32_t w0 = std::max(c->split[sq], c->load_end[sq]);
        if (c->length[sq] < w0)
            return fail(WSK_ERANGE, "position %d of sequence %d is below the start %d of its GPU pool range",
                        c->length[sq], sq, w0);
    }
    std::vector<Pending> pend;
    for (int32_t j = 0; j < n; ++j) {
        const int32_t sq = ids[order[j]];
        int rc = plan(c, sq, c->length[sq], 1, pend);
        if (rc) return rc;
    }
    // the routes are committed, and the lengths bumped, only once every launch
    // has been enqueued: a failed launch leaves the cache as it was (a new
    // block's device table entry is written by the kernel, and a later append
    // that routes the block again sends it again)
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) {
        undo(c, pend);
        return hip_fail(guard.err, "hipSetDevice");
    }
    hipStream_t st = (hipStream_t)stream;
    const int hkv = sp.kind == WSK_KIND_GQA ? sp.n_kv_heads : 1;
    hipError_t e = hipSuccess;
    for (int32_t r0 = 0; r0 < n && e == hipSuccess; r0 += kMaxLaunchSeqs) {
        const int32_t m = std::min(kMaxLaunchSeqs, n - r0);
        AppendParams ap{};
        ap.k_new = (const uint16_t *)k_new + (int64_t)r0 * hkv * c->row_elems;
        ap.v_new = v_new ? (const uint16_t *)v_new + (int64_t)r0 * hkv * c->row_elems : nullptr;
        ap.pool = c->dpool;
        ap.table = c->dtab;
        ap.n = m;
        ap.kind = sp.kind;
        ap.n_kv_heads = hkv;
        ap.block_tokens = sp.block_tokens;
        ap.row_elems = c->row_elems;
        for (int32_t r = 0; r < m; ++r) {
            const int32_t sq = ids[r0 + r];
            const int32_t pos = c->length[sq];
            const int32_t blk = pos / sp.block_tokens;
            int32_t slot = tab(c, WSK_PART_GPU, sq, blk);
            ap.tab_index[r] = -1;
            for (const Pending &p : pend)
                if (p.seq == sq && p.part == WSK_PART_GPU && p.blk == blk) {
                    slot = p.slot;
                    ap.tab_index[r] = (int32_t)((size_t)sq * c->max_blocks + blk);
                    ap.tab_slot[r] = slot;
                }
            ap.slot_elem0[r] = (int64_t)slot * c->slot_elems;
            ap.row[r] = pos % sp.block_tokens;
        }
        e = launch_append(ap, st);
    }
    if (e != hipSuccess) {
        undo(c, pend);
        return hip_fail(e, "wsk_append");
    }
    commit(c, pend);
    for (int32_t i = 0; i < n; ++i) c->length[ids[i]] += 1;
    return WSK_OK;
}

int wsk_route(const wsk_cache *c, int32_t seq, int32_t pos, wsk_loc *out) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    if (!out) return fail(WSK_EINVAL, "out is NULL");
    if (pos < 0 || pos >= c->length[seq]) return fail(WSK_ERANGE, "position %d outside [0, %d)", pos, c->length[seq]);
    const int part = home_of(c, seq, pos);
    const int32_t blk = pos / c->spec.block_tokens;
    out->part = part;
    out->logical_block = blk;
    out->slot = c->htab[part][(size_t)seq * c->max_blocks + blk];
    out->offset = pos % c->spec.block_tokens;
    return WSK_OK;
}

int wsk_views(const wsk_cache *c, int32_t seq, wsk_view *cpu, wsk_view *gpu) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    const int64_t slot_bytes = c->slot_elems * 2;
    const int64_t row_bytes = (int64_t)c->row_elems * 2;
    const bool gqa = c->spec.kind == WSK_KIND_GQA;
    const int32_t s = c->split[seq], L = c->length[seq];
    for (int side = 0; side < 2; ++side) {
        wsk_view *v = side == 0 ? cpu : gpu;
        if (!v) continue;
        v->slot_bytes = slot_bytes;
        v->head_bytes = gqa ? 2 * c->spec.block_tokens * row_bytes : 0;
        v->v_bytes = gqa ? (side == 0 ? c->spec.block_tokens * row_bytes : kTile * row_bytes) : 0;
        v->row_bytes = row_bytes;
        v->block_tokens = c->spec.block_tokens;
        v->layout = side == 0 ? WSK_LAYOUT_ROWS : gqa ? WSK_LAYOUT_TILED64 : WSK_LAYOUT_MLA32;
        v->reserved = 0;
        if (side == 0) {
            v->pool = c->hpool;
            v->table = c->htab[0].data() + (size_t)seq * c->max_blocks;
            v->start = 0;
            v->end = std::min(s, L);
            v->is_device = 0;
        } else {
            v->pool = c->dpool;
            v->table = c->dtab ? c->dtab + (size_t)seq * c->max_blocks : nullptr;
            v->start = std::min(c->window[seq], L);
            v->end = L;
            v->is_device = 1;
        }
    }
    return WSK_OK;
}

int wsk_attend_workspace(const wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start,
                         const int32_t *end, size_t *bytes) {
    if (!c || !bytes) return fail(WSK_EINVAL, "NULL argument");
    AttendPlan pl;
    int rc = make_plan(c, n, ids, start, end, pl);
    if (rc) return rc;
    *bytes = pl.bytes;
    return WSK_OK;
}

}  // extern "C"

void wsk::attend_params(const wsk_cache *c, const AttendPlan &pl, AttendParams &ap) {
    const wsk_partition_spec &sp = c->spec;
    const bool gqa = sp.kind == WSK_KIND_GQA;
    const int qw = gqa ? kHeadDim : kLatent + kRope;
    ap.slot_elems = c->slot_elems;
    ap.q_row = (int64_t)sp.n_q_heads * qw;
    ap.n_q_heads = sp.n_q_heads;
    ap.n_kv_heads = gqa ? sp.n_kv_heads : 1;
    ap.group = sp.n_q_heads / ap.n_kv_heads;
    ap.head_groups = gqa ? pl.head_groups : 1;
    ap.block_tokens = sp.block_tokens;
    ap.scale_log2 = sp.softmax_scale * 1.4426950408889634f;
}

int wsk::fill_attend(const wsk_cache *c, const RowLaunch &rl, int32_t i0, int32_t m, const void *q, float *part_o,
                     float *part_lse, AttendParams &ap) {
    ap = AttendParams{};
    attend_params(c, rl.plan, ap);
    ap.pool = rl.pool;
    ap.table = rl.table;
    ap.table_stride = rl.table_stride;
    ap.q = (const uint16_t *)q + (int64_t)i0 * ap.q_row;
    ap.part_o = part_o;
    ap.part_lse = part_lse;
    ap.n = m;
    const int units = ap.n_kv_heads * ap.head_groups;
    for (int32_t r = 0; r < m; ++r) {
        const int32_t i = i0 + r;
        const int32_t nc = rl.plan.nchunks[i];
        // an empty range (an empty partial of a decode step) reads no tile
        const bool live = nc && rl.end[i] > rl.start[i];
        ap.seq[r] = live ? rl.trow[i] : 0;
        ap.start[r] = live ? rl.start[i] : 0;
        ap.end[r] = live ? rl.end[i] : 0;
        ap.tpc[r] = rl.plan.tpc[i];
        ap.chunk_begin[r] = (int32_t)rl.pbase[i];
    }
    // one past the last sequence's partials (contiguous when nothing is streamed)
    ap.chunk_begin[m] = (int32_t)(rl.pbase[i0 + m - 1] + rl.plan.nchunks[i0 + m - 1]);
    const size_t k = (size_t)(i0 / kMaxLaunchSeqs);
    ap.flat_wgs = rl.plan.launch_wgs[k];
    if (ap.flat_wgs > 0) {   // the flat split (GQA)
        for (int32_t r = 0; r < m; ++r) {
            ap.flat_begin[r] = rl.plan.flat_first[i0 + r];
            ap.wfirst[r] = rl.plan.wfirst[i0 + r];
        }
        ap.flat_begin[m] = rl.plan.launch_tiles[k];
        return ap.flat_wgs * units;
    }
    ap.wg_begin[0] = 0;
    for (int32_t r = 0; r < m; ++r) ap.wg_begin[r + 1] = ap.wg_begin[r] + rl.plan.nchunks[i0 + r] * units;
    for (int32_t r = m + 1; r <= kMaxLaunchSeqs; ++r) ap.wg_begin[r] = ap.wg_begin[m];
    return ap.wg_begin[m];
}

hipError_t wsk::launch_rows(const wsk_cache *c, const RowLaunch &rl, int32_t n, const void *q, float *part_o,
                            float *part_lse, hipStream_t st) {
    hipError_t e = hipSuccess;
    for (int32_t i0 = 0; i0 < n && e == hipSuccess; i0 += kMaxLaunchSeqs) {
        const int32_t m = std::min(kMaxLaunchSeqs, n - i0);
        AttendParams ap;
        const int n_wg = fill_attend(c, rl, i0, m, q, part_o, part_lse, ap);
        if (n_wg == 0) continue;
        if (c->spec.kind == WSK_KIND_GQA)
            e = launch_gqa_attend(ap, rl.plan.heads_per_wg, n_wg, st);
        else
            e = launch_mla_attend(ap, n_wg, st);
    }
    return e;
}

hipError_t wsk::launch_combine_all(const wsk_cache *c, int32_t n, const std::vector<int64_t> &pb,
                                   const float *part_o, const float *part_lse, const float *o_x,
                                   const float *lse_x, float *o, float *lse, hipStream_t st) {
    const wsk_partition_spec &sp = c->spec;
    const int width = sp.kind == WSK_KIND_GQA ? kHeadDim : kLatent;
    hipError_t e = hipSuccess;
    for (int32_t i0 = 0; i0 < n && e == hipSuccess; i0 += kMaxLaunchSeqs) {
        const int32_t m = std::min(kMaxLaunchSeqs, n - i0);
        CombineParams cp{};
        cp.part_o = part_o + pb[i0] * sp.n_q_heads * width;
        cp.part_lse = part_lse + pb[i0] * sp.n_q_heads;
        cp.o = o + (int64_t)i0 * sp.n_q_heads * width;
        cp.lse = lse + (int64_t)i0 * sp.n_q_heads;
        cp.o_x = o_x ? o_x + (int64_t)i0 * sp.n_q_heads * width : nullptr;
        cp.lse_x = lse_x ? lse_x + (int64_t)i0 * sp.n_q_heads : nullptr;
        cp.n = m;
        cp.n_q_heads = sp.n_q_heads;
        for (int32_t r = 0; r <= kMaxLaunchSeqs; ++r) cp.chunk_begin[r] = (int32_t)(pb[i0 + std::min(r, m)] - pb[i0]);
        e = launch_combine(cp, width, st);
    }
    return e;
}

int wsk::check_outputs(const void *q, const float *o, const float *lse, const float *o_x, const float *lse_x,
                       bool pass1, bool pass2) {
    if (pass1 && !q) return fail(WSK_EINVAL, "q must not be NULL");
    if (pass2 && (!o || !lse)) return fail(WSK_EINVAL, "o/lse must not be NULL");
    if (!aligned16(q) || !aligned16(o)) return fail(WSK_EINVAL, "q and o must be 16-byte aligned");
    if ((o_x == nullptr) != (lse_x == nullptr)) return fail(WSK_EINVAL, "o_x and lse_x must both be given or both NULL");
    if (!aligned16(o_x)) return fail(WSK_EINVAL, "o_x must be 16-byte aligned");
    return WSK_OK;
}

namespace {

// wsk_attend and its two passes over ranges of the GPU pool: pass 1 writes
// the chunk partials into ws, pass 2 merges them (and o_x) into o / lse.
int attend_passes(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
                  const void *q, float *o, float *lse, void *ws, size_t ws_bytes, void *stream, bool pass1,
                  bool pass2, const float *o_x = nullptr, const float *lse_x = nullptr) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    RowLaunch rl;
    int rc = make_plan(c, n, ids, start, end, rl.plan);
    if (rc) return rc;
    if (n == 0) return WSK_OK;
    if (c->device < 0) return fail(WSK_ESTATE, "host-only cache");
    rc = check_outputs(q, o, lse, o_x, lse_x, pass1, pass2);
    if (rc) return rc;
    const AttendPlan &pl = rl.plan;
    if (pl.bytes && (!ws || ws_bytes < pl.bytes)) return fail(WSK_EINVAL, "workspace of %zu bytes needed", pl.bytes);
    if (((uintptr_t)ws & 255) != 0) return fail(WSK_EINVAL, "workspace must be 256-byte aligned");
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    hipStream_t st = (hipStream_t)stream;
    float *part_o = (float *)ws;
    float *part_lse = (float *)((char *)ws + pl.part_o_bytes);
    rl.pool = c->dpool;
    rl.table = c->dtab;
    rl.table_stride = c->max_blocks;
    rl.trow.assign(ids, ids + n);
    rl.start.assign(start, start + n);
    rl.end.assign(end, end + n);
    rl.pbase.assign(n + 1, 0);
    for (int32_t i = 0; i < n; ++i) rl.pbase[i + 1] = rl.pbase[i] + pl.nchunks[i];
    hipError_t e = hipSuccess;
    if (pass1) e = launch_rows(c, rl, n, q, part_o, part_lse, st);
    if (e == hipSuccess && pass2) e = launch_combine_all(c, n, rl.pbase, part_o, part_lse, o_x, lse_x, o, lse, st);
    if (e != hipSuccess) return hip_fail(e, "wsk_attend");
    return WSK_OK;
}

}  // namespace

extern "C" {

int wsk_attend(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
               const void *q, float *o, float *lse, void *ws, size_t ws_bytes, void *stream) {
    return attend_passes(c, n, ids, start, end, q, o, lse, ws, ws_bytes, stream, true, true);
}

int wsk_attend_pass1(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
                     const void *q, void *ws, size_t ws_bytes, void *stream) {
    return attend_passes(c, n, ids, start, end, q, nullptr, nullptr, ws, ws_bytes, stream, true, false);
}

int wsk_attend_pass2(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
                     const float *o_x, const float *lse_x, float *o, float *lse, void *ws, size_t ws_bytes,
                     void *stream) {
    return attend_passes(c, n, ids, start, end, nullptr, o, lse, ws, ws_bytes, stream, false, true, o_x, lse_x);
}

int wsk_merge(int32_t rows, int32_t width, const float *o_a, const float *lse_a, const float *o_b,
              const float *lse_b, float *o_out, float *lse_out, uint16_t *o_bf16, void *stream) {
    if (rows < 0 || width <= 0 || width % 4) return fail(WSK_EINVAL, "rows %d width %d", rows, width);
    if (rows == 0) return WSK_OK;
    if (!o_a || !lse_a || !o_b || !lse_b || !o_out || !lse_out) return fail(WSK_EINVAL, "NULL pointer");
    if (!aligned16(o_a) || !aligned16(o_b) || !aligned16(o_out))
        return fail(WSK_EINVAL, "o_a, o_b and o_out must be 16-byte aligned");
    hipError_t e = launch_merge(rows, width, o_a, lse_a, o_b, lse_b, o_out, lse_out, o_bf16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "wsk_merge");
    return WSK_OK;
}

int wsk_mla_absorb(int32_t n, int32_t H, int32_t dn, int32_t dl, const uint16_t *q_nope, const uint16_t *w_uk,
                   uint16_t *out, int64_t out_stride, void *stream) {
    if (n < 0 || H <= 0 || dn < 1 || dn > 256 || dl <= 0 || dl % 64 || out_stride < dl)
        return fail(WSK_EINVAL, "absorb sizes n=%d H=%d dn=%d dl=%d stride=%lld", n, H, dn, dl, (long long)out_stride);
    if (n == 0) return WSK_OK;
    if (!q_nope || !w_uk || !out) return fail(WSK_EINVAL, "NULL pointer");
    if (!aligned16(w_uk)) return fail(WSK_EINVAL, "w_uk must be 16-byte aligned");
    hipError_t e = launch_mla_absorb(n, H, dn, dl, q_nope, w_uk, out, out_stride, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "wsk_mla_absorb");
    return WSK_OK;
}

int wsk_mla_expand(int32_t n, int32_t H, int32_t dl, int32_t dv, const float *o_lat, const uint16_t *w_uv, float *o,
                   void *stream) {
    if (n < 0 || H <= 0 || dl < 1 || dl > 1024 || dv <= 0 || dv % 64)
        return fail(WSK_EINVAL, "expand sizes n=%d H=%d dl=%d dv=%d", n, H, dl, dv);
    if (n == 0) return WSK_OK;
    if (!o_lat || !w_uv || !o) return fail(WSK_EINVAL, "NULL pointer");
    if (!aligned16(w_uv)) return fail(WSK_EINVAL, "w_uv must be 16-byte aligned");
    hipError_t e = launch_mla_expand(n, H, dl, dv, o_lat, w_uv, o, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "wsk_mla_expand");
    return WSK_OK;
}

int wsk_cpu_attend(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *start, const int32_t *end,
                   const void *q, float *o, float *lse, int32_t threads) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    if (n < 0) return fail(WSK_EINVAL, "n < 0");
    if (n == 0) return WSK_OK;
    if (!ids || !start || !end || !q || !o || !lse) return fail(WSK_EINVAL, "NULL argument");
    std::vector<const int32_t *> tables(n);
    for (int32_t i = 0; i < n; ++i) {
        int rc = check_seq(c, ids[i]);
        if (rc) return rc;
        if (!range_in(c, ids[i], start[i], end[i], WSK_PART_CPU))
            return fail(WSK_ERANGE, "range [%d, %d) of sequence %d is not all in its CPU partition", start[i], end[i],
                        ids[i]);
        tables[i] = c->htab[WSK_PART_CPU].data() + (size_t)ids[i] * c->max_blocks;
    }
    const wsk_partition_spec &sp = c->spec;
    const bool mla = sp.kind == WSK_KIND_MLA;
    CpuAttendArgs x{};
    x.pool = c->hpool;
    x.tables = tables.data();
    x.start = start;
    x.end = end;
    x.q = (const uint16_t *)q;
    x.o = o;
    x.lse = lse;
    x.slot_elems = c->slot_elems;
    x.n = n;
    x.n_q_heads = sp.n_q_heads;
    x.group = mla ? sp.n_q_heads : sp.n_q_heads / sp.n_kv_heads;
    x.row_elems = c->row_elems;
    x.dv = mla ? sp.latent_dim : sp.head_dim;
    x.q_row = (int64_t)sp.n_q_heads * c->row_elems;
    x.block_tokens = sp.block_tokens;
    x.mla = mla;
    x.scale_log2 = sp.softmax_scale * 1.4426950408889634f;
    x.threads = threads > 0 ? threads : (int)std::max(1u, std::thread::hardware_concurrency());
    return cpu_attend(x);
}

int wsk_host_read(const void *p, size_t bytes, int32_t threads, uint64_t *out) {
    if (!p || !out || bytes == 0 || bytes % 8) return fail(WSK_EINVAL, "host_read arguments");
    *out = host_read(p, bytes, threads > 0 ? threads : (int)std::max(1u, std::thread::hardware_concurrency()));
    return WSK_OK;
}

int wsk_stream_read(const void *p, size_t bytes, int32_t workgroups, uint32_t *out, void *stream) {
    if (!p || !out || bytes == 0 || bytes % 32768 || !aligned16(p)) return fail(WSK_EINVAL, "stream_read arguments");
    int dev = 0, cus = 256;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int n_wg = workgroups > 0 ? workgroups : std::max(1, gqa_resident_slots(cus));
    if (e == hipSuccess) e = launch_stream_read(p, (int64_t)bytes, out, n_wg, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "wsk_stream_read");
    return WSK_OK;
}

}  // extern "C"
