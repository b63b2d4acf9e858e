// The GPU side's host-resident data (Sec. 4.2, 4.3, 4.4): the pinned load
// region, its streaming through a ping-pong pair of HBM buffers into the
// pass-1 kernels, D-window eviction (flush), block-sparse selections with the
// gather into pinned staging, and the CPU engine over every CPU position.
//
// The load region stores slots in the GPU pool's layout, so a DMA lands
// blocks the kernels read unchanged: the host places rows into that layout
// when it writes them (the paper's layout attribute fixed by the format).
// A sequence's GPU-side positions are its load-region segments plus the
// D-window [window, L) in HBM; blocks never mix the two (load_end and every
// flush boundary after it are block-aligned), and the only partial blocks
// are the one holding s (positions >= s) and the one holding L - 1.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

#include "cache.h"

using namespace wsk;

namespace {

// Whether pinned host memory at p is mapped for the device at the same
// address, so that a kernel can store into it directly.
bool device_maps(void *p) {
    void *d = nullptr;
    return hipHostGetDevicePointer(&d, p, 0) == hipSuccess && d == p;
}

// ---- GPU slot layouts, host side -------------------------------------------
// Pieces are 16 bytes (8 bf16).  GQA (64-token tiles, per KV head): K piece j
// (dims 8j..8j+7) of token t, and V element (t, d); MLA (32-token tiles):
// piece c (dims 8c..8c+7) of token u.
constexpr int kPiece = 8;
constexpr int kGqaTilePieces = 2048;   // K 1024 + V 1024
constexpr int kMlaTilePieces = 2304;

inline int gqa_k_piece(int t, int j) {
    const int mt = 2 * (t / 32) + (t % 8) / 4;
    const int nk = 4 * ((t % 32) / 8) + t % 4;
    return (4 * mt + j / 4) * 64 + 16 * (j % 4) + nk;
}
inline int64_t gqa_v_elem(int t, int d) {   // element index inside the V half of a tile
    return (int64_t)((2 * (d / 16) + t / 32) * 64 + 16 * ((t % 32) / 8) + d % 16) * kPiece + t % 8;
}
inline int mla_piece(int u, int c) { return (2 * (c / 4) + (u / 4) % 2) * 64 + 16 * (c % 4) + 4 * (u / 8) + u % 4; }

// Places the rows of one position (row offset off in its block) into a slot
// of GPU layout.  GQA: k[g], v[g] = the head_dim row of KV head g; MLA: k[0].
void put_position(const wsk_cache *c, uint16_t *slot, int off, const uint16_t *const *k,
                  const uint16_t *const *v) {
    const int bk = c->spec.block_tokens;
    if (c->spec.kind == WSK_KIND_MLA) {
        uint16_t *tile = slot + (int64_t)(off / 32) * kMlaTilePieces * kPiece;
        const int u = off % 32;
        for (int p = 0; p < (kLatent + kRope) / kPiece; ++p)
            memcpy(tile + (int64_t)mla_piece(u, p) * kPiece, k[0] + p * kPiece, 16);
        return;
    }
    const int t = off % 64;
    for (int g = 0; g < c->spec.n_kv_heads; ++g) {
        uint16_t *tile = slot + ((int64_t)g * (bk / 64) + off / 64) * kGqaTilePieces * kPiece;
        for (int j = 0; j < kHeadDim / kPiece; ++j) memcpy(tile + (int64_t)gqa_k_piece(t, j) * kPiece, k[g] + j * kPiece, 16);
        uint16_t *vt = tile + 1024 * kPiece;
        for (int d = 0; d < kHeadDim; ++d) vt[gqa_v_elem(t, d)] = v[g][d];
    }
}

// The inverse: reads the rows of one position out of a slot of GPU layout.
int32_t arena_blocks(const wsk_cache *c) { return c->spec.load_arena_blocks; }
int32_t sp_pingpong(const wsk_cache *c) { return c->spec.pingpong_blocks; }

// Host threads for the block gathers and row rewrites: one thread copies
// ~20 GB/s, the host-to-device link takes ~57, so a few threads keep the
// link busy.
int gather_threads() { return (int)std::min(8u, std::max(1u, std::thread::hardware_concurrency())); }

// Allocates arena k: pinned (hipHostMalloc) on a device cache, plain aligned
// host memory on a host-only one, and writes zeros over it.  The first write
// is where the pages are really faulted in and locked (measured on an MI355X
// system: the allocation call ~0.003 ms/MiB, the first touch by one thread
// ~0.37 ms/MiB), so it is done here, off the critical path, in 2 MiB pieces
// on several threads.  Records the time spent.
int pin_arena(wsk_cache *c, size_t k) {
    if (c->arenas[k]) return WSK_OK;
    const int64_t first = (int64_t)k * arena_blocks(c);
    const int64_t slots = std::min<int64_t>(arena_blocks(c), c->spec.load_pool_blocks - first);
    const size_t bytes = (size_t)slots * slot_bytes(c);
    const auto t0 = std::chrono::steady_clock::now();
    void *p = nullptr;
    if (c->device >= 0) {
        DeviceGuard guard(c->device);
        if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
        hipError_t e = hipHostMalloc(&p, bytes, hipHostMallocDefault);
        if (e != hipSuccess) return fail(WSK_ENOMEM, "pinning %zu bytes of the load region: %s", bytes,
                                         hipGetErrorString(e));
    } else {
        p = aligned_alloc(64, (bytes + 63) / 64 * 64);
        if (!p) return fail(WSK_ENOMEM, "load region arena of %zu bytes", bytes);
    }
    const size_t piece = 2u << 20;
    parallel_tasks((int)((bytes + piece - 1) / piece), gather_threads(), [&](int t) {
        const size_t a = (size_t)t * piece;
        memset((char *)p + a, 0, std::min(piece, bytes - a));
    });
    c->pin_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    c->pinned_bytes += (int64_t)bytes;
    c->arenas[k] = (uint16_t *)p;
    c->arena_mapped[k] = c->device >= 0 && device_maps(p);
    return WSK_OK;
}

}  // namespace

// ---- region management ---------------------------------------------------------

uint16_t *wsk::load_slot_ptr(const wsk_cache *c, int32_t slot) {
    return c->arenas[slot / arena_blocks(c)] + (int64_t)(slot % arena_blocks(c)) * c->slot_elems;
}

int wsk::load_ensure(wsk_cache *c, const std::vector<Pending> &pend) {
    int32_t hi = -1;
    for (const Pending &p : pend) {
        if (p.part != WSK_PART_LOAD) continue;
        int rc = pin_arena(c, (size_t)(p.slot / arena_blocks(c)));
        if (rc) return rc;
        hi = std::max(hi, p.slot);
    }
    // pin one arena ahead once the current one is half used, so that later
    // writes and evictions find their memory already pinned
    if (hi >= 0 && hi % arena_blocks(c) >= arena_blocks(c) / 2) {
        const size_t next = (size_t)(hi / arena_blocks(c)) + 1;
        if (next < c->arenas.size()) (void)pin_arena(c, next);   // a failure here is retried when needed
    }
    return WSK_OK;
}

int wsk::load_init(wsk_cache *c) {
    const int64_t A = arena_blocks(c);
    c->arenas.assign((size_t)((c->spec.load_pool_blocks + A - 1) / A), nullptr);
    c->arena_mapped.assign(c->arenas.size(), 0);
    if (c->device < 0) return WSK_OK;
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    const int32_t P = c->spec.pingpong_blocks;
    const size_t buf = (size_t)P * slot_bytes(c);
    hipError_t e = hipSuccess;
    for (int b = 0; b < 2 && e == hipSuccess; ++b) e = hipMalloc((void **)&c->pingpong[b], buf);
    if (e == hipSuccess) e = hipMalloc((void **)&c->dident, (size_t)P * sizeof(int32_t));
    if (e == hipSuccess) {
        std::vector<int32_t> ident(P);
        for (int32_t i = 0; i < P; ++i) ident[i] = i;
        e = hipMemcpy(c->dident, ident.data(), (size_t)P * sizeof(int32_t), hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->copy_stream, hipStreamNonBlocking);
    hipEvent_t *evs[] = {&c->filled[0], &c->filled[1], &c->consumed[0], &c->consumed[1],
                         &c->staged[0], &c->staged[1], &c->flush_ev};
    for (hipEvent_t *ev : evs)
        if (e == hipSuccess) e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
    // every wait on these events is valid from the start
    for (hipEvent_t *ev : evs)
        if (e == hipSuccess) e = hipEventRecord(*ev, c->copy_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->copy_stream);
    if (e != hipSuccess) return hip_fail(e, "load region set-up");
    return WSK_OK;
}

// Blocks of one eviction round: what the device staging holds, at most
// kEvictMax (the gather kernel's argument list).
static size_t evict_round_blocks(const wsk_cache *c) {
    return std::max<size_t>(1, std::min<size_t>(kEvictMax, kStageBytes / slot_bytes(c)));
}

// The pinned bounce that evictions to the CPU pool land in, sized for one
// batch of every sequence (capped at one round), and its piece events:
// allocated and touched here, so a flush does not pin memory on its way.
int wsk::evict_init(wsk_cache *c) {
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    const int bk = c->spec.block_tokens;
    const size_t blocks = std::min<size_t>(evict_round_blocks(c),
                                           (size_t)c->spec.max_seqs * (size_t)(c->spec.evict_tokens / bk + 1));
    const size_t bytes = blocks * slot_bytes(c);
    hipError_t e = hipHostMalloc((void **)&c->hbounce, bytes, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(e, "pinned eviction bounce");
    c->hbounce_bytes = bytes;
    memset(c->hbounce, 0, bytes);
    c->bounce_mapped = device_maps(c->hbounce);
    for (hipEvent_t &ev : c->bounce_ev) {
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
    return WSK_OK;
}

void wsk::load_destroy(wsk_cache *c) {
    if (c->device >= 0) {
        DeviceGuard guard(c->device);
        if (c->copy_stream) (void)hipStreamSynchronize(c->copy_stream);
        if (c->flush_ev) (void)hipEventSynchronize(c->flush_ev);
        for (int b = 0; b < 2; ++b) {
            if (c->consumed[b]) (void)hipEventSynchronize(c->consumed[b]);
            if (c->pingpong[b]) (void)hipFree(c->pingpong[b]);
            if (c->hgather[b]) (void)hipHostFree(c->hgather[b]);
        }
        if (c->dident) (void)hipFree(c->dident);
        if (c->hbounce) (void)hipHostFree(c->hbounce);
        hipEvent_t evs[] = {c->filled[0], c->filled[1], c->consumed[0], c->consumed[1],
                            c->staged[0], c->staged[1], c->flush_ev};
        for (hipEvent_t ev : evs)
            if (ev) (void)hipEventDestroy(ev);
        for (hipEvent_t ev : c->bounce_ev)
            if (ev) (void)hipEventDestroy(ev);
        if (c->copy_stream) (void)hipStreamDestroy(c->copy_stream);
        for (uint16_t *a : c->arenas)
            if (a) (void)hipHostFree(a);
    } else {
        for (uint16_t *a : c->arenas) free(a);
    }
    c->arenas.clear();
}

void wsk::load_write_rows(wsk_cache *c, int32_t seq, int32_t pos0, int32_t p0, int32_t p1, const uint16_t *k,
                          const uint16_t *v) {
    const int bk = c->spec.block_tokens;
    const bool gqa = c->spec.kind == WSK_KIND_GQA;
    const int hkv = gqa ? c->spec.n_kv_heads : 1;
    if (p1 <= p0) return;
    // one task per block: each writes its own slot
    const int32_t b0 = p0 / bk, b1 = (p1 - 1) / bk;
    parallel_tasks(b1 - b0 + 1, gather_threads(), [&](int t) {
        const int32_t blk = b0 + t;
        uint16_t *slot = load_slot_ptr(c, tab(c, WSK_PART_LOAD, seq, blk));
        std::vector<const uint16_t *> kp(hkv), vp(hkv);
        for (int32_t p = std::max(p0, blk * bk); p < std::min(p1, (blk + 1) * bk); ++p) {
            for (int g = 0; g < hkv; ++g) {
                kp[g] = k + ((int64_t)(p - pos0) * hkv + g) * c->row_elems;
                vp[g] = gqa ? v + ((int64_t)(p - pos0) * hkv + g) * c->row_elems : nullptr;
            }
            put_position(c, slot, p % bk, kp.data(), vp.data());
        }
    });
}

// ---- the GPU side of a step: plan ---------------------------------------------
namespace {

// One load-region block to stream: call row i, load slot, the positions
// [lo, hi) of the block that are attended.
struct LoadPiece {
    int32_t i, slot, lo, hi;
};

// The work of one wsk_attend_gpu / wsk_attend_blocks call.
struct GpuPlan {
    RowLaunch hbm;                   // GPU-pool rows, read in place
    std::vector<int32_t> sel_tab;    // compacted table rows (selections only)
    int32_t sel_width = 0;
    std::vector<LoadPiece> pieces;   // in call-row order; a row's partial pieces at its ends
    std::vector<size_t> chunk_first; // first piece of each ping-pong chunk, then pieces.size()
    std::vector<RowLaunch> chunks;
    std::vector<int64_t> pb;         // partials of row i: [pb[i], pb[i + 1])
    size_t part_o_bytes = 0, part_lse_bytes = 0, sel_off = 0, bytes = 0;
};

inline size_t up256(size_t x) { return (x + 255) / 256 * 256; }

// Rows of the ping-pong chunks and the partial layout, once hbm and pieces
// are set.
void finish_plan(const wsk_cache *c, int32_t n, GpuPlan &g) {
    const int32_t P = std::max(c->spec.pingpong_blocks, 1);
    const int bk = c->spec.block_tokens;
    g.chunk_first.clear();
    for (size_t j = 0; j < g.pieces.size(); j += (size_t)P) g.chunk_first.push_back(j);
    g.chunk_first.push_back(g.pieces.size());
    const size_t nch = g.chunk_first.size() - 1;
    g.chunks.assign(nch, RowLaunch());
    for (size_t k = 0; k < nch; ++k) {
        RowLaunch &rl = g.chunks[k];
        rl.trow.assign(n, 0);
        rl.start.assign(n, 0);
        rl.end.assign(n, 0);
        const size_t j0 = g.chunk_first[k], j1 = g.chunk_first[k + 1];
        for (size_t j = j0; j < j1;) {
            const int32_t i = g.pieces[j].i;
            size_t e = j;
            while (e < j1 && g.pieces[e].i == i) ++e;
            rl.trow[i] = (int32_t)(j - j0);   // staged slots of row i: j - j0 .. e - j0 - 1
            rl.start[i] = g.pieces[j].lo;
            rl.end[i] = (int32_t)(e - j - 1) * bk + g.pieces[e - 1].hi;
            j = e;
        }
        plan_chunks(c, n, rl.start.data(), rl.end.data(), rl.plan);
    }
    g.pb.assign(n + 1, 0);
    for (int32_t i = 0; i < n; ++i) {
        int64_t cnt = g.hbm.plan.nchunks[i];
        for (const RowLaunch &rl : g.chunks) cnt += rl.plan.nchunks[i];
        g.pb[i + 1] = g.pb[i] + cnt;
    }
    g.hbm.pbase.assign(n, 0);
    for (RowLaunch &rl : g.chunks) rl.pbase.assign(n, 0);
    for (int32_t i = 0; i < n; ++i) {
        int64_t p = g.pb[i];
        g.hbm.pbase[i] = p;
        p += g.hbm.plan.nchunks[i];
        for (RowLaunch &rl : g.chunks) {
            rl.pbase[i] = p;
            p += rl.plan.nchunks[i];
        }
    }
    const int width = c->spec.kind == WSK_KIND_GQA ? kHeadDim : kLatent;
    const int64_t partials = g.pb[n];
    g.part_o_bytes = up256((size_t)partials * c->spec.n_q_heads * width * sizeof(float));
    g.part_lse_bytes = up256((size_t)partials * c->spec.n_q_heads * sizeof(float));
    g.sel_off = g.part_o_bytes + g.part_lse_bytes;
    g.bytes = g.sel_off + up256(g.sel_tab.size() * sizeof(int32_t));
}

int check_ids(const wsk_cache *c, int32_t n, const int32_t *ids) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    if (n < 0) return fail(WSK_EINVAL, "n < 0");
    if (n > 0 && !ids) return fail(WSK_EINVAL, "seq_ids is NULL");
    for (int32_t i = 0; i < n; ++i) {
        int rc = check_seq(c, ids[i]);
        if (rc) return rc;
    }
    return WSK_OK;
}

// Every GPU-side position of each sequence: the D-window in place, every
// load-region block streamed.  fused_step: the plan of a GQA decode step,
// whose pass 2 runs inside its pass-1 launch when nothing is streamed (then
// every sequence gets at least one chunk).
int plan_dense(const wsk_cache *c, int32_t n, const int32_t *ids, GpuPlan &g, bool fused_step = false) {
    int rc = check_ids(c, n, ids);
    if (rc) return rc;
    const int bk = c->spec.block_tokens;
    g.hbm.trow.assign(ids, ids + n);
    g.hbm.start.resize(n);
    g.hbm.end.resize(n);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t sq = ids[i], L = c->length[sq];
        g.hbm.start[i] = std::min(c->window[sq], L);
        g.hbm.end[i] = L;
        for (const Seg &s : c->segs[sq]) {
            if (s.part != WSK_PART_LOAD) continue;
            const int32_t e = std::min(s.e, L);
            for (int32_t blk = s.a / bk; blk * bk < e; ++blk) {
                const int32_t lo = std::max(s.a - blk * bk, 0), hi = std::min(e - blk * bk, bk);
                g.pieces.push_back({i, tab(c, WSK_PART_LOAD, sq, blk), lo, hi});
            }
        }
    }
    plan_chunks(c, n, g.hbm.start.data(), g.hbm.end.data(), g.hbm.plan, fused_step && g.pieces.empty());
    finish_plan(c, n, g);
    return WSK_OK;
}

// A block selection: selected GPU-pool blocks through a compacted table row
// (the window's first block first, the block holding L - 1 last), selected
// load-region blocks streamed (a partial first block first).
int plan_selection(const wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *sel_begin, const int32_t *sel,
                   GpuPlan &g) {
    int rc = check_ids(c, n, ids);
    if (rc) return rc;
    if (n > 0 && !sel_begin) return fail(WSK_EINVAL, "sel_begin is NULL");
    if (n > 0 && sel_begin[0] != 0) return fail(WSK_EINVAL, "sel_begin[0] must be 0");
    const int bk = c->spec.block_tokens;
    int32_t width = 1;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t k = sel_begin[i + 1] - sel_begin[i];
        if (k < 0) return fail(WSK_EINVAL, "sel_begin must not decrease");
        if (k > 0 && !sel) return fail(WSK_EINVAL, "sel is NULL");
        width = std::max(width, k);
    }
    g.sel_width = width;
    g.sel_tab.assign((size_t)n * width, 0);
    g.hbm.trow.resize(n);
    g.hbm.start.assign(n, 0);
    g.hbm.end.assign(n, 0);
    std::vector<uint8_t> seen;
    for (int32_t i = 0; i < n; ++i) {
        g.hbm.trow[i] = i;
        const int32_t sq = ids[i], L = c->length[sq];
        const int32_t k = sel_begin[i + 1] - sel_begin[i];
        if (k == 0) continue;
        const int32_t w = std::min(c->window[sq], L);
        const int32_t first = w / bk, last = (L - 1) / bk;   // GPU-pool blocks [first, last] when w < L
        seen.assign(c->max_blocks, 0);
        bool has_first = false, has_last = false;
        std::vector<int32_t> mid;
        std::vector<LoadPiece> lhead, lmid, ltail;
        for (int32_t j = 0; j < k; ++j) {
            const int32_t b = sel[sel_begin[i] + j];
            if (b < 0 || b >= c->max_blocks || b * bk >= L)
                return fail(WSK_ERANGE, "block %d of sequence %d is not written", b, sq);
            if (seen[b]) return fail(WSK_EINVAL, "block %d of sequence %d selected twice", b, sq);
            seen[b] = 1;
            if (w < L && b >= first) {
                if (b == first) has_first = true;
                if (b == last) has_last = true;
                if (b != first && b != last) mid.push_back(b);
                continue;
            }
            // a load-region block: its load positions are one run [lo, hi)
            int32_t lo = -1, hi = -1;
            for (const Seg &s : c->segs[sq]) {
                if (s.part != WSK_PART_LOAD) continue;
                const int32_t a = std::max(s.a, b * bk), e = std::min({s.e, (b + 1) * bk, L});
                if (a < e) {
                    lo = a - b * bk;
                    hi = e - b * bk;
                }
            }
            if (lo < 0) return fail(WSK_ERANGE, "block %d of sequence %d has no GPU-side positions", b, sq);
            const LoadPiece pc{i, tab(c, WSK_PART_LOAD, sq, b), lo, hi};
            (lo > 0 ? lhead : hi < bk ? ltail : lmid).push_back(pc);
        }
        std::vector<int32_t> order;
        if (has_first) order.push_back(first);
        order.insert(order.end(), mid.begin(), mid.end());
        if (has_last && last != first) order.push_back(last);
        for (size_t j = 0; j < order.size(); ++j)
            g.sel_tab[(size_t)i * width + j] = tab(c, WSK_PART_GPU, sq, order[j]);
        if (!order.empty()) {
            g.hbm.start[i] = has_first ? w - first * bk : 0;
            g.hbm.end[i] = (int32_t)(order.size() - 1) * bk + (has_last ? L - last * bk : bk);
        }
        g.pieces.insert(g.pieces.end(), lhead.begin(), lhead.end());
        g.pieces.insert(g.pieces.end(), lmid.begin(), lmid.end());
        g.pieces.insert(g.pieces.end(), ltail.begin(), ltail.end());
    }
    plan_chunks(c, n, g.hbm.start.data(), g.hbm.end.data(), g.hbm.plan);
    finish_plan(c, n, g);
    return WSK_OK;
}

// ---- the GPU side of a step: execution --------------------------------------------
int check_run(const wsk_cache *c, const GpuPlan &g, const void *q, const float *o_x, const float *lse_x, float *o,
              float *lse, void *ws, size_t ws_bytes, bool pass1, bool pass2) {
    if (c->device < 0) return fail(WSK_ESTATE, "host-only cache");
    int rc = check_outputs(q, o, lse, o_x, lse_x, pass1, pass2);
    if (rc) return rc;
    if (!ws || ws_bytes < g.bytes) return fail(WSK_EINVAL, "workspace of %zu bytes needed", g.bytes);
    if (((uintptr_t)ws & 255) != 0) return fail(WSK_EINVAL, "workspace must be 256-byte aligned");
    if (!g.chunks.empty() && !c->copy_stream) return fail(WSK_ESTATE, "the cache has no load region");
    return WSK_OK;
}

// Pass 1 of a plan (pass1) and its combine (pass2).  The combine is skipped
// when step is set: the caller launches its own pass 2.
int run_plan(wsk_cache *c, int32_t n, GpuPlan &g, bool gather, const void *q, const float *o_x, const float *lse_x,
             float *o, float *lse, void *ws, size_t ws_bytes, void *stream, bool pass1 = true, bool pass2 = true) {
    if (n == 0) return WSK_OK;
    int rc = check_run(c, g, q, o_x, lse_x, o, lse, ws, ws_bytes, pass1, pass2);
    if (rc) return rc;
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    hipStream_t st = (hipStream_t)stream, cs = c->copy_stream;
    float *part_o = (float *)ws;
    float *part_lse = (float *)((char *)ws + g.part_o_bytes);
    hipError_t e = hipSuccess;
    if (!pass1) {
        e = launch_combine_all(c, n, g.pb, part_o, part_lse, o_x, lse_x, o, lse, st);
        if (e != hipSuccess) return hip_fail(e, "GPU-side attention, pass 2");
        return WSK_OK;
    }

    // GPU-pool rows, in place
    g.hbm.pool = c->dpool;
    if (!g.sel_tab.empty()) {
        int32_t *dsel = (int32_t *)((char *)ws + g.sel_off);
        const size_t bytes = g.sel_tab.size() * sizeof(int32_t);
        if (!c->hsel_ev) e = hipEventCreateWithFlags(&c->hsel_ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventSynchronize(c->hsel_ev);   // the previous upload has left the buffer
        if (e == hipSuccess && c->hsel_bytes < bytes) {
            if (c->hsel) (void)hipHostFree(c->hsel);
            c->hsel = nullptr;
            c->hsel_bytes = 0;
            e = hipHostMalloc((void **)&c->hsel, bytes, hipHostMallocDefault);
            if (e == hipSuccess) c->hsel_bytes = bytes;
        }
        if (e == hipSuccess) {
            memcpy(c->hsel, g.sel_tab.data(), bytes);
            e = hipMemcpyAsync(dsel, c->hsel, bytes, hipMemcpyHostToDevice, st);
        }
        if (e == hipSuccess) e = hipEventRecord(c->hsel_ev, st);
        g.hbm.table = dsel;
        g.hbm.table_stride = g.sel_width;
    } else {
        g.hbm.table = c->dtab;
        g.hbm.table_stride = c->max_blocks;
    }
    if (e == hipSuccess) e = launch_rows(c, g.hbm, n, q, part_o, part_lse, st);

    // load-region blocks through the ping-pong pair
    const size_t nch = g.chunks.size();
    const size_t sb = slot_bytes(c);
    if (nch && e == hipSuccess) {
        if (gather) e = hipEventSynchronize(c->flush_ev);   // evicted blocks are in place before the host reads them
        else e = hipStreamWaitEvent(cs, c->flush_ev, 0);     // ... before the DMA reads them
    }
    for (size_t k = 0; k < nch && e == hipSuccess; ++k) {
        const int b = (int)(k & 1);
        const size_t j0 = g.chunk_first[k], j1 = g.chunk_first[k + 1];
        e = hipStreamWaitEvent(cs, c->consumed[b], 0);   // the kernels that read buffer b are done
        if (e != hipSuccess) break;
        if (gather) {
            // gather the selected blocks into staging b (one memcpy each, on
            // several threads) and send them as one contiguous DMA per ~8 MB
            // piece, so that the gather of the next piece overlaps this DMA
            e = hipEventSynchronize(c->staged[b]);
            if (e == hipSuccess && !c->hgather[b])   // pinned on first use
                e = hipHostMalloc((void **)&c->hgather[b], (size_t)sp_pingpong(c) * sb, hipHostMallocDefault);
            const size_t piece = std::max<size_t>(1, (8u << 20) / sb);
            for (size_t p0 = j0; p0 < j1 && e == hipSuccess; p0 += piece) {
                const size_t p1 = std::min(j1, p0 + piece);
                parallel_tasks((int)(p1 - p0), gather_threads(), [&](int t) {
                    memcpy(c->hgather[b] + (int64_t)(p0 - j0 + t) * c->slot_elems,
                           load_slot_ptr(c, g.pieces[p0 + t].slot), sb);
                });
                e = hipMemcpyAsync(c->pingpong[b] + (int64_t)(p0 - j0) * c->slot_elems,
                                   c->hgather[b] + (int64_t)(p0 - j0) * c->slot_elems, (p1 - p0) * sb,
                                   hipMemcpyHostToDevice, cs);
            }
            if (e == hipSuccess) e = hipEventRecord(c->staged[b], cs);
        } else {
            // one DMA per run of consecutive slots of one arena
            for (size_t j = j0; j < j1 && e == hipSuccess;) {
                size_t r = j + 1;
                while (r < j1 && g.pieces[r].slot == g.pieces[r - 1].slot + 1 &&
                       g.pieces[r].slot % arena_blocks(c) != 0)
                    ++r;
                e = hipMemcpyAsync(c->pingpong[b] + (int64_t)(j - j0) * c->slot_elems,
                                   load_slot_ptr(c, g.pieces[j].slot), (r - j) * sb, hipMemcpyHostToDevice, cs);
                j = r;
            }
        }
        c->h2d_bytes += (int64_t)((j1 - j0) * sb);
        if (e == hipSuccess) e = hipEventRecord(c->filled[b], cs);
        if (e == hipSuccess) e = hipStreamWaitEvent(st, c->filled[b], 0);
        if (e != hipSuccess) break;
        RowLaunch &rl = g.chunks[k];
        rl.pool = c->pingpong[b];
        rl.table = c->dident;
        rl.table_stride = 1;
        e = launch_rows(c, rl, n, q, part_o, part_lse, st);
        if (e == hipSuccess) e = hipEventRecord(c->consumed[b], st);
    }
    if (e == hipSuccess && pass2) e = launch_combine_all(c, n, g.pb, part_o, part_lse, o_x, lse_x, o, lse, st);
    if (e != hipSuccess) return hip_fail(e, "GPU-side attention");
    return WSK_OK;
}

}  // namespace

extern "C" {

int wsk_attend_gpu_workspace(const wsk_cache *c, int32_t n, const int32_t *ids, size_t *bytes) {
    if (!bytes) return fail(WSK_EINVAL, "bytes is NULL");
    GpuPlan g;
    int rc = plan_dense(c, n, ids, g);
    if (rc) return rc;
    *bytes = g.bytes;
    return WSK_OK;
}

int wsk_attend_gpu(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, const float *o_x, const float *lse_x,
                   float *o, float *lse, void *ws, size_t ws_bytes, void *stream) {
    GpuPlan g;
    int rc = plan_dense(c, n, ids, g);
    if (rc) return rc;
    return run_plan(c, n, g, false, q, o_x, lse_x, o, lse, ws, ws_bytes, stream);
}

int wsk_attend_gpu_pass1(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, void *ws, size_t ws_bytes,
                         void *stream) {
    GpuPlan g;
    int rc = plan_dense(c, n, ids, g);
    if (rc) return rc;
    return run_plan(c, n, g, false, q, nullptr, nullptr, nullptr, nullptr, ws, ws_bytes, stream, true, false);
}

int wsk_attend_gpu_pass2(wsk_cache *c, int32_t n, const int32_t *ids, const float *o_x, const float *lse_x, float *o,
                         float *lse, void *ws, size_t ws_bytes, void *stream) {
    GpuPlan g;
    int rc = plan_dense(c, n, ids, g);
    if (rc) return rc;
    return run_plan(c, n, g, false, nullptr, o_x, lse_x, o, lse, ws, ws_bytes, stream, false, true);
}

int wsk_decode_step_workspace(const wsk_cache *c, int32_t n, const int32_t *ids, size_t *bytes) {
    if (!bytes) return fail(WSK_EINVAL, "bytes is NULL");
    GpuPlan g;
    int rc = plan_dense(c, n, ids, g, c && c->spec.kind == WSK_KIND_GQA);
    if (rc) return rc;
    *bytes = g.bytes;
    return WSK_OK;
}

}  // extern "C"

namespace {

// The output expansion a decode step may fold into its pass 2 (MLA).
struct StepExpand {
    const uint16_t *w_uv;
    int32_t dv;
    float *o;   // expanded output; the step's o (the latent output) may then be NULL
};

int decode_step(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, const void *k_new, const void *v_new,
                const float *o_x, const float *lse_x, float *o, float *lse, void *ws, size_t ws_bytes, void *stream,
                const StepExpand *ex) {
    int rc = check_ids(c, n, ids);
    if (rc) return rc;
    if (n == 0) return fail(WSK_EINVAL, "n must be positive");
    const wsk_partition_spec &sp = c->spec;
    const bool gqa = sp.kind == WSK_KIND_GQA;
    if (!k_new || (gqa && !v_new) || (!gqa && v_new)) return fail(WSK_EINVAL, "k_new / v_new");
    if (!aligned16(k_new) || !aligned16(v_new)) return fail(WSK_EINVAL, "k_new/v_new must be 16-byte aligned");
    std::vector<int32_t> sorted(ids, ids + n);
    std::sort(sorted.begin(), sorted.end());
    for (int32_t j = 1; j < n; ++j)
        if (sorted[j] == sorted[j - 1]) return fail(WSK_EINVAL, "sequence %d listed twice", sorted[j]);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t sq = ids[i];
        if (c->length[sq] >= sp.max_seq_len) return fail(WSK_ERANGE, "sequence %d is full", sq);
        if (c->length[sq] < std::max(c->split[sq], c->load_end[sq]))
            return fail(WSK_ERANGE, "position %d of sequence %d is below the start of its GPU pool range",
                        c->length[sq], sq);
    }
    // pass 1 covers the positions written so far; the new row joins in pass 2
    GpuPlan g;
    rc = plan_dense(c, n, ids, g, gqa);
    if (rc) return rc;
    rc = check_run(c, g, q, o_x, lse_x, ex ? ex->o : o, lse, ws, ws_bytes, true, true);
    if (rc) return rc;
    if (ex && !aligned16(o)) return fail(WSK_EINVAL, "o_lat must be 16-byte aligned");
    // routing of the new rows (as wsk_append)
    std::vector<Pending> pend;
    for (int32_t j = 0; j < n; ++j) {
        rc = plan(c, sorted[j], c->length[sorted[j]], 1, pend);
        if (rc) return rc;
    }
    // pass 1 reads only positions routed before this call; the new routes are
    // committed, and the lengths bumped, once both passes are enqueued, so a
    // failed launch leaves the cache as it was (pass 2 writes a new block's
    // device table entry, and a later step that routes the block again sends
    // it again)
    // The slot and row of each sequence's new position (launch-local r of
    // the launch that starts at call row i0), and the device table entry of
    // a block the step opens.
    auto place = [&](int32_t i0, int32_t m, int64_t *slot_elem0, int32_t *row, int32_t *tab_index,
                     int32_t *tab_slot) {
        for (int32_t r = 0; r < m; ++r) {
            const int32_t sq = ids[i0 + r];
            const int32_t pos = c->length[sq];
            const int32_t blk = pos / sp.block_tokens;
            int32_t slot = tab(c, WSK_PART_GPU, sq, blk);
            tab_index[r] = -1;
            for (const Pending &pd : pend)
                if (pd.seq == sq && pd.part == WSK_PART_GPU && pd.blk == blk) {
                    slot = pd.slot;
                    tab_index[r] = (int32_t)((size_t)sq * c->max_blocks + blk);
                    tab_slot[r] = pd.slot;
                }
            slot_elem0[r] = (int64_t)slot * c->slot_elems;
            row[r] = pos % sp.block_tokens;
        }
    };
    const int hkv = gqa ? sp.n_kv_heads : 1;
    const int width = gqa ? kHeadDim : kLatent;
    const int re = c->row_elems;
    float *part_o = (float *)ws;
    float *part_lse = (float *)((char *)ws + g.part_o_bytes);
    if (gqa && g.chunks.empty()) {
        // one launch per (up to) kMaxLaunchSeqs sequences: pass 1 with pass 2
        // in the last workgroup of each (sequence, KV head, head group)
        DeviceGuard guard(c->device);
        hipError_t e = guard.err;
        g.hbm.pool = c->dpool;
        g.hbm.table = c->dtab;
        g.hbm.table_stride = c->max_blocks;
        for (int32_t i0 = 0; i0 < n && e == hipSuccess; i0 += kMaxLaunchSeqs) {
            const int32_t m = std::min(kMaxLaunchSeqs, n - i0);
            AttendParams ap;
            const int n_wg = fill_attend(c, g.hbm, i0, m, q, part_o, part_lse, ap);
            StepTail t{};
            t.done = c->dstep_done;
            t.o = o + (int64_t)i0 * sp.n_q_heads * width;
            t.lse = lse + (int64_t)i0 * sp.n_q_heads;
            t.o_x = o_x ? o_x + (int64_t)i0 * sp.n_q_heads * width : nullptr;
            t.lse_x = lse_x ? lse_x + (int64_t)i0 * sp.n_q_heads : nullptr;
            t.k_new = (const uint16_t *)k_new + (int64_t)i0 * hkv * re;
            t.v_new = (const uint16_t *)v_new + (int64_t)i0 * hkv * re;
            t.pool = c->dpool;
            t.table = c->dtab;
            t.scale = sp.softmax_scale;
            place(i0, m, t.slot_elem0, t.row, t.tab_index, t.tab_slot);
            e = launch_gqa_step(ap, t, g.hbm.plan.heads_per_wg, n_wg, (hipStream_t)stream);
        }
        if (e != hipSuccess) {
            undo(c, pend);
            return hip_fail(e, "wsk_decode_step");
        }
        commit(c, pend);
        for (int32_t i = 0; i < n; ++i) c->length[ids[i]] += 1;
        return WSK_OK;
    }
    rc = run_plan(c, n, g, false, q, nullptr, nullptr, nullptr, nullptr, ws, ws_bytes, stream, true, false);
    DeviceGuard guard(c->device);
    hipError_t e = guard.err;
    for (int32_t i0 = 0; i0 < n && !rc && e == hipSuccess; i0 += kMaxLaunchSeqs) {
        const int32_t m = std::min(kMaxLaunchSeqs, n - i0);
        StepCombineParams p{};
        CombineParams &cp = p.cp;
        cp.part_o = part_o + g.pb[i0] * sp.n_q_heads * width;
        cp.part_lse = part_lse + g.pb[i0] * sp.n_q_heads;
        cp.o = o ? o + (int64_t)i0 * sp.n_q_heads * width : nullptr;
        cp.lse = lse + (int64_t)i0 * sp.n_q_heads;
        cp.o_x = o_x ? o_x + (int64_t)i0 * sp.n_q_heads * width : nullptr;
        cp.lse_x = lse_x ? lse_x + (int64_t)i0 * sp.n_q_heads : nullptr;
        cp.n = m;
        cp.n_q_heads = sp.n_q_heads;
        for (int32_t r = 0; r <= kMaxLaunchSeqs; ++r) cp.chunk_begin[r] = (int32_t)(g.pb[i0 + std::min(r, m)] - g.pb[i0]);
        p.q_row = (int64_t)sp.n_q_heads * re;
        p.q = (const uint16_t *)q + (int64_t)i0 * p.q_row;
        p.k_new = (const uint16_t *)k_new + (int64_t)i0 * hkv * re;
        p.v_new = v_new ? (const uint16_t *)v_new + (int64_t)i0 * hkv * re : nullptr;
        p.pool = c->dpool;
        p.table = c->dtab;
        p.kind = sp.kind;
        p.n_kv_heads = hkv;
        p.group = sp.n_q_heads / hkv;
        p.row_elems = re;
        p.block_tokens = sp.block_tokens;
        p.scale = sp.softmax_scale;
        place(i0, m, p.slot_elem0, p.row, p.tab_index, p.tab_slot);
        if (ex) {
            StepExpandParams xp{};
            xp.sc = p;
            xp.w_uv = ex->w_uv;
            xp.o = ex->o + (int64_t)i0 * sp.n_q_heads * ex->dv;
            xp.dv = ex->dv;
            // split each (sequence, head) over up to 4 workgroups of >= 32
            // output columns while the grid still fits the compute units
            const int64_t rows = (int64_t)m * sp.n_q_heads;
            int slices = 1;
            while (slices < 4 && rows * slices * 2 <= c->cu_count && ex->dv / (slices * 2) >= 32) slices *= 2;
            e = launch_step_expand(xp, slices, (hipStream_t)stream);
        } else {
            e = launch_step_combine(p, width, (hipStream_t)stream);
        }
    }
    if (rc || e != hipSuccess) {
        undo(c, pend);
        return rc ? rc : hip_fail(e, ex ? "wsk_decode_step_mla" : "wsk_decode_step");
    }
    commit(c, pend);
    for (int32_t i = 0; i < n; ++i) c->length[ids[i]] += 1;
    return WSK_OK;
}

}  // namespace

extern "C" {

int wsk_decode_step(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, const void *k_new, const void *v_new,
                    const float *o_x, const float *lse_x, float *o, float *lse, void *ws, size_t ws_bytes,
                    void *stream) {
    return decode_step(c, n, ids, q, k_new, v_new, o_x, lse_x, o, lse, ws, ws_bytes, stream, nullptr);
}

int wsk_decode_step_mla(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, const void *k_new,
                        const float *o_x, const float *lse_x, const uint16_t *w_uv, int32_t dv, float *o_lat,
                        float *lse, float *o, void *ws, size_t ws_bytes, void *stream) {
    if (!c) return fail(WSK_EINVAL, "cache is NULL");
    if (c->spec.kind != WSK_KIND_MLA) return fail(WSK_EINVAL, "wsk_decode_step_mla needs an MLA cache");
    if (dv != 64 && dv != 128 && dv != 256) return fail(WSK_EINVAL, "dv %d: supported 64, 128, 256", dv);
    if (!w_uv || !aligned16(w_uv)) return fail(WSK_EINVAL, "w_uv must be non-NULL and 16-byte aligned");
    if (!o) return fail(WSK_EINVAL, "o must not be NULL");
    const StepExpand ex{w_uv, dv, o};
    return decode_step(c, n, ids, q, k_new, nullptr, o_x, lse_x, o_lat, lse, ws, ws_bytes, stream, &ex);
}

int wsk_attend_blocks_workspace(const wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *sel_begin,
                                const int32_t *sel, size_t *bytes) {
    if (!bytes) return fail(WSK_EINVAL, "bytes is NULL");
    GpuPlan g;
    int rc = plan_selection(c, n, ids, sel_begin, sel, g);
    if (rc) return rc;
    *bytes = g.bytes;
    return WSK_OK;
}

int wsk_attend_blocks(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *sel_begin, const int32_t *sel,
                      const void *q, const float *o_x, const float *lse_x, float *o, float *lse, void *ws,
                      size_t ws_bytes, void *stream) {
    GpuPlan g;
    int rc = plan_selection(c, n, ids, sel_begin, sel, g);
    if (rc) return rc;
    return run_plan(c, n, g, true, q, o_x, lse_x, o, lse, ws, ws_bytes, stream);
}

int wsk_flush(wsk_cache *c, int32_t n, const int32_t *ids, const int32_t *part, int32_t *moved, void *stream) {
    int rc = check_ids(c, n, ids);
    if (rc) return rc;
    if (n > 0 && !part) return fail(WSK_EINVAL, "part is NULL");
    const int32_t D = c->spec.evict_tokens;
    if (D <= 0) return fail(WSK_ESTATE, "the cache has no eviction batch (evict_tokens = 0)");
    if (c->device < 0) return fail(WSK_ESTATE, "host-only cache");
    std::vector<int32_t> sorted(ids, ids + n);
    std::sort(sorted.begin(), sorted.end());
    for (int32_t j = 1; j < n; ++j)
        if (sorted[j] == sorted[j - 1]) return fail(WSK_EINVAL, "sequence %d listed twice", sorted[j]);
    for (int32_t i = 0; i < n; ++i) {
        if (part[i] != WSK_PART_CPU && part[i] != WSK_PART_LOAD) return fail(WSK_EINVAL, "part[%d] = %d", i, part[i]);
        if (part[i] == WSK_PART_LOAD && !has_load_region(c)) return fail(WSK_ESTATE, "the cache has no load region");
    }
    const int bk = c->spec.block_tokens;
    // batches and their destination slots (all-or-nothing); slots are taken in
    // ascending sequence id, whatever order the call lists the sequences in
    std::vector<int32_t> order(n);
    for (int32_t i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return ids[a] < ids[b]; });
    std::vector<int32_t> w0(n), w1(n);
    std::vector<Pending> pend;
    for (const int32_t i : order) {
        const int32_t sq = ids[i];
        w0[i] = c->window[sq];
        w1[i] = (w0[i] + D) / bk * bk;
        if (w1[i] > c->length[sq]) {
            w1[i] = w0[i];
            continue;
        }
        for (int32_t blk = w0[i] / bk; blk < w1[i] / bk; ++blk) {
            if (tab(c, part[i], sq, blk) >= 0) continue;   // the CPU slot of the block holding s
            if (c->free_slots[part[i]].empty()) {
                undo(c, pend);
                return fail(WSK_ENOMEM, "%s pool exhausted", part[i] == WSK_PART_CPU ? "CPU" : "load");
            }
            pend.push_back({part[i], sq, blk, c->free_slots[part[i]].top()});
            c->free_slots[part[i]].pop();
        }
    }
    rc = load_ensure(c, pend);
    if (rc) {
        undo(c, pend);
        return rc;
    }
    DeviceGuard guard(c->device);
    if (guard.err != hipSuccess) {
        undo(c, pend);
        return hip_fail(guard.err, "hipSetDevice");
    }
    commit(c, pend);
    hipStream_t st = (hipStream_t)stream;
    const size_t sb = slot_bytes(c);
    hipError_t e = hipSuccess;
    // the evicted blocks: destination slot, GPU-pool slot, first row held
    // (rows below it belong to the CPU side of the block holding s)
    struct Mv {
        int32_t dst, src, lo;
    };
    std::vector<Mv> to_load, to_cpu;
    for (int32_t i = 0; i < n; ++i)
        for (int32_t blk = w0[i] / bk; blk < w1[i] / bk; ++blk) {
            const Mv m{tab(c, part[i], ids[i], blk), tab(c, WSK_PART_GPU, ids[i], blk), std::max(w0[i] - blk * bk, 0)};
            (part[i] == WSK_PART_LOAD ? to_load : to_cpu).push_back(m);
        }
    const auto by_dst = [](const Mv &x, const Mv &y) { return x.dst < y.dst; };
    std::sort(to_load.begin(), to_load.end(), by_dst);
    std::sort(to_cpu.begin(), to_cpu.end(), by_dst);
    // blocks gathered per round into the device staging buffer, in
    // destination order (one kernel for all of them, HBM-resident slots are
    // scattered), then sent device -> host
    const size_t cap = evict_round_blocks(c);
    // blocks j0 .. j0 + m - 1 of v, one after another from dst (the device
    // staging buffer, or pinned host memory mapped for the device)
    const auto gather = [&](const std::vector<Mv> &v, size_t j0, size_t m, bool rows, uint16_t *dst) {
        EvictParams ep{};
        ep.pool = c->dpool;
        ep.stage = dst;
        ep.slot_elems = c->slot_elems;
        ep.m = (int32_t)m;
        ep.kind = c->spec.kind;
        ep.n_kv_heads = c->spec.kind == WSK_KIND_GQA ? c->spec.n_kv_heads : 1;
        ep.block_tokens = bk;
        ep.row_elems = c->row_elems;
        ep.to_rows = rows;
        for (size_t k = 0; k < m; ++k) ep.src_slot[k] = v[j0 + k].src;
        return launch_evict(ep, st);
    };
    // to the load region (same slot layout), per run of consecutive load
    // slots of one arena: the gather kernel stores the run straight into the
    // pinned slots over the link when the arena is mapped for the device;
    // else it gathers into the device staging buffer and one DMA per run
    // follows.  (A copy launched after the kernel leaves the link idle for
    // tens of microseconds first.)
    for (size_t j0 = 0; j0 < to_load.size() && e == hipSuccess; j0 += cap) {
        const size_t m = std::min(cap, to_load.size() - j0);
        bool all_mapped = true;
        for (size_t j = 0; j < m; ++j) all_mapped &= c->arena_mapped[to_load[j0 + j].dst / arena_blocks(c)] != 0;
        if (!all_mapped) e = gather(to_load, j0, m, false, c->dstage);
        for (size_t j = 0; j < m && e == hipSuccess;) {
            size_t r = j + 1;
            while (r < m && to_load[j0 + r].dst == to_load[j0 + r - 1].dst + 1 &&
                   to_load[j0 + r].dst % arena_blocks(c) != 0)
                ++r;
            uint16_t *slot = load_slot_ptr(c, to_load[j0 + j].dst);
            if (all_mapped)
                e = gather(to_load, j0 + j, r - j, false, slot);
            else
                e = hipMemcpyAsync(slot, c->dstage + (int64_t)j * c->slot_elems, (r - j) * sb, hipMemcpyDeviceToHost,
                                   st);
            c->d2h_bytes += (int64_t)((r - j) * sb);
            j = r;
        }
    }
    if (!to_load.empty() && e == hipSuccess) e = hipEventRecord(c->flush_ev, st);
    // to the CPU pool: rewritten into its token-major rows by the same
    // kernel and sent into the pinned bounce in pieces of ~2 MB, each piece's
    // rows copied into their slots on the host's threads as soon as it has
    // landed, while the next pieces are still on the link
    if (!to_cpu.empty() && e == hipSuccess) {
        const size_t bytes = std::min(cap, to_cpu.size()) * sb;
        if (c->hbounce_bytes < bytes) {   // more blocks than one batch of every sequence
            if (c->hbounce) (void)hipHostFree(c->hbounce);
            c->hbounce = nullptr;
            c->hbounce_bytes = 0;
            e = hipHostMalloc((void **)&c->hbounce, bytes, hipHostMallocDefault);
            if (e == hipSuccess) c->hbounce_bytes = bytes;
            c->bounce_mapped = e == hipSuccess && device_maps(c->hbounce);
        }
        const bool mla = c->spec.kind == WSK_KIND_MLA;
        const int runs = mla ? 1 : 2 * c->spec.n_kv_heads;   // (head, K | V) row runs per slot
        const size_t n_ev = sizeof(c->bounce_ev) / sizeof(c->bounce_ev[0]);
        for (size_t j0 = 0; j0 < to_cpu.size() && e == hipSuccess; j0 += cap) {
            const size_t m = std::min(cap, to_cpu.size() - j0);
            const size_t per = std::max((m + n_ev - 1) / n_ev, std::max<size_t>(1, (2u << 20) / sb));
            // the rows go straight into the bounce, a kernel per piece, when
            // it is mapped for the device; else through the device staging
            // buffer and one DMA per piece
            const bool direct = c->bounce_mapped;
            if (!direct) e = gather(to_cpu, j0, m, true, c->dstage);
            size_t pieces = 0;
            for (size_t a = 0; a < m && e == hipSuccess; a += per, ++pieces) {
                const size_t k = std::min(per, m - a);
                if (direct)
                    e = gather(to_cpu, j0 + a, k, true, c->hbounce + (int64_t)a * c->slot_elems);
                else
                    e = hipMemcpyAsync(c->hbounce + (int64_t)a * c->slot_elems, c->dstage + (int64_t)a * c->slot_elems,
                                       k * sb, hipMemcpyDeviceToHost, st);
                if (e == hipSuccess) e = hipEventRecord(c->bounce_ev[pieces], st);
            }
            // one parallel region for the round: the tasks are the blocks in
            // bounce order, and each waits for its piece's event first
            std::atomic<int> bad{0};
            if (e == hipSuccess)
                parallel_tasks((int)m, gather_threads(), [&](int t) {
                    if (hipEventSynchronize(c->bounce_ev[t / per]) != hipSuccess) {
                        bad = 1;
                        return;
                    }
                    const Mv &mv = to_cpu[j0 + t];
                    const int64_t off = (int64_t)mv.lo * c->row_elems, len = (int64_t)(bk - mv.lo) * c->row_elems;
                    for (int r = 0; r < runs; ++r) {
                        const int64_t base = (int64_t)r * bk * c->row_elems + off;
                        memcpy(c->hpool + (int64_t)mv.dst * c->slot_elems + base,
                               c->hbounce + (int64_t)t * c->slot_elems + base, (size_t)len * 2);
                    }
                });
            if (e == hipSuccess && bad) e = hipErrorUnknown;
            if (e == hipSuccess) c->d2h_bytes += (int64_t)(m * sb);
        }
    }
    // the batch now lives in its new home: free the GPU-pool slots, extend
    // the segments, move the window
    for (int32_t i = 0; i < n; ++i) {
        if (moved) moved[i] = w1[i] - w0[i];
        if (w1[i] == w0[i]) continue;
        const int32_t sq = ids[i];
        for (int32_t blk = w0[i] / bk; blk < w1[i] / bk; ++blk) {
            int32_t &t = tab(c, WSK_PART_GPU, sq, blk);
            c->free_slots[WSK_PART_GPU].push(t);
            t = -1;
        }
        std::vector<Seg> &sg = c->segs[sq];
        if (!sg.empty() && sg.back().part == part[i] && sg.back().e == w0[i])
            sg.back().e = w1[i];
        else
            sg.push_back({w0[i], w1[i], part[i]});
        c->window[sq] = w1[i];
    }
    if (e != hipSuccess) return hip_fail(e, "wsk_flush");
    return WSK_OK;
}

int wsk_cpu_attend_all(wsk_cache *c, int32_t n, const int32_t *ids, const void *q, float *o, float *lse,
                       int32_t threads) {
    int rc = check_ids(c, n, ids);
    if (rc) return rc;
    if (n == 0) return WSK_OK;
    if (!q || !o || !lse) return fail(WSK_EINVAL, "NULL argument");
    std::vector<const int32_t *> tables(n);
    std::vector<int32_t> rbegin(n + 1, 0), ra, re;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t sq = ids[i], L = c->length[sq];
        for (const Seg &s : c->segs[sq])
            if (s.part == WSK_PART_CPU && s.a < L) {
                ra.push_back(s.a);
                re.push_back(std::min(s.e, L));
            }
        rbegin[i + 1] = (int32_t)ra.size();
        tables[i] = c->htab[WSK_PART_CPU].data() + (size_t)sq * c->max_blocks;
    }
    const wsk_partition_spec &sp = c->spec;
    const bool mla = sp.kind == WSK_KIND_MLA;
    CpuAttendArgs x{};
    x.pool = c->hpool;
    x.tables = tables.data();
    x.start = ra.data();
    x.end = re.data();
    x.rbegin = rbegin.data();
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

int wsk_seq_segments(const wsk_cache *c, int32_t seq, int32_t cap, int32_t *start, int32_t *end, int32_t *part,
                     int32_t *count) {
    int rc = check_seq(c, seq);
    if (rc) return rc;
    if (!count || cap < 0 || (cap > 0 && (!start || !end || !part))) return fail(WSK_EINVAL, "output arrays");
    const int32_t L = c->length[seq];
    int32_t k = 0;
    auto emit = [&](int32_t a, int32_t e, int32_t p) {
        if (a >= e) return;
        if (k < cap) {
            start[k] = a;
            end[k] = e;
            part[k] = p;
        }
        ++k;
    };
    for (const Seg &s : c->segs[seq]) emit(s.a, std::min(s.e, L), s.part);
    emit(std::min(c->window[seq], L), L, WSK_PART_GPU);
    *count = k;
    return WSK_OK;
}

int wsk_load_slot(const wsk_cache *c, int32_t slot, const void **ptr) {
    if (!c || !ptr) return fail(WSK_EINVAL, "NULL argument");
    if (!has_load_region(c) || slot < 0 || slot >= c->spec.load_pool_blocks)
        return fail(WSK_ERANGE, "load slot %d", slot);
    if (!c->arenas[slot / arena_blocks(c)]) return fail(WSK_ERANGE, "load slot %d is not allocated", slot);
    *ptr = load_slot_ptr(c, slot);
    return WSK_OK;
}

int wsk_load_stats(const wsk_cache *c, wsk_load_info *out) {
    if (!c || !out) return fail(WSK_EINVAL, "NULL argument");
    memset(out, 0, sizeof *out);
    out->pinned_bytes = c->pinned_bytes;
    out->pin_seconds = c->pin_seconds;
    out->slots_used = has_load_region(c) ? c->spec.load_pool_blocks - (int64_t)c->free_slots[WSK_PART_LOAD].size() : 0;
    out->h2d_bytes = c->h2d_bytes;
    out->d2h_bytes = c->d2h_bytes;
    for (uint16_t *a : c->arenas) out->arenas += a != nullptr;
    return WSK_OK;
}

}  // extern "C"
