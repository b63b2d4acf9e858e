// Internal state of a partitioned KV cache and the helpers its two host
// sources share: wsk_host.cpp (spec, allocator, writes, range attention) and
// load.cpp (the pinned load region, ping-pong streaming, eviction).  Not part
// of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <functional>
#include <queue>
#include <vector>

#include "../../include/wsk.h"
#include "wsk_internal.h"

namespace wsk {

typedef std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> MinHeap;

// Bytes of device staging used by wsk_write for the GPU partition's rows.
constexpr size_t kStageBytes = 64u << 20;

// Positions [a, e) of one sequence placed in one home (WSK_PART_CPU or
// WSK_PART_LOAD); a sequence's segments cover [0, window) in order.
struct Seg {
    int32_t a, e, part;
};

// One slot taken from a pool and not yet entered in a table.
struct Pending {
    int part;
    int32_t seq;
    int32_t blk;
    int32_t slot;
};

}  // namespace wsk

struct wsk_cache {
    wsk_partition_spec spec;
    int device = -1;
    int cu_count = 256;           // compute units of the device (MI355X: 256)
    int32_t max_blocks = 0;       // logical blocks per sequence
    int32_t row_elems = 0;        // bf16 elements of one cached row (one head's K, or one MLA row)
    int32_t rows_per_pos = 0;     // rows one position stores (GQA: 2 * Hkv; MLA: 1)
    int64_t slot_elems = 0;       // bf16 elements per slot
    uint16_t *hpool = nullptr;    // CPU partition pool (pageable, 64-byte aligned)
    uint16_t *dpool = nullptr;    // GPU partition pool (HBM)
    int32_t *dtab = nullptr;      // device copy of the GPU block table
    uint16_t *dstage = nullptr;   // device staging for wsk_write
    uint32_t *dstep_done = nullptr; // GQA decode step: arrival counters [kMaxLaunchSeqs][n_q_heads], zero between launches
    int32_t *hsel = nullptr;      // pinned host staging of block-selection tables
    size_t hsel_bytes = 0;
    hipEvent_t hsel_ev = nullptr; // marks the end of the last selection-table upload
    std::vector<int32_t> htab[3]; // host block tables [part][seq * max_blocks + k]
    std::vector<uint8_t> is_open;
    std::vector<int32_t> split;     // s: positions [0, s) are written to the CPU pool
    std::vector<int32_t> load_end;  // positions [s, load_end) are written to the load region
    std::vector<int32_t> window;    // positions [window, length) are in the GPU pool (the D-window)
    std::vector<int32_t> length;
    std::vector<std::vector<wsk::Seg>> segs;   // homes of [0, window), in order
    wsk::MinHeap free_slots[3];

    // ---- load region (pinned host, GPU slot layout) and its streaming ----
    std::vector<uint16_t *> arenas;       // arena k holds slots [k * A, (k + 1) * A)
    std::vector<uint8_t> arena_mapped;    // arena k is mapped for the device at its host address
    int64_t pinned_bytes = 0;
    double pin_seconds = 0.0;
    int32_t *dident = nullptr;            // device identity table 0 .. pingpong_blocks - 1
    uint16_t *pingpong[2] = {nullptr, nullptr};
    hipStream_t copy_stream = nullptr;    // H2D of the load region
    hipEvent_t filled[2] = {nullptr, nullptr};     // ping-pong buffer b holds its chunk
    hipEvent_t consumed[2] = {nullptr, nullptr};   // the kernels reading buffer b are done
    hipEvent_t staged[2] = {nullptr, nullptr};     // the DMA out of gather staging b is done
    hipEvent_t flush_ev = nullptr;        // end of the last eviction into the load region
    uint16_t *hgather[2] = {nullptr, nullptr};     // pinned gather staging (sparse selections), on first use
    uint16_t *hbounce = nullptr;          // pinned bounce of evictions into the CPU pool
    size_t hbounce_bytes = 0;
    hipEvent_t bounce_ev[8] = {};         // pieces of one eviction round landed in the bounce
    bool bounce_mapped = false;           // the bounce is mapped for the device at its host address
    int64_t h2d_bytes = 0, d2h_bytes = 0; // load-region traffic since init
};

namespace wsk {

// Sets the calling thread's error message; returns code.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int hip_fail(hipError_t e, const char *what);

// Makes the cache's device current for the duration of a call and restores
// the caller's device afterwards.
struct DeviceGuard {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int dev) {
        if (dev < 0) return;
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) err = hipSetDevice(dev);
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

int check_seq(const wsk_cache *c, int32_t seq);

// Device address of wsk_decode_step_noalloc's scratch array on `device`,
// resolved once per device (noalloc.hip).
int noalloc_scratch(int device, void **out);

inline int32_t &tab(wsk_cache *c, int part, int32_t seq, int32_t blk) {
    return c->htab[part][(size_t)seq * c->max_blocks + blk];
}
inline int32_t tab(const wsk_cache *c, int part, int32_t seq, int32_t blk) {
    return c->htab[part][(size_t)seq * c->max_blocks + blk];
}

// Device buffers read or written with 16-byte vector accesses must be
// 16-byte aligned.
inline bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

inline bool has_load_region(const wsk_cache *c) { return c->spec.load_pool_blocks > 0; }
inline size_t slot_bytes(const wsk_cache *c) { return (size_t)c->slot_elems * 2; }

// Slot allocation (write-time routing).  plan() takes the lowest free slot
// of each pool a write of positions [pos0, pos0 + n) touches for the first
// time; commit() enters them in the tables, undo() returns them.
int plan(wsk_cache *c, int32_t seq, int32_t pos0, int32_t n, std::vector<Pending> &pend);
void commit(wsk_cache *c, const std::vector<Pending> &pend);
void undo(wsk_cache *c, const std::vector<Pending> &pend);
// Offset (elements) of position pos, KV head g, K (which = 0) or V (1), in
// its slot of the CPU pool, where every row is token-major.
inline int64_t row_offset(const wsk_cache *c, int32_t pos, int g, int which) {
    const int bk = c->spec.block_tokens;
    const int off = pos % bk;
    if (c->spec.kind == WSK_KIND_MLA) return (int64_t)off * c->row_elems;
    return ((int64_t)(g * 2 + which) * bk + off) * c->row_elems;
}

// Home (WSK_PART_*) of a written position.
int home_of(const wsk_cache *c, int32_t seq, int32_t pos);
// Whether every position of [a, e) is written and has home part.
bool range_in(const wsk_cache *c, int32_t seq, int32_t a, int32_t e, int part);

// Split-KV chunking of one pass-1 launch family: chunks are whole 64-token
// tiles of each range's tile grid; each range gets chunks in proportion to
// its tiles so that the grid is about one round of resident workgroups.
struct AttendPlan {
    int heads_per_wg = 1;
    int head_groups = 1;
    std::vector<int32_t> tpc;       // tiles per chunk, per sequence (per-sequence chunks)
    std::vector<int32_t> nchunks;   // partials per sequence
    // the flat split (GQA), per launch of kMaxLaunchSeqs sequences: the
    // sequence's first flat position within its launch, the first
    // workgroup that reads it; per launch: its flat positions and its
    // workgroups per unit (0: per-sequence chunks)
    std::vector<int32_t> flat_first, wfirst, launch_tiles, launch_wgs;
    int64_t partials = 0;           // sum of nchunks
    size_t part_o_bytes = 0;
    size_t bytes = 0;
};
inline int64_t n_tiles(int32_t a, int32_t e) { return e > a ? (int64_t)((e - 1) / kTile - a / kTile + 1) : 0; }
// min_one: every range gets at least one chunk, an empty range an empty
// chunk (a decode step's pass 2 runs in the workgroups of its pass 1).
void plan_chunks(const wsk_cache *c, int32_t n, const int32_t *start, const int32_t *end, AttendPlan &pl,
                 bool min_one = false);

// Fills the launch-invariant fields of AttendParams (strides, head counts,
// scale) for this cache.
void attend_params(const wsk_cache *c, const AttendPlan &pl, AttendParams &ap);

// One family of pass-1 launches over the n sequences of a call (query row i
// of the call is sequence i): sequence i reads row trow[i] of table (stride
// table_stride, slots of pool) over the range [start[i], end[i]) of that
// row's tile grid, and writes its plan.nchunks[i] partials at partial
// indices pbase[i], pbase[i] + 1, ...
struct RowLaunch {
    const uint16_t *pool = nullptr;
    const int32_t *table = nullptr;
    int32_t table_stride = 0;
    std::vector<int32_t> trow, start, end;
    AttendPlan plan;
    std::vector<int64_t> pbase;
};
hipError_t launch_rows(const wsk_cache *c, const RowLaunch &rl, int32_t n, const void *q, float *part_o,
                       float *part_lse, hipStream_t st);
// The pass-1 parameters of call rows i0 .. i0 + m - 1 (m <= kMaxLaunchSeqs)
// of rl; returns the launch's workgroup count.
int fill_attend(const wsk_cache *c, const RowLaunch &rl, int32_t i0, int32_t m, const void *q, float *part_o,
                float *part_lse, AttendParams &ap);
// Pass 2: merges partials [pb[i], pb[i + 1]) of every sequence i (and, if
// given, o_x / lse_x as one more partial) into o / lse.
hipError_t launch_combine_all(const wsk_cache *c, int32_t n, const std::vector<int64_t> &pb, const float *part_o,
                              const float *part_lse, const float *o_x, const float *lse_x, float *o, float *lse,
                              hipStream_t st);
// Argument checks shared by the attention entry points.
int check_outputs(const void *q, const float *o, const float *lse, const float *o_x, const float *lse_x, bool pass1,
                  bool pass2);

// Load region (load.cpp).
uint16_t *load_slot_ptr(const wsk_cache *c, int32_t slot);
int load_ensure(wsk_cache *c, const std::vector<Pending> &pend);   // pins the arenas new slots fall in
int load_init(wsk_cache *c);                                       // ping-pong, streams, events
int evict_init(wsk_cache *c);                                      // bounce of evictions to the CPU pool
void load_destroy(wsk_cache *c);
// Copies positions [p0, p1) of the host rows (layout as wsk_write's k/v,
// row 0 = position pos0) into their load-region slots (GPU slot layout).
void load_write_rows(wsk_cache *c, int32_t seq, int32_t pos0, int32_t p0, int32_t p1, const uint16_t *k,
                     const uint16_t *v);

}  // namespace wsk
