// Internal declarations shared by the host library (wsk_host.cpp) and the
// HIP kernels.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <functional>

namespace wsk {

// Sequences handled by one kernel launch; a call with more is split.
constexpr int kMaxLaunchSeqs = 64;
// What starting one more range costs a GQA pass-1 workgroup (the query
// load, the refill of its load pipeline, one more partial and, in a decode
// step, one more arrival), in tiles of streaming: the flat split's gap
// before each range.
constexpr int kSegmentTiles = 8;
// Tokens per attention tile: one token per lane of a 64-wide wavefront.
constexpr int kTile = 64;
// GQA key/value width.
constexpr int kHeadDim = 128;
// MLA latent and RoPE widths.
constexpr int kLatent = 512;
constexpr int kRope = 64;
// Cache policy of loads that stream KV rows read once per step: non-temporal
// (gfx950 "nt"), so they do not displace reusable lines in L2 and the
// Infinity Cache.
constexpr int kStreamLoad = 2;

// ---------------------------------------------------------------------------
// Split-KV attention (pass 1).  Sequence i attends positions [start, end) on
// the absolute 64-token tile grid; every workgroup writes a normalised
// partial O and its LSE per (sequence it reads, head) into part_o /
// part_lse, sequence i's partials numbered from chunk_begin[i].
//   Per-sequence chunks (flat_wgs == 0): workgroup (sequence i, chunk c,
//   unit u) reads tpc[i] tiles from the sequence's first + c * tpc[i], for
//   partial chunk_begin[i] + c; sequence i's workgroups are
//   [wg_begin[i], wg_begin[i + 1]), unit fastest.
//   The flat split (GQA, flat_wgs > 0): the launch's tiles in sequence order,
//   sequence i's from flat position flat_begin[i] (after a gap of
//   kSegmentTiles), flat_begin[n] positions in all, are cut into flat_wgs
//   equal runs per (KV head, head group) unit; workgroup w * units + u reads
//   run w for unit u, one segment per sequence it crosses, and writes
//   partial chunk_begin[i] + w - wfirst[i] of each.
// ---------------------------------------------------------------------------
struct AttendParams {
    const uint16_t *pool;    // device pool base (bf16)
    const int32_t *table;    // device block table [max_seqs][table_stride]
    const uint16_t *q;       // launch-local query rows: row i at q + i * q_row
    float *part_o;           // [partials][n_q_heads][width]
    float *part_lse;         // [partials][n_q_heads]
    int64_t slot_elems;      // bf16 elements per slot
    int64_t q_row;           // bf16 elements per query row (n_q_heads * q width)
    int32_t table_stride;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t group;           // query heads per KV head
    int32_t head_groups;     // workgroups per KV head along the query heads
    int32_t block_tokens;
    int32_t n;
    float scale_log2;        // softmax scale * log2(e)
    int32_t seq[kMaxLaunchSeqs];
    int32_t tpc[kMaxLaunchSeqs];   // tiles per chunk of each sequence
    int32_t start[kMaxLaunchSeqs];
    int32_t end[kMaxLaunchSeqs];
    int32_t wg_begin[kMaxLaunchSeqs + 1];
    int32_t chunk_begin[kMaxLaunchSeqs + 1];
    int32_t flat_begin[kMaxLaunchSeqs + 1];
    int32_t wfirst[kMaxLaunchSeqs];
    int32_t flat_wgs;
};

// A GQA decode step in one launch: pass 1 as AttendParams describes it, and
// the work of pass 2 (the chunk combine, the step's new token scored and
// merged, the merge of the CPU partial, the new row stored into the pool)
// done by the last workgroup of each (sequence, KV head, head group) to
// finish its chunk.  done[] counts those arrivals and is back at zero when
// the launch ends.
struct StepTail {
    uint32_t *done;          // [kMaxLaunchSeqs][units] arrival counters
    float *o;                // launch-local [n][n_q_heads][128]
    float *lse;              // launch-local [n][n_q_heads]
    const float *o_x;        // optional CPU partial, launch-local; NULL when absent
    const float *lse_x;
    const uint16_t *k_new;   // launch-local [n][n_kv_heads][128]
    const uint16_t *v_new;
    uint16_t *pool;
    int32_t *table;
    float scale;             // softmax scale (natural-log domain)
    int64_t slot_elem0[kMaxLaunchSeqs];
    int32_t row[kMaxLaunchSeqs];
    int32_t tab_index[kMaxLaunchSeqs];
    int32_t tab_slot[kMaxLaunchSeqs];
};

// Chunk combine (pass 2): merges the partials of each (sequence, head).
struct CombineParams {
    const float *part_o;
    const float *part_lse;
    float *o;                // launch-local [n][n_q_heads][width]
    float *lse;              // launch-local [n][n_q_heads]
    const float *o_x;        // optional partial over other keys (the CPU range), merged in
    const float *lse_x;      //   as one more chunk: launch-local [n][n_q_heads][width], [n][n_q_heads]
    int32_t n;
    int32_t n_q_heads;
    int32_t chunk_begin[kMaxLaunchSeqs + 1];
};

// Pass 2 of a decode step run as its own launch (a GQA step that streams
// load-region blocks; the MLA step's step_expand_kernel): the chunk combine,
// plus the step's new token of every sequence taken straight from its input
// row (its score q.k_new and its value row enter as one more partial), plus
// the append of that row into the GPU pool (as AppendParams describes it).
struct StepCombineParams {
    CombineParams cp;
    const uint16_t *q;       // launch-local query rows, q_row elements per sequence
    const uint16_t *k_new;   // launch-local new rows (GQA [n][n_kv_heads][128]; MLA [n][576])
    const uint16_t *v_new;   // GQA only
    uint16_t *pool;
    int32_t *table;
    int64_t q_row;
    int32_t kind;
    int32_t n_kv_heads;
    int32_t group;           // query heads per KV head (MLA: n_q_heads)
    int32_t row_elems;       // GQA: 128; MLA: 576
    int32_t block_tokens;
    float scale;             // softmax scale (natural-log domain)
    int64_t slot_elem0[kMaxLaunchSeqs];
    int32_t row[kMaxLaunchSeqs];
    int32_t tab_index[kMaxLaunchSeqs];
    int32_t tab_slot[kMaxLaunchSeqs];
};

// Pass 2 of an MLA decode step with the output expansion: sc as for
// step_combine (cp.o, the merged latent output, may be NULL), then
// o[i][h] = W_UV[h]^T O_lat[i][h] for every sequence and head.
struct StepExpandParams {
    StepCombineParams sc;
    const uint16_t *w_uv;    // bf16 [n_q_heads][512][dv]
    float *o;                // launch-local fp32 [n][n_q_heads][dv]
    int32_t dv;              // 64, 128 or 256
};

// Decode append: row r of the source goes to row row[r] of the slot whose
// first element is slot_elem0[r]; GQA rows carry K and V for every KV head
// (V stored transposed in the GPU pool).  tab_index[r] >= 0 also stores
// tab_slot[r] into the device table (a newly opened block).
struct AppendParams {
    const uint16_t *k_new;
    const uint16_t *v_new;   // GQA only
    uint16_t *pool;
    int32_t *table;
    int32_t n;
    int32_t kind;
    int32_t n_kv_heads;
    int32_t block_tokens;
    int32_t row_elems;       // GQA: head_dim; MLA: latent + rope
    int64_t slot_elem0[kMaxLaunchSeqs];
    int32_t row[kMaxLaunchSeqs];
    int32_t tab_index[kMaxLaunchSeqs];
    int32_t tab_slot[kMaxLaunchSeqs];
};

// Bulk scatter of staged rows [p0, p0 + m) of one sequence into its GPU
// partition, slots taken from the device table row.
struct ScatterParams {
    const uint16_t *src_k;   // staged [m][n_kv_heads][head_dim] or [m][row]
    const uint16_t *src_v;   // GQA only
    uint16_t *pool;
    const int32_t *table_row;
    int64_t slot_elems;
    int32_t p0;
    int32_t m;
    int32_t kind;
    int32_t n_kv_heads;
    int32_t block_tokens;
    int32_t row_elems;
};

// Eviction gather: copies whole GPU-pool slots src_slot[0 .. m) into a
// contiguous device staging buffer (slot j at j * slot_elems), either
// unchanged (to_rows = 0: the load region keeps the GPU slot layout) or
// rewritten into the CPU pool's token-major rows (to_rows = 1: GQA
// [n_kv_heads][K | V][block_tokens][128], MLA [block_tokens][576]).
constexpr int kEvictMax = 256;
struct EvictParams {
    const uint16_t *pool;
    uint16_t *stage;
    int64_t slot_elems;
    int32_t m;
    int32_t kind;
    int32_t n_kv_heads;
    int32_t block_tokens;
    int32_t row_elems;
    int32_t to_rows;
    int32_t src_slot[kEvictMax];
};

// In-place CPU attention over host-pool rows (cpu_attend.cpp).
struct CpuAttendArgs {
    const uint16_t *pool;          // host pool base
    const int32_t *const *tables;  // per sequence: its CPU block-table row
    const int32_t *start, *end;    // token ranges: per sequence, or per range when rbegin is set
    const int32_t *rbegin;         // optional [n + 1]: sequence i attends ranges rbegin[i] .. rbegin[i+1]-1
    const uint16_t *q;             // [n][n_q_heads][row_elems] bf16
    float *o;                      // [n][n_q_heads][dv]
    float *lse;                    // [n][n_q_heads]
    int64_t slot_elems;
    int64_t q_row;
    int n, n_q_heads, group;       // group: query heads per KV head (MLA: n_q_heads)
    int row_elems, dv, block_tokens;
    bool mla;
    float scale_log2;
    int threads;
};
int cpu_attend(const CpuAttendArgs &args);
// Runs task(0 .. n_tasks-1) on up to `threads` host threads (the calling one
// and the CPU engine's persistent pool); returns when all are done.
void parallel_tasks(int n_tasks, int threads, const std::function<void(int)> &task);
// Reads host memory [p, p + bytes) once on `threads` threads of that pool
// (bytes a multiple of 8) and returns the XOR of its 64-bit words.
uint64_t host_read(const void *p, size_t bytes, int threads);

// Sets the calling thread's last error message; returns code.
int policy_fail(int code, const char *msg);

hipError_t launch_gqa_attend(const AttendParams &p, int heads_per_wg, int n_wg, hipStream_t s);
hipError_t launch_gqa_step(const AttendParams &p, const StepTail &t, int heads_per_wg, int n_wg, hipStream_t s);
hipError_t launch_mla_attend(const AttendParams &p, int n_wg, hipStream_t s);
hipError_t launch_combine(const CombineParams &p, int width, hipStream_t s);
hipError_t launch_step_combine(const StepCombineParams &p, int width, hipStream_t s);
// slices: workgroups per (sequence, head), each expanding dv / slices columns
// (32, 64, 128 or 256 of them)
hipError_t launch_step_expand(const StepExpandParams &p, int slices, hipStream_t s);
hipError_t launch_append(const AppendParams &p, hipStream_t s);
hipError_t launch_scatter(const ScatterParams &p, hipStream_t s);
hipError_t launch_evict(const EvictParams &p, hipStream_t s);
hipError_t launch_merge(int32_t rows, int32_t width, const float *o_a, const float *lse_a,
                        const float *o_b, const float *lse_b, float *o_out, float *lse_out,
                        uint16_t *o_bf16, hipStream_t s);
hipError_t launch_stream_read(const void *p, int64_t bytes, uint32_t *out, int n_wg, hipStream_t s);
hipError_t launch_mla_absorb(int32_t n, int32_t H, int32_t dn, int32_t dl, const uint16_t *q_nope,
                             const uint16_t *w_uk, uint16_t *out, int64_t out_stride, hipStream_t s);
hipError_t launch_mla_expand(int32_t n, int32_t H, int32_t dl, int32_t dv, const float *o_lat,
                             const uint16_t *w_uv, float *o, hipStream_t s);

// Workgroups a GQA pass-1 grid aims at on a GPU with `cus` compute units:
// 3/4 per CU.  HBM reads with these 16-byte non-temporal loads peak with
// about that many 4-wavefront streams (MI355X, 2 GiB read: 192 workgroups
// 7.24 TB/s, 256 6.99, 512 6.81, 1024 6.33); more in flight lowers the rate.
inline int gqa_resident_slots(int cus) { return cus * 3 / 4; }

// Heads per workgroup used by the GQA kernel for a group size G: the largest
// power of two dividing G, at most 16 (the matrix-core tile height).
inline int gqa_heads_per_wg(int G) {
    for (int d = 16; d > 1; d >>= 1)
        if (G % d == 0) return d;
    return 1;
}

}  // namespace wsk
