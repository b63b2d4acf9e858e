// Small kernels of the decode path, gfx950: chunk combine, LSE merge, the
// decode step's pass 2 (GQA and MLA; the MLA form also expands by W_UV),
// decode append, bulk scatter, MLA query absorption and output expansion.

#include "device_rows.h"
#include "wsk_internal.h"

namespace wsk {
namespace {

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------------------
// Chunk combine: O = sum_c w_c O_c / sum_c w_c, w_c = exp(lse_c - max lse),
// LSE = max + ln sum w_c.  Workgroup = (sequence, head, 128-column slice);
// its 256 threads are 8 chunk groups x 32 float4 columns; the partials of
// the first 32 chunks are loaded together with every LSE before any is used,
// so up to 32 chunks cost one wait for memory; the groups are summed through
// LDS.  An optional partial over other keys (o_x, lse_x:
// the CPU range) enters as one more chunk, which makes this the LSE merge of
// the CPU and GPU partials too.  Nothing to merge: O = 0, LSE = -inf.
// ---------------------------------------------------------------------------
constexpr int kCombineCols4 = 32;                   // float4 columns per workgroup
constexpr int kCombineGroups = 256 / kCombineCols4; // chunk groups
constexpr int kCombineW = 1024;                     // chunk weights kept in LDS
constexpr int kCombineRegs = 4;                     // chunk partials per thread loaded up front

__device__ __forceinline__ float block_reduce(float v, bool is_max, float *s_red) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const float u = __shfl_xor(v, d);
        v = is_max ? fmaxf(v, u) : v + u;
    }
    __syncthreads();                                 // s_red free (earlier use finished)
    if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
    __syncthreads();
    float r = s_red[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) r = is_max ? fmaxf(r, s_red[w]) : r + s_red[w];
    return r;
}

// What one thread of a combine workgroup reads.  combine_load issues all of
// it at once -- the partials of the first kCombineGroups x kCombineRegs
// chunks, their LSEs, the other partial and the new token's value columns --
// so that the combine waits for memory once, not once per dependent step.
struct CombineIn {
    f32x4 po[kCombineRegs];   // chunk g + kCombineGroups j, this thread's float4 column
    f32x4 ox;                 // other partial's columns (chunk group 0)
    f32x4 vn;                 // new token's value columns (chunk group 0)
    float lse_c;              // LSE of chunk tid (tid < nc), else -inf
    float lx;                 // other partial's LSE
    int nc;
};

// v_new: the new token's value row (bf16) from this workgroup's first column,
// or NULL when there is none.
__device__ __forceinline__ CombineIn combine_load(const CombineParams &p, int width, const uint16_t *v_new) {
    const int row = blockIdx.x;                 // i * H + h
    const int H = p.n_q_heads;
    const int i = row / H;
    const int h = row - i * H;
    const int c0 = p.chunk_begin[i];
    const int tid = threadIdx.x;
    const int g = tid / kCombineCols4;
    const int c4 = tid - g * kCombineCols4;
    const int col0 = blockIdx.y * 4 * kCombineCols4;
    CombineIn in;
    in.nc = p.chunk_begin[i + 1] - c0;
    // loads that only some lanes need read a valid stand-in address (this
    // workgroup's own output row) in the others, whose values go unused: no
    // branch, so none waits for the loads issued before it
    const f32x4 *po = reinterpret_cast<const f32x4 *>(p.part_o + ((int64_t)c0 * H + h) * width + col0) + c4;
    const f32x4 *stand_in = reinterpret_cast<const f32x4 *>(p.o + (int64_t)row * width + col0) + c4;
    const int64_t cstride = (int64_t)H * width / 4;
#pragma unroll
    for (int j = 0; j < kCombineRegs; ++j) {
        const int c = g + kCombineGroups * j;
        in.po[j] = *(c < in.nc ? po + c * cstride : stand_in);
    }
    const float lse_r = *(tid < in.nc ? p.part_lse + (int64_t)(c0 + tid) * H + h : p.lse + row);
    in.lse_c = tid < in.nc ? lse_r : -INFINITY;
    in.lx = p.lse_x ? p.lse_x[row] : -INFINITY;
    // (used by the lanes of chunk group 0 only)
    in.ox = p.o_x ? reinterpret_cast<const f32x4 *>(p.o_x + (int64_t)row * width + col0)[c4] : f32x4{0.f, 0.f, 0.f, 0.f};
    in.vn = f32x4{0.f, 0.f, 0.f, 0.f};
    if (v_new) {
        const uint2 v2 = reinterpret_cast<const uint2 *>(v_new)[c4];
        in.vn = f32x4{__uint_as_float(v2.x << 16), __uint_as_float(v2.x & 0xffff0000u),
                      __uint_as_float(v2.y << 16), __uint_as_float(v2.y & 0xffff0000u)};
    }
    return in;
}

// One workgroup's part of the combine, from what combine_load read.  s_new:
// the score of an optional partial made of the single token whose value row
// combine_load was given (natural-log domain), -INFINITY when absent.
__device__ __forceinline__ void combine_finish(const CombineParams &p, int width, const CombineIn &in, float s_new,
                                               float *s_w, float *s_red, f32x4 (*s_acc)[kCombineCols4]) {
    const int row = blockIdx.x;
    const int H = p.n_q_heads;
    const int i = row / H;
    const int h = row - i * H;
    const int c0 = p.chunk_begin[i];
    const int nc = in.nc;
    const int tid = threadIdx.x;
    const int col0 = blockIdx.y * 4 * kCombineCols4;
    f32x4 *out = reinterpret_cast<f32x4 *>(p.o + (int64_t)row * width + col0);
    if (nc == 0 && in.lx == -INFINITY && s_new == -INFINITY) {
        if (tid < kCombineCols4) out[tid] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (tid == 0 && blockIdx.y == 0) p.lse[row] = -INFINITY;
        return;
    }
    const float *pl = p.part_lse + (int64_t)c0 * H + h;
    float m = fmaxf(fmaxf(in.lx, s_new), in.lse_c);
    for (int c = tid + 256; c < nc; c += 256) m = fmaxf(m, pl[(int64_t)c * H]);
    m = block_reduce(m, true, s_red);
    // the other partials' weights (0 when absent or empty; then their columns are not used)
    const float wx = in.lx == -INFINITY ? 0.f : __expf(in.lx - m);
    const float wn = s_new == -INFINITY ? 0.f : __expf(s_new - m);
    float dsum = tid == 0 ? wx + wn : 0.f;
    if (tid < nc) {
        const float w = __expf(in.lse_c - m);
        s_w[tid] = w;
        dsum += w;
    }
    for (int c = tid + 256; c < nc; c += 256) {
        const float w = __expf(pl[(int64_t)c * H] - m);
        if (c < kCombineW) s_w[c] = w;
        dsum += w;
    }
    const float den = block_reduce(dsum, false, s_red);   // its barriers also publish s_w
    const int g = tid / kCombineCols4;
    const int c4 = tid - g * kCombineCols4;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    if (g == 0 && wx != 0.f) acc = wx * in.ox;
    if (g == 0 && wn != 0.f) acc += wn * in.vn;
#pragma unroll
    for (int j = 0; j < kCombineRegs; ++j) {
        const int c = g + kCombineGroups * j;
        if (c < nc) acc += s_w[c] * in.po[j];
    }
    const f32x4 *po = reinterpret_cast<const f32x4 *>(p.part_o + ((int64_t)c0 * H + h) * width + col0) + c4;
    const int64_t cstride = (int64_t)H * width / 4;
#pragma unroll 8
    for (int c = g + kCombineGroups * kCombineRegs; c < nc; c += kCombineGroups) {
        const float w = c < kCombineW ? s_w[c] : __expf(pl[(int64_t)c * H] - m);
        acc += w * po[c * cstride];
    }
    s_acc[g][c4] = acc;
    __syncthreads();
    if (tid < kCombineCols4) {
        f32x4 t = s_acc[0][tid];
#pragma unroll
        for (int gg = 1; gg < kCombineGroups; ++gg) t += s_acc[gg][tid];
        out[tid] = t * (1.f / den);
    }
    if (tid == 0 && blockIdx.y == 0) p.lse[row] = m + __logf(den);
}

__global__ __launch_bounds__(256) void combine_kernel(const CombineParams p, int width) {
    __shared__ float s_w[kCombineW];
    __shared__ float s_red[4];
    __shared__ f32x4 s_acc[kCombineGroups][kCombineCols4];
    const CombineIn in = combine_load(p, width, nullptr);
    combine_finish(p, width, in, -INFINITY, s_w, s_red, s_acc);
}

// ---------------------------------------------------------------------------
// Pass 2 of a decode step run as two launches (GQA with load-region blocks
// streamed, MLA inside step_expand_kernel; a GQA step over HBM alone folds
// this into gqa_step_kernel).  Workgroup (sequence i, head h, column slice) as
// in combine_kernel; it also scores the step's new token against its query
// row (q . k_new, fp32 from bf16, the whole row, formed by each wavefront
// with shuffles), merges that token as one more partial, and -- in the
// workgroup of the first query head of each KV head and the first column
// slice -- stores the new row into the GPU pool (the decode append; the
// pass-1 kernels of this step did not read it).  The combine's loads, the
// dot product's and the new row's are issued before any is used; the row is
// stored after the combine.
// ---------------------------------------------------------------------------
// The two rows of a q . k product, as 16-byte pieces: lane l holds pieces l
// and l + 64 (zero past the row's re / 8; re <= 1024, the widest row here is
// MLA's 576).  Rows start 16-byte aligned.
struct RowPair {
    u32x4 q0, k0, q1, k1;
};
__device__ __forceinline__ RowPair load_row_pair(const uint16_t *q, const uint16_t *k, int re) {
    const int lane = threadIdx.x & 63;
    const int np = re / 8;
    const u32x4 *q16 = reinterpret_cast<const u32x4 *>(q), *k16 = reinterpret_cast<const u32x4 *>(k);
    RowPair r;
    r.q0 = r.k0 = r.q1 = r.k1 = u32x4{0u, 0u, 0u, 0u};
    if (lane < np) {
        r.q0 = q16[lane];
        r.k0 = k16[lane];
    }
    if (lane + 64 < np) {
        r.q1 = q16[lane + 64];
        r.k1 = k16[lane + 64];
    }
    return r;
}
// q . k in fp32 from the bf16 pieces, the same sum in every lane
__device__ __forceinline__ float row_dot(const RowPair &r) {
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        d = fmaf(__uint_as_float(r.q0[e] << 16), __uint_as_float(r.k0[e] << 16), d);
        d = fmaf(__uint_as_float(r.q0[e] & 0xffff0000u), __uint_as_float(r.k0[e] & 0xffff0000u), d);
        d = fmaf(__uint_as_float(r.q1[e] << 16), __uint_as_float(r.k1[e] << 16), d);
        d = fmaf(__uint_as_float(r.q1[e] & 0xffff0000u), __uint_as_float(r.k1[e] & 0xffff0000u), d);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) d += __shfl_xor(d, o);
    return d;
}

__global__ __launch_bounds__(256) void step_combine_kernel(const StepCombineParams sp, int width) {
    __shared__ float s_w[kCombineW];
    __shared__ float s_red[4];
    __shared__ f32x4 s_acc[kCombineGroups][kCombineCols4];
    const int H = sp.cp.n_q_heads;
    const int i = blockIdx.x / H;
    const int h = blockIdx.x - i * H;
    const int g = h / sp.group;
    const int tid = threadIdx.x;
    const int re = sp.row_elems;
    const bool gqa = sp.kind == 0;
    const uint16_t *kr = sp.k_new + (gqa ? ((int64_t)i * sp.n_kv_heads + g) * re : (int64_t)i * re);
    const uint16_t *qr = sp.q + (int64_t)i * sp.q_row + (int64_t)h * re;
    const uint16_t *vr = gqa ? sp.v_new + ((int64_t)i * sp.n_kv_heads + g) * re : kr;
    const CombineIn in = combine_load(sp.cp, width, vr + blockIdx.y * 4 * kCombineCols4);
    // the append of the new row: its 16-byte pieces are loaded here, with the
    // rest, and stored after the combine (off the combine's critical path)
    const bool append = blockIdx.y == 0 && h % sp.group == 0;
    const int row16 = re / 8;
    const int n_pieces = gqa ? 2 * row16 : row16;   // GQA: K then V pieces; MLA: the latent row
    const int which = gqa && tid >= row16 ? 1 : 0;
    const int piece = tid - which * row16;
    u32x4 pv = u32x4{0u, 0u, 0u, 0u};
    if (append && tid < n_pieces) pv = reinterpret_cast<const u32x4 *>(which ? vr : kr)[piece];
    // every wavefront forms the whole dot product (no barrier on this path)
    const float d = row_dot(load_row_pair(qr, kr, re));
    combine_finish(sp.cp, width, in, d * sp.scale, s_w, s_red, s_acc);
    if (append) {
        if (tid == 0 && h == 0 && sp.tab_index[i] >= 0) sp.table[sp.tab_index[i]] = sp.tab_slot[i];
        if (tid < n_pieces) {
            if (gqa)
                put_tiled(sp.pool + sp.slot_elem0[i] + (int64_t)g * 2 * sp.block_tokens * re, sp.row[i], which,
                          piece, pv);
            else
                put_mla32(sp.pool + sp.slot_elem0[i], sp.row[i], piece, pv);
        }
    }
}

// ---------------------------------------------------------------------------
// Pass 2 of an MLA decode step with the output expansion folded in (Sec. 6.1:
// the merged latent output is expanded by W_UV[h], which commutes with the
// merge).  Workgroup (sequence i, head h, slice y of DVS output columns)
// merges all 512 latent columns -- the chunk partials, the CPU partial and
// the step's new row, as step_combine_kernel does per 128-column slice -- and
// multiplies the merged row by columns [y DVS, (y + 1) DVS) of W_UV[h].  The
// slices of one (i, h) repeat the merge, which reads far less than W_UV[h]:
// slicing spreads the weight reads over more compute units when the batch
// leaves some idle.  Loads go out in the order they are used -- the merge's
// scalars, the chunk partials, the weights -- so the merge runs while the
// weights arrive; slice 0 stores the latent row and its LSE, and that of
// head 0 also stores the new row into the GPU pool.
// ---------------------------------------------------------------------------
constexpr int kSxThreads = 512;
constexpr int kSxWaves = kSxThreads / 64;
constexpr int kSxCols4 = kLatent / 4;               // 128 float4 columns
constexpr int kSxGroups = kSxThreads / kSxCols4;    // 4 chunk groups
constexpr int kSxRegs = 8;                          // chunk partials per thread loaded up front

__device__ __forceinline__ float sx_block_reduce(float v, bool is_max, float *s_red) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const float u = __shfl_xor(v, d);
        v = is_max ? fmaxf(v, u) : v + u;
    }
    __syncthreads();                                 // s_red free (earlier use finished)
    if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
    __syncthreads();
    float r = s_red[0];
#pragma unroll
    for (int w = 1; w < kSxWaves; ++w) r = is_max ? fmaxf(r, s_red[w]) : r + s_red[w];
    return r;
}

template <int DVS>
__global__ __launch_bounds__(kSxThreads) void step_expand_kernel(const StepExpandParams xp) {
    constexpr int kCg = DVS / 8;                     // 16-byte column groups of a W_UV row slice
    constexpr int kRg = kSxThreads / kCg;            // row groups
    constexpr int kRows = kLatent / kRg;             // W_UV rows per thread
    constexpr int kParts = kSxThreads / DVS;         // threads per output column in the final sum
    static_assert(kRg % kParts == 0 && kRg / kParts == 8, "each first-level sum adds 8 row groups");
    __shared__ float s_w[kCombineW];
    __shared__ float s_red[kSxWaves];
    __shared__ f32x4 s_acc[kSxGroups][kSxCols4];
    __shared__ float s_lat[kLatent];
    __shared__ float s_out[kRg][DVS];
    const StepCombineParams &sp = xp.sc;
    const CombineParams &p = sp.cp;
    const int H = p.n_q_heads;
    const int row = blockIdx.x;                      // i * H + h
    const int i = row / H;
    const int h = row - i * H;
    const int col0 = blockIdx.y * DVS;
    const bool lead = blockIdx.y == 0;               // stores the latent row, its LSE and the new row
    const int tid = threadIdx.x;
    const int re = sp.row_elems;                     // 576
    const uint16_t *kr = sp.k_new + (int64_t)i * re;
    const uint16_t *qr = sp.q + (int64_t)i * sp.q_row + (int64_t)h * re;

    // ---- loads, in the order they are used: the new row's score operands,
    //      chunk LSEs, CPU partial, new row; chunk partials; W_UV rows ----
    // (loads whose lanes differ in whether they are needed read a valid
    // stand-in address instead, and their values are then left unused: no
    // branch, so none waits for the loads issued before it)
    const RowPair qk = load_row_pair(qr, kr, re);
    const int c0 = p.chunk_begin[i];
    const int nc = p.chunk_begin[i + 1] - c0;
    const float lse_r = *(tid < nc ? p.part_lse + (int64_t)(c0 + tid) * H + h : p.lse + row);
    const float lse_c = tid < nc ? lse_r : -INFINITY;
    const float lx = p.lse_x ? p.lse_x[row] : -INFINITY;
    const int g = tid / kSxCols4;
    const int c4 = tid - g * kSxCols4;
    const f32x4 ox = p.o_x ? reinterpret_cast<const f32x4 *>(p.o_x + (int64_t)row * kLatent)[c4]
                           : f32x4{0.f, 0.f, 0.f, 0.f};
    const uint2 v2 = reinterpret_cast<const uint2 *>(kr)[c4];
    const f32x4 vn = f32x4{__uint_as_float(v2.x << 16), __uint_as_float(v2.x & 0xffff0000u),
                           __uint_as_float(v2.y << 16), __uint_as_float(v2.y & 0xffff0000u)};
    const bool append = lead && h == 0;
    const int n_pieces = re / 8;
    const u32x4 pv = reinterpret_cast<const u32x4 *>(kr)[min(tid, n_pieces - 1)];
    const f32x4 *po = reinterpret_cast<const f32x4 *>(p.part_o + ((int64_t)c0 * H + h) * kLatent) + c4;
    const f32x4 *stand_in = reinterpret_cast<const f32x4 *>(xp.w_uv);
    const int64_t cstride = (int64_t)H * kLatent / 4;
    f32x4 pr[kSxRegs];
#pragma unroll
    for (int j = 0; j < kSxRegs; ++j) {
        const int c = g + kSxGroups * j;
        pr[j] = *(c < nc ? po + c * cstride : stand_in);
    }
    const int rg = tid / kCg, cg = tid - (tid / kCg) * kCg;
    const uint16_t *wrow = xp.w_uv + (int64_t)h * kLatent * xp.dv + col0 + 8 * cg;
    u32x4 wv[kRows];
#pragma unroll
    for (int j = 0; j < kRows; ++j) wv[j] = *reinterpret_cast<const u32x4 *>(wrow + (int64_t)(rg + kRg * j) * xp.dv);

    // ---- the new row's score (every wavefront forms the whole dot product) ----
    const float s_new = row_dot(qk) * sp.scale;

    // ---- merge: O_lat = (sum_c w_c O_c + w_x O_x + w_n v_new) / sum w ----
    const float *pl = p.part_lse + (int64_t)c0 * H + h;
    float m = fmaxf(fmaxf(lx, s_new), lse_c);
    for (int c = tid + kSxThreads; c < nc; c += kSxThreads) m = fmaxf(m, pl[(int64_t)c * H]);
    m = sx_block_reduce(m, true, s_red);
    const bool empty = m == -INFINITY;               // nothing to merge: O = 0, LSE = -inf
    const float wx = lx == -INFINITY ? 0.f : __expf(lx - m);
    const float wn = s_new == -INFINITY ? 0.f : __expf(s_new - m);
    float dsum = tid == 0 ? wx + wn : 0.f;
    if (tid < nc) {
        const float w = __expf(lse_c - m);
        s_w[tid] = w;
        dsum += w;
    }
    for (int c = tid + kSxThreads; c < nc; c += kSxThreads) {
        const float w = __expf(pl[(int64_t)c * H] - m);
        if (c < kCombineW) s_w[c] = w;
        dsum += w;
    }
    const float den = sx_block_reduce(empty ? 0.f : dsum, false, s_red);   // its barriers also publish s_w
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    if (!empty) {
        if (g == 0 && wx != 0.f) acc = wx * ox;
        if (g == 0 && wn != 0.f) acc += wn * vn;
#pragma unroll
        for (int j = 0; j < kSxRegs; ++j) {
            const int c = g + kSxGroups * j;
            if (c < nc) acc += s_w[c] * pr[j];
        }
        for (int c = g + kSxGroups * kSxRegs; c < nc; c += kSxGroups) {
            const float w = c < kCombineW ? s_w[c] : __expf(pl[(int64_t)c * H] - m);
            acc += w * po[c * cstride];
        }
    }
    s_acc[g][c4] = acc;
    __syncthreads();
    if (tid < kSxCols4) {
        f32x4 t = s_acc[0][tid];
#pragma unroll
        for (int gg = 1; gg < kSxGroups; ++gg) t += s_acc[gg][tid];
        t = empty ? f32x4{0.f, 0.f, 0.f, 0.f} : t * (1.f / den);
        reinterpret_cast<f32x4 *>(s_lat)[tid] = t;
        if (lead && p.o) reinterpret_cast<f32x4 *>(p.o + (int64_t)row * kLatent)[tid] = t;
    }
    if (lead && tid == 0) p.lse[row] = empty ? -INFINITY : m + __logf(den);
    __syncthreads();

    // ---- O[i][h][col0 ..] = W_UV[h]^T O_lat: row group rg sums its rows for 8 columns ----
    float a8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
        const float x = s_lat[rg + kRg * j];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            a8[2 * e] = fmaf(x, __uint_as_float(wv[j][e] << 16), a8[2 * e]);
            a8[2 * e + 1] = fmaf(x, __uint_as_float(wv[j][e] & 0xffff0000u), a8[2 * e + 1]);
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) s_out[rg][8 * cg + e] = a8[e];
    __syncthreads();
    // the row groups' sums: 8 per thread into the first of them, then kParts per column
    {
        const int c = tid % DVS, q = tid / DVS;
        float t = s_out[8 * q][c];
#pragma unroll
        for (int r = 1; r < 8; ++r) t += s_out[8 * q + r][c];
        s_out[8 * q][c] = t;
    }
    __syncthreads();
    if (tid < DVS) {
        float t = s_out[0][tid];
#pragma unroll
        for (int q = 1; q < kParts; ++q) t += s_out[8 * q][tid];
        xp.o[(int64_t)row * xp.dv + col0 + tid] = t;
    }
    if (append) {
        if (tid == 0 && sp.tab_index[i] >= 0) sp.table[sp.tab_index[i]] = sp.tab_slot[i];
        if (tid < n_pieces) put_mla32(sp.pool + sp.slot_elem0[i], sp.row[i], tid, pv);
    }
}

// ---------------------------------------------------------------------------
// LSE merge of two partials.  A workgroup owns whole rows: thread t first
// reads the LSEs of row t into LDS and writes that row's merged LSE, so
// lse_out may alias lse_a or lse_b; O is then merged 4 elements per thread.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void merge_kernel(int32_t rows, int32_t width, int32_t rows_per_wg,
                                                    const float *o_a, const float *lse_a, const float *o_b,
                                                    const float *lse_b, float *o_out, float *lse_out,
                                                    uint16_t *o_bf16) {
    __shared__ float s_wa[256], s_wb[256];
    const int r0 = blockIdx.x * rows_per_wg;
    const int nr = min(rows_per_wg, rows - r0);
    if ((int)threadIdx.x < nr) {
        const int r = r0 + threadIdx.x;
        const float la = lse_a[r], lb = lse_b[r];
        const float m = fmaxf(la, lb);
        float wa = 0.f, wb = 0.f, lo = -INFINITY;
        if (m != -INFINITY) {
            wa = __expf(la - m);
            wb = __expf(lb - m);
            lo = m + __logf(wa + wb);
            const float inv = 1.f / (wa + wb);
            wa *= inv;
            wb *= inv;
        }
        s_wa[threadIdx.x] = wa;
        s_wb[threadIdx.x] = wb;
        lse_out[r] = lo;
    }
    __syncthreads();
    const int w4 = width / 4;
    for (int f = threadIdx.x; f < nr * w4; f += blockDim.x) {
        const int rr = f / w4;
        const int64_t e0 = (int64_t)(r0 + rr) * width + (int64_t)(f - rr * w4) * 4;
        const float wa = s_wa[rr], wb = s_wb[rr];
        f32x4 y = f32x4{0.f, 0.f, 0.f, 0.f};
        if (wa != 0.f || wb != 0.f) {
            // a side with zero weight is not read: an empty partial's O may be anything
            const f32x4 a = wa != 0.f ? *reinterpret_cast<const f32x4 *>(o_a + e0) : f32x4{0.f, 0.f, 0.f, 0.f};
            const f32x4 b = wb != 0.f ? *reinterpret_cast<const f32x4 *>(o_b + e0) : f32x4{0.f, 0.f, 0.f, 0.f};
            y = wa * a + wb * b;
        }
        *reinterpret_cast<f32x4 *>(o_out + e0) = y;
        if (o_bf16) {
            uint16_t *d = o_bf16 + e0;
            d[0] = f32_to_bf16(y.x);
            d[1] = f32_to_bf16(y.y);
            d[2] = f32_to_bf16(y.z);
            d[3] = f32_to_bf16(y.w);
        }
    }
}

// ---------------------------------------------------------------------------
// Decode append: one workgroup per appended row (all KV heads, K and V).
// GPU-pool rows go to the TILED64 (GQA) or MLA32 (MLA) format.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void append_kernel(const AppendParams p) {
    const int r = blockIdx.x;
    const int64_t slot0 = p.slot_elem0[r];
    const int row = p.row[r];
    if (threadIdx.x == 0 && p.tab_index[r] >= 0) p.table[p.tab_index[r]] = p.tab_slot[r];
    const int row16 = p.row_elems / 8;                 // 16-byte pieces per row
    const int bk = p.block_tokens;
    if (p.kind == 0) {
        const int pieces = p.n_kv_heads * row16;
        for (int t = threadIdx.x; t < 2 * pieces; t += blockDim.x) {
            const int which = t / pieces;              // 0 = K, 1 = V
            const int q = t - which * pieces;
            const int g = q / row16;
            const int k = q - g * row16;
            const uint16_t *src = (which ? p.v_new : p.k_new) + ((int64_t)r * p.n_kv_heads + g) * p.row_elems;
            uint16_t *head = p.pool + slot0 + (int64_t)g * 2 * bk * p.row_elems;
            put_tiled(head, row, which, k, reinterpret_cast<const u32x4 *>(src)[k]);
        }
    } else {
        const uint16_t *src = p.k_new + (int64_t)r * p.row_elems;
        for (int k = threadIdx.x; k < row16; k += blockDim.x)
            put_mla32(p.pool + slot0, row, k, reinterpret_cast<const u32x4 *>(src)[k]);
    }
}

// ---------------------------------------------------------------------------
// Bulk scatter of staged rows into the GPU partition (same slot layout).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void scatter_kernel(const ScatterParams p) {
    const int row16 = p.row_elems / 8;
    const int per_pos = (p.kind == 0) ? 2 * p.n_kv_heads * row16 : row16;
    const int64_t total = (int64_t)p.m * per_pos;
    const int bk = p.block_tokens;
    const int bshift = __builtin_ctz(bk);
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int j = (int)(t / per_pos);
        int q = (int)(t - (int64_t)j * per_pos);
        const int pos = p.p0 + j;
        const int blk = pos >> bshift;
        const int off = pos - (blk << bshift);
        const int64_t slot = p.table_row[blk];
        if (p.kind == 0) {
            const int which = q / (p.n_kv_heads * row16);
            q -= which * p.n_kv_heads * row16;
            const int g = q / row16;
            const int k = q - g * row16;
            const uint16_t *src = (which ? p.src_v : p.src_k) + ((int64_t)j * p.n_kv_heads + g) * p.row_elems;
            uint16_t *head = p.pool + slot * p.slot_elems + (int64_t)g * 2 * bk * p.row_elems;
            put_tiled(head, off, which, k, reinterpret_cast<const u32x4 *>(src)[k]);
        } else {
            const uint16_t *src = p.src_k + (int64_t)j * p.row_elems;
            put_mla32(p.pool + slot * p.slot_elems, off, q, reinterpret_cast<const u32x4 *>(src)[q]);
        }
    }
}

// ---------------------------------------------------------------------------
// Eviction gather: whole GPU-pool slots into contiguous staging, unchanged
// or as the CPU pool's token-major rows.  One 16-byte output piece per
// thread and step; the writes are coalesced, the reads stay inside one slot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void evict_kernel(const EvictParams p) {
    const int64_t units = p.slot_elems / 8;           // 16-byte pieces per slot
    const int64_t total = (int64_t)p.m * units;
    const int bk = p.block_tokens;
    const int row16 = p.row_elems / 8;
    for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += (int64_t)gridDim.x * blockDim.x) {
        const int j = (int)(u / units);
        const int64_t x = u - (int64_t)j * units;
        const uint16_t *src = p.pool + (int64_t)p.src_slot[j] * p.slot_elems;
        u32x4 v;
        if (!p.to_rows) {
            v = reinterpret_cast<const u32x4 *>(src)[x];
        } else if (p.kind == 1) {   // MLA: row r, piece c
            const int r = (int)(x / row16), c = (int)(x - (int64_t)r * row16);
            v = get_mla32(src, r, c);
        } else {                     // GQA: head g, K or V, row r, piece k
            const int per_head = 2 * bk * row16;
            const int g = (int)(x / per_head);
            int q = (int)(x - (int64_t)g * per_head);
            const int which = q / (bk * row16);
            q -= which * bk * row16;
            const int r = q / row16, k = q - r * row16;
            v = get_tiled(src + (int64_t)g * 2 * bk * p.row_elems, r, which, k);
        }
        reinterpret_cast<u32x4 *>(p.stage + (int64_t)j * p.slot_elems)[x] = v;
    }
}

// ---------------------------------------------------------------------------
// MLA absorption and expansion: per head, a batch of up to 8 token rows times
// a bf16 weight matrix, fp32 accumulation:
//   absorb  q_lat[i][h][l] = sum_k q_nope[i][h][k] W_UK[h][k][l]  (bf16 out, one rounding)
//   expand  o[i][h][j]     = sum_l o_lat[i][h][l]  W_UV[h][l][j]  (fp32 out)
// Workgroup = (head, CB output columns, 8 tokens); its 256 threads are CB/8
// column groups x (2048/CB) row slices, so each thread fetches its few weight
// rows (16-byte loads) in one round and the grid has 128-256 workgroups.  The
// inputs of the 8 tokens are staged in LDS; the row slices are summed through
// LDS in a fixed order.
// ---------------------------------------------------------------------------
constexpr int kProjTok = 8;

template <int CB, int KMAX, typename Tin, bool kBf16Out>
__global__ __launch_bounds__(256) void proj_kernel(int32_t n, int32_t H, int32_t K, int32_t C, const Tin *x,
                                                   const uint16_t *w, void *out, int64_t out_stride) {
    constexpr int CG = CB / 8;          // column groups of 8
    constexpr int SL = 256 / CG;        // row slices
    __shared__ float sx[kProjTok * KMAX];               // [kProjTok][K]
    __shared__ float red[SL * kProjTok * CB];           // [SL][kProjTok][CB], 64 KB
    const int h = blockIdx.x;
    const int cb = blockIdx.y * CB;
    const int i0 = blockIdx.z * kProjTok;
    const int nt = min(kProjTok, n - i0);
    const int cg = threadIdx.x % CG, sl = threadIdx.x / CG;
    const int col0 = cb + 8 * cg;
    const bool col_ok = col0 < C;
    const uint16_t *wc = w + (int64_t)h * K * C + col0;
    // this thread's first four weight rows, issued before anything waits
    u32x4 wv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int k = sl + q * SL;
        wv[q] = (col_ok && k < K) ? *reinterpret_cast<const u32x4 *>(wc + (int64_t)k * C) : u32x4{0u, 0u, 0u, 0u};
    }
    // the 8 tokens' input rows into LDS as fp32, 16 bytes per load where the
    // width allows; a thread's loads (at most kStage) are all issued before
    // the first is stored, so staging waits for memory once
    constexpr int kVec = 16 / sizeof(Tin);
    constexpr int kStage = (kProjTok * KMAX / kVec + 255) / 256;
    if (K % kVec == 0 && ((uintptr_t)x & 15) == 0) {
        const int nv = kProjTok * K / kVec;
        u32x4 raw[kStage];
#pragma unroll
        for (int r = 0; r < kStage; ++r) {
            const int t = threadIdx.x + 256 * r;
            const int e = t * kVec, ii = e / K, k = e - ii * K;
            raw[r] = (t < nv && ii < nt) ? *reinterpret_cast<const u32x4 *>(x + ((int64_t)(i0 + ii) * H + h) * K + k)
                                         : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int r = 0; r < kStage; ++r) {
            const int t = threadIdx.x + 256 * r;
            if (t < nv) {
#pragma unroll
                for (int j = 0; j < kVec; ++j) {
                    if constexpr (sizeof(Tin) == 2)
                        sx[t * kVec + j] = __uint_as_float((j & 1) ? (raw[r][j >> 1] & 0xffff0000u)
                                                                   : (raw[r][j >> 1] << 16));
                    else
                        sx[t * kVec + j] = __uint_as_float(raw[r][j]);
                }
            }
        }
    } else {
        for (int t = threadIdx.x; t < kProjTok * K; t += 256) {
            const int ii = t / K, k = t - ii * K;
            float v = 0.f;
            if (ii < nt) {
                const Tin xv = x[((int64_t)(i0 + ii) * H + h) * K + k];
                if constexpr (sizeof(Tin) == 2)
                    v = bf16_to_f32(xv);
                else
                    v = xv;
            }
            sx[t] = v;
        }
    }
    __syncthreads();
    float acc[kProjTok][8];
#pragma unroll
    for (int ii = 0; ii < kProjTok; ++ii)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[ii][c] = 0.f;
    auto fma_rows = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + q * SL;
            if (k >= K) break;
            float wf[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                wf[2 * e] = __uint_as_float(wv[q][e] << 16);
                wf[2 * e + 1] = __uint_as_float(wv[q][e] & 0xffff0000u);
            }
#pragma unroll
            for (int ii = 0; ii < kProjTok; ++ii) {
                const float xv = sx[ii * K + k];
#pragma unroll
                for (int c = 0; c < 8; ++c) acc[ii][c] = fmaf(xv, wf[c], acc[ii][c]);
            }
        }
    };
    fma_rows(sl);
    for (int k0 = sl + 4 * SL; k0 < K; k0 += 4 * SL) {   // rows beyond the first four (wide K only)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + q * SL;
            wv[q] = (col_ok && k < K) ? *reinterpret_cast<const u32x4 *>(wc + (int64_t)k * C)
                                      : u32x4{0u, 0u, 0u, 0u};
        }
        fma_rows(k0);
    }
#pragma unroll
    for (int ii = 0; ii < kProjTok; ++ii)
#pragma unroll
        for (int c = 0; c < 8; ++c) red[(sl * kProjTok + ii) * CB + 8 * cg + c] = acc[ii][c];
    __syncthreads();
    for (int t = threadIdx.x; t < kProjTok * CB; t += 256) {
        const int ii = t / CB, c = t - ii * CB;
        if (ii >= nt || cb + c >= C) continue;
        float part[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};   // 8 loads in flight
#pragma unroll
        for (int q = 0; q < SL; q += 8)
#pragma unroll
            for (int u = 0; u < 8; ++u) part[u] += red[((q + u) * kProjTok + ii) * CB + c];
        const float v = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
        const int64_t o = ((int64_t)(i0 + ii) * H + h) * out_stride + cb + c;
        if constexpr (kBf16Out)
            reinterpret_cast<uint16_t *>(out)[o] = f32_to_bf16(v);
        else
            reinterpret_cast<float *>(out)[o] = v;
    }
}

// ---------------------------------------------------------------------------
// Streaming read probe: every wavefront reads 32 KB tiles (32 loads of 1 KB
// in flight, non-temporal buffer loads like the attention kernels),
// grid-stride over the buffer, and folds them.
// ---------------------------------------------------------------------------
constexpr int kProbeTileBytes = 32768;

__global__ __launch_bounds__(256) void stream_read_kernel(const char *a, int64_t ntiles, uint32_t *out) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t acc = 0;
    for (int64_t t = (int64_t)blockIdx.x * 4 + wave; t < ntiles; t += (int64_t)gridDim.x * 4) {
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void *)(a + t * kProbeTileBytes), 0, kProbeTileBytes, 0x00020000);
        u32x4 v[kProbeTileBytes / 1024];
#pragma unroll
        for (int k = 0; k < kProbeTileBytes / 1024; ++k)
            v[k] = __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, k * 1024, kStreamLoad);
#pragma unroll
        for (int k = 0; k < kProbeTileBytes / 1024; ++k) acc ^= v[k][0] ^ v[k][1] ^ v[k][2] ^ v[k][3];
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) acc ^= __shfl_xor(acc, d);
    if (lane == 0) atomicXor(out, acc);
}

constexpr int kAbsorbCols = 32;   // 16 heads x 512 / 32 = 256 workgroups
constexpr int kExpandCols = 16;   // 16 heads x 128 / 16 = 128 workgroups

constexpr int kAbsorbMaxK = 256;  // q_nope width limit (wsk_mla_absorb)
constexpr int kExpandMaxK = 1024; // latent width limit (wsk_mla_expand)

}  // namespace

hipError_t launch_combine(const CombineParams &p, int width, hipStream_t s) {
    if (p.n <= 0) return hipSuccess;
    if (width <= 0 || width % (4 * kCombineCols4)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(combine_kernel, dim3(p.n * p.n_q_heads, width / (4 * kCombineCols4)), dim3(256), 0, s, p,
                       width);
    return hipGetLastError();
}

hipError_t launch_merge(int32_t rows, int32_t width, const float *o_a, const float *lse_a,
                        const float *o_b, const float *lse_b, float *o_out, float *lse_out,
                        uint16_t *o_bf16, hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    int rpw = 1024 / width;
    if (rpw < 1) rpw = 1;
    if (rpw > 256) rpw = 256;
    const int blocks = (rows + rpw - 1) / rpw;
    hipLaunchKernelGGL(merge_kernel, dim3(blocks), dim3(256), 0, s, rows, width, rpw, o_a, lse_a, o_b, lse_b,
                       o_out, lse_out, o_bf16);
    return hipGetLastError();
}

hipError_t launch_step_combine(const StepCombineParams &p, int width, hipStream_t s) {
    if (p.cp.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(step_combine_kernel, dim3(p.cp.n * p.cp.n_q_heads, width / (4 * kCombineCols4)), dim3(256),
                       0, s, p, width);
    return hipGetLastError();
}

hipError_t launch_step_expand(const StepExpandParams &p, int slices, hipStream_t s) {
    if (p.sc.cp.n <= 0) return hipSuccess;
    if (slices <= 0 || p.dv % slices) return hipErrorInvalidValue;
    const dim3 grid(p.sc.cp.n * p.sc.cp.n_q_heads, slices), block(kSxThreads);
    switch (p.dv / slices) {
        case 32: hipLaunchKernelGGL(step_expand_kernel<32>, grid, block, 0, s, p); break;
        case 64: hipLaunchKernelGGL(step_expand_kernel<64>, grid, block, 0, s, p); break;
        case 128: hipLaunchKernelGGL(step_expand_kernel<128>, grid, block, 0, s, p); break;
        case 256: hipLaunchKernelGGL(step_expand_kernel<256>, grid, block, 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_append(const AppendParams &p, hipStream_t s) {
    if (p.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(append_kernel, dim3(p.n), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_scatter(const ScatterParams &p, hipStream_t s) {
    if (p.m <= 0) return hipSuccess;
    const int row16 = p.row_elems / 8;
    const int64_t per_pos = (p.kind == 0) ? 2 * p.n_kv_heads * row16 : row16;
    int64_t blocks = ((int64_t)p.m * per_pos + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_evict(const EvictParams &p, hipStream_t s) {
    if (p.m <= 0) return hipSuccess;
    if (p.m > kEvictMax) return hipErrorInvalidValue;
    int64_t blocks = ((int64_t)p.m * (p.slot_elems / 8) + 255) / 256;
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL(evict_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_stream_read(const void *p, int64_t bytes, uint32_t *out, int n_wg, hipStream_t s) {
    hipLaunchKernelGGL(stream_read_kernel, dim3(n_wg), dim3(256), 0, s, (const char *)p, bytes / kProbeTileBytes, out);
    return hipGetLastError();
}

hipError_t launch_mla_absorb(int32_t n, int32_t H, int32_t dn, int32_t dl, const uint16_t *q_nope,
                             const uint16_t *w_uk, uint16_t *out, int64_t out_stride, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const dim3 grid(H, (dl + kAbsorbCols - 1) / kAbsorbCols, (n + kProjTok - 1) / kProjTok);
    hipLaunchKernelGGL((proj_kernel<kAbsorbCols, kAbsorbMaxK, uint16_t, true>), grid, dim3(256), 0, s, n, H, dn, dl,
                       q_nope, w_uk, (void *)out, out_stride);
    return hipGetLastError();
}

hipError_t launch_mla_expand(int32_t n, int32_t H, int32_t dl, int32_t dv, const float *o_lat,
                             const uint16_t *w_uv, float *o, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const dim3 grid(H, (dv + kExpandCols - 1) / kExpandCols, (n + kProjTok - 1) / kProjTok);
    hipLaunchKernelGGL((proj_kernel<kExpandCols, kExpandMaxK, float, false>), grid, dim3(256), 0, s, n, H, dl, dv,
                       o_lat, w_uv, (void *)o, (int64_t)dv);
    return hipGetLastError();
}

}  // namespace wsk
