// Split-KV decode attention over a GQA partition (pass 1), gfx950.
//
// For every query head served by one KV head, computes the exact softmax
// attention over one chunk of the sequence range (the GPU engine of
// Sec. 5.1) and writes the normalised partial output and its natural-log LSE
// (the partial result with its normaliser that Sec. 4.2 merges by LSE).
//
// The G query heads of a KV head share every K and V row, so both products
// are dense contractions and run on the matrix cores
// (v_mfma_f32_16x16x32_bf16, query heads padded to 16 rows):
//
//   S^T [64 tokens x 16 heads] = K [64 x 128] . Q^T [128 x 16]
//   O   [16 heads x 128]      += P [16 x 64]  . V [64 x 128]
//
// The GPU pool keeps each 64-token tile of a KV head as 2 x 1024 16-byte
// pieces in exactly the order the matrix-core lanes consume them (the
// TILED64 format, fixed when the rows are written): every operand load is
// one 16-byte load per lane and 1 KB contiguous per wavefront instruction.
//   - QK A-operand (mt, ks), lane (grp, n): K[token tile_token(mt, n)]
//     [dims 32ks + 8grp .. +8]
//   - P.V B-operand (nt, ks), lane (grp, n): V[tokens 32ks + 8grp .. +8]
//     [dim 16nt + n]
// tile_token() permutes the tokens of each QK M-tile so that the QK output of
// a lane already holds, per K-step of P.V, the 8 consecutive tokens its P
// A-operand needs: nothing moves between the two products.  P is split into
// bf16 hi + lo parts (two MFMAs), which keeps P.V accurate to ~2^-16
// relative, like fp32 probabilities.
//
// Work mapping: workgroup = (KV head, group of GH <= 16 query heads, a run
// of 64-token tiles): a chunk of one sequence (per-sequence chunks), or, for
// ragged batches, an equal share of the launch's tiles that may cross from
// one sequence into the next (the flat split: one partial per sequence it
// reads).  Its 4 wavefronts take every 4th tile of a run with their own
// online softmax and are merged through LDS at the end of each sequence's
// part.  Each wavefront issues the next tile's K loads as soon as QK has
// consumed the current ones, and the next V loads right after P.V.
//
// gqa_step_kernel is the same pass 1 with a decode step's pass 2 folded in
// (Sec. 4.2: one LSE join per step): every workgroup stores its partial
// device-coherent, waits for the stores and counts itself on a device-scope
// atomic; the last of each (sequence, KV head, head group) merges the chunk
// partials of its heads with the step's new token and the CPU partial and
// stores the new row into the pool.  The step then costs one launch instead
// of two, and no L2-wide fence.

#include "device_rows.h"

namespace wsk {
namespace {

constexpr int kWaves = 4;
constexpr int kTailW = 64;   // chunk weights per head the step's last workgroup keeps in LDS
constexpr int kTileBytes = 2 * kTile * kHeadDim * 2;   // K and V pieces of one 64-token tile: 32 KB

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Token (0..63) of row r (0..15) of QK M-tile mt (0..3).  Rows 4g..4g+3 of
// M-tiles 2k and 2k+1 are tokens 32k + 8g .. 32k + 8g + 7.
__device__ __forceinline__ int tile_token(int mt, int r) {
    return 32 * (mt >> 1) + 8 * (r >> 2) + 4 * (mt & 1) + (r & 3);
}

// A load that sees what another XCD stored device-coherent in this launch.
__device__ __forceinline__ float coherent_load(const float *a) {
    return __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// What pass 2 of a decode step reads besides the chunk partials, for heads
// h0 .. h0 + GH - 1 of launch-local sequence i (KV head g): loaded after a
// workgroup's last segment, before it is counted, so that these loads
// overlap the wait for its partial stores; only the last workgroup uses
// them.
template <int GH>
struct TailIn {
    static constexpr int kItems = (GH * 32 + 255) / 256;           // float4 output columns per thread
    static constexpr int kHeads = (GH + kWaves - 1) / kWaves;      // heads scored per wavefront
    uint32_t kw;                 // k_new[2 lane .. 2 lane + 1]
    uint32_t qw[kHeads];         // q of head wave + 4 k, same two dims
    float lx[kHeads];            // lse_x of that head
    uint2 vn[kItems];            // v_new columns 4 c4 .. 4 c4 + 3
    f32x4 ox[kItems];            // o_x of (head, column) item
    u32x4 piece;                 // 16-byte piece of the new K/V row this thread stores
};

template <int GH>
__device__ __forceinline__ TailIn<GH> tail_load(const AttendParams &p, const StepTail &t, int i, int g, int h0) {
    TailIn<GH> in;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int H = p.n_q_heads;
    const int64_t kv_row = ((int64_t)i * p.n_kv_heads + g) * kHeadDim;
    in.kw = reinterpret_cast<const uint32_t *>(t.k_new + kv_row)[lane];
#pragma unroll
    for (int k = 0; k < TailIn<GH>::kHeads; ++k) {
        const int hh = wave + kWaves * k;
        in.qw[k] = 0u;
        in.lx[k] = -INFINITY;
        if (hh < GH) {
            const int h = h0 + hh;
            in.qw[k] = reinterpret_cast<const uint32_t *>(p.q + (int64_t)i * p.q_row + (int64_t)h * kHeadDim)[lane];
            if (t.lse_x) in.lx[k] = t.lse_x[(int64_t)i * H + h];
        }
    }
#pragma unroll
    for (int j = 0; j < TailIn<GH>::kItems; ++j) {
        const int idx = threadIdx.x + 256 * j;
        in.vn[j] = uint2{0u, 0u};
        in.ox[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (idx < GH * 32) {
            const int hh = idx >> 5, c4 = idx & 31;
            in.vn[j] = reinterpret_cast<const uint2 *>(t.v_new + kv_row)[c4];
            if (t.o_x) in.ox[j] = reinterpret_cast<const f32x4 *>(t.o_x + ((int64_t)i * H + h0 + hh) * kHeadDim)[c4];
        }
    }
    in.piece = u32x4{0u, 0u, 0u, 0u};
    if (threadIdx.x < 32)
        in.piece = reinterpret_cast<const u32x4 *>((threadIdx.x >> 4 ? t.v_new : t.k_new) + kv_row)[threadIdx.x & 15];
    return in;
}

// Pass 2 of a decode step for heads h0 .. h0 + GH - 1 of launch-local
// sequence i (KV head g, head group hg), by the workgroup that finished the
// last of its nc chunk partials (partials pb .. pb + nc - 1, all visible).
// Same arithmetic as the separate pass-2 kernel: the new token enters as a
// partial of one key (score q . k_new * scale, value v_new), the CPU partial
// as one more; weights exp(lse - max), natural-log domain.  The first
// kTailRegs partials of every output column are loaded together with the
// LSEs, in one round trip.
constexpr int kTailRegs = 8;

template <int GH>
__device__ __forceinline__ void step_tail(const AttendParams &p, const StepTail &t, const TailIn<GH> &in, int i,
                                          int g, int hg, int h0, int nc, int pb) {
    __shared__ float s_w[GH][kTailW];
    __shared__ float s_sc[GH][4];   // per head: max, CPU-partial weight, new-token weight, 1 / normaliser
    constexpr int kItems = TailIn<GH>::kItems;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int H = p.n_q_heads;
    const float *po = p.part_o + ((int64_t)pb * H + h0) * kHeadDim;
    const int64_t cstride = (int64_t)H * kHeadDim;   // floats between chunks
    f32x4 pr[kItems][kTailRegs];
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int idx = threadIdx.x + 256 * j;
        const float *e0 = po + (int64_t)(idx >> 5) * kHeadDim + 4 * (idx & 31);
#pragma unroll
        for (int c = 0; c < kTailRegs; ++c) {
            pr[j][c] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (idx < GH * 32 && c < nc) {
                const float *e = e0 + c * cstride;
                pr[j][c] = f32x4{coherent_load(e), coherent_load(e + 1), coherent_load(e + 2), coherent_load(e + 3)};
            }
        }
    }
    // ---- per head: new-token score, maximum, weights, normaliser ----
#pragma unroll
    for (int k = 0; k < TailIn<GH>::kHeads; ++k) {
        const int hh = wave + kWaves * k;
        if (hh >= GH) break;
        const int64_t row = (int64_t)i * H + h0 + hh;
        const float *pl = p.part_lse + (int64_t)pb * H + h0 + hh;
        const float l0 = lane < nc ? coherent_load(pl + (int64_t)lane * H) : -INFINITY;
        const float lx = in.lx[k];
        const uint32_t qw = in.qw[k];
        float d = __uint_as_float(qw << 16) * __uint_as_float(in.kw << 16);
        d = fmaf(__uint_as_float(qw & 0xffff0000u), __uint_as_float(in.kw & 0xffff0000u), d);
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) d += __shfl_xor(d, o);
        const float s_new = d * t.scale;
        float m = fmaxf(fmaxf(s_new, lx), l0);
        for (int c = lane + 64; c < nc; c += 64) m = fmaxf(m, coherent_load(pl + (int64_t)c * H));
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
        float den = 0.f;
        if (lane < nc) {
            const float w = __expf(l0 - m);
            s_w[hh][lane] = w;
            den = w;
        }
        for (int c = lane + 64; c < nc; c += 64) den += __expf(coherent_load(pl + (int64_t)c * H) - m);
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) den += __shfl_xor(den, o);
        const float wx = lx == -INFINITY ? 0.f : __expf(lx - m);
        const float wn = __expf(s_new - m);
        den += wx + wn;
        if (lane == 0) {
            s_sc[hh][0] = m;
            s_sc[hh][1] = wx;
            s_sc[hh][2] = wn;
            s_sc[hh][3] = 1.f / den;
            t.lse[row] = m + __logf(den);
        }
    }
    __syncthreads();
    // ---- merged rows: 32 float4 columns per head ----
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int idx = threadIdx.x + 256 * j;
        if (idx >= GH * 32) break;
        const int hh = idx >> 5;
        const int c4 = idx & 31;
        const int64_t row = (int64_t)i * H + h0 + hh;
        const float m = s_sc[hh][0], wx = s_sc[hh][1], wn = s_sc[hh][2], inv = s_sc[hh][3];
        const uint2 v2 = in.vn[j];
        f32x4 acc = wn * f32x4{__uint_as_float(v2.x << 16), __uint_as_float(v2.x & 0xffff0000u),
                               __uint_as_float(v2.y << 16), __uint_as_float(v2.y & 0xffff0000u)};
        if (wx != 0.f) acc += wx * in.ox[j];
#pragma unroll
        for (int c = 0; c < kTailRegs; ++c)
            if (c < nc) acc += s_w[hh][c] * pr[j][c];
        // the rest, kTailRegs partials at a time, every load of a batch
        // issued before any is used
        const float *e0 = po + (int64_t)hh * kHeadDim + 4 * c4;
        for (int c0 = kTailRegs; c0 < nc; c0 += kTailRegs) {
            f32x4 b[kTailRegs];
            float wb[kTailRegs];
#pragma unroll
            for (int k = 0; k < kTailRegs; ++k) {
                const int c = c0 + k;
                b[k] = f32x4{0.f, 0.f, 0.f, 0.f};
                wb[k] = 0.f;
                if (c < nc) {
                    const float *e = e0 + c * cstride;
                    b[k] = f32x4{coherent_load(e), coherent_load(e + 1), coherent_load(e + 2), coherent_load(e + 3)};
                    wb[k] = c < kTailW ? s_w[hh][c]
                                       : __expf(coherent_load(p.part_lse + (int64_t)(pb + c) * H + h0 + hh) - m);
                }
            }
#pragma unroll
            for (int k = 0; k < kTailRegs; ++k) acc += wb[k] * b[k];
        }
        reinterpret_cast<f32x4 *>(t.o + row * kHeadDim)[c4] = acc * inv;
    }
    // ---- the new row into the pool (once per KV head: head group 0) ----
    // No workgroup of this KV head reads it this launch: the chunks of head
    // group 0 are done, and those of other head groups mask every position
    // at or past the step's start length.
    if (hg == 0 && threadIdx.x < 32)
        put_tiled(t.pool + t.slot_elem0[i] + (int64_t)g * 2 * p.block_tokens * kHeadDim, t.row[i], threadIdx.x >> 4,
                  threadIdx.x & 15, in.piece);
    if (hg == 0 && g == 0 && threadIdx.x == 0 && t.tab_index[i] >= 0) t.table[t.tab_index[i]] = t.tab_slot[i];
}

// Pass 1 over tiles [tile0, tile_end) of launch-local sequence i for query
// heads h0 .. h0 + GH - 1 of KV head g: writes partial `part` (an empty
// range writes a zero row of LSE -inf); device-coherent stores for a decode
// step, whose last workgroups read the partials back in the same launch.
template <int GH, bool STEP>
__device__ __forceinline__ void attend_segment(const AttendParams &p, int i, int g, int h0, int tile0, int tile_end,
                                               int part, float (*s_o)[GH][kHeadDim], float (*s_m)[GH],
                                               float (*s_l)[GH]) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;     // MFMA column: query head (QK) / dim within an N-tile (P.V)
    const int grp = lane >> 4;   // MFMA k-group 0..3

    const int seq = p.seq[i];
    const int t_start = p.start[i];
    const int t_end = p.end[i];
    typedef const __attribute__((address_space(4))) int32_t ci32;
    ci32 *trow = (ci32 *)(p.table + (int64_t)seq * p.table_stride);   // read-only here
    const int bk = p.block_tokens;
    const int bshift = __builtin_ctz(bk);
    const int64_t head_off = (int64_t)g * 2 * bk * kHeadDim;
    const int head_bytes = 2 * bk * kHeadDim * 2;     // all tiles of one head in one slot

    // Q^T operand (constant): lane (grp, n) holds q[h0 + n][32ks + 8grp .. +8]
    bf16x8 qop[4];
    {
        const u32x4 *qrow = reinterpret_cast<const u32x4 *>(p.q + (int64_t)i * p.q_row +
                                                            (int64_t)(h0 + (n < GH ? n : 0)) * kHeadDim);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const u32x4 v = qrow[ks * 4 + grp];
            qop[ks] = as_bf16x8(n < GH ? v : u32x4{0u, 0u, 0u, 0u});
        }
    }

    float m_run = -INFINITY;   // running max of head n (exp2 domain)
    float l_lane = 0.f;        // this lane's share of head n's normaliser
    f32x4 o[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Buffer descriptor over the tiles of KV head g in the slot holding tile
    // t; toff = byte offset of the tile inside it.  The descriptor's extent
    // bounds every load to that (slot, head).
    auto tile_rsrc = [&](int t, int &toff) -> __amdgpu_buffer_rsrc_t {
        const int tok0 = t * kTile;
        const int blk = tok0 >> bshift;
        toff = ((tok0 - (blk << bshift)) >> 6) * kTileBytes;
        const int slot = __builtin_amdgcn_readfirstlane(trow[blk]);
        // a missing table entry (< 0) gets an empty extent: its loads read
        // zeros instead of memory outside the pool
        const uint16_t *base = p.pool + (slot < 0 ? 0 : (int64_t)slot * p.slot_elems) + head_off;
        return __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, slot < 0 ? 0 : head_bytes, 0x00020000);
    };
    const int loff = lane * 16;
    u32x4 ka[4][4], vb[8][2];
    auto load_k = [&](int t) {
        int toff;
        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(t, toff);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                ka[mt][ks] = __builtin_amdgcn_raw_buffer_load_b128(rs, loff, toff + (mt * 4 + ks) * 1024, kStreamLoad);
    };
    auto load_v = [&](int t) {
        int toff;
        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(t, toff);
#pragma unroll
        for (int nt = 0; nt < 8; ++nt)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                vb[nt][ks] = __builtin_amdgcn_raw_buffer_load_b128(
                    rs, loff, toff + kTileBytes / 2 + (nt * 2 + ks) * 1024, kStreamLoad);
    };

    int t = tile0 + wave;
    if (t < tile_end) {
        load_k(t);
        load_v(t);
    }
    for (; t < tile_end; t += kWaves) {
        const int tok0 = t * kTile;
        const int tn = t + kWaves;

        // ---- QK on the matrix cores ----
        f32x4 s[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            s[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                s[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka[mt][ks]), qop[ks], s[mt], 0, 0, 0);
        }
        if (tn < tile_end) load_k(tn);

        // ---- online softmax (exp2 domain) for head n over this tile ----
        const bool partial = tok0 < t_start || tok0 + kTile > t_end;
        float sv[4][4];
        float mloc = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tok = tok0 + 32 * (mt >> 1) + 8 * grp + 4 * (mt & 1) + r;
                const bool ok = !partial || (tok >= t_start && tok < t_end);
                sv[mt][r] = ok ? s[mt][r] * p.scale_log2 : -INFINITY;
                mloc = fmaxf(mloc, sv[mt][r]);
            }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        const float m_new = fmaxf(m_run, mloc);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        float psum = 0.f;
        bf16x8 phi[2], plo[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float pv = __builtin_amdgcn_exp2f(sv[2 * ks + (j >> 2)][j & 3] - m_new);
                psum += pv;
                const __bf16 hi = (__bf16)pv;
                phi[ks][j] = hi;
                plo[ks][j] = (__bf16)(pv - (float)hi);
            }
        l_lane = fmaf(l_lane, alpha, psum);

        // rows of O are heads 4grp..4grp+3: fetch their rescale factors
        float alpha_r[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) alpha_r[r] = __shfl(alpha, 4 * grp + r);
#pragma unroll
        for (int nt = 0; nt < 8; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) o[nt][r] *= alpha_r[r];

        // rows outside [start, end) may hold anything (even NaN): zero their V
        if (partial) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                uint32_t mask[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int tk = tok0 + 32 * ks + 8 * grp + 2 * e;
                    mask[e] = ((tk >= t_start && tk < t_end) ? 0x0000ffffu : 0u) |
                              ((tk + 1 >= t_start && tk + 1 < t_end) ? 0xffff0000u : 0u);
                }
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) vb[nt][ks] &= u32x4{mask[0], mask[1], mask[2], mask[3]};
            }
        }

        // ---- P.V on the matrix cores ----
#pragma unroll
        for (int nt = 0; nt < 8; ++nt)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi[ks], as_bf16x8(vb[nt][ks]), o[nt], 0, 0, 0);
                o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo[ks], as_bf16x8(vb[nt][ks]), o[nt], 0, 0, 0);
            }
        if (tn < tile_end) load_v(tn);
    }

    // ---- merge the four wavefront states through LDS ----
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (grp == 0 && n < GH) {
        s_m[wave][n] = m_run;
        s_l[wave][n] = l_tot;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int h = 4 * grp + r;
        if (h < GH) {
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) s_o[wave][h][16 * nt + n] = o[nt][r];
        }
    }
    __syncthreads();

    for (int idx = threadIdx.x; idx < GH * kHeadDim; idx += 256) {
        const int h = idx / kHeadDim;
        const int d = idx - h * kHeadDim;
        float M = s_m[0][h];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
        float num = 0.f, den = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float a = __builtin_amdgcn_exp2f(s_m[w][h] - M);
            num = fmaf(a, s_o[w][h][d], num);
            den = fmaf(a, s_l[w][h], den);
        }
        const int64_t row = (int64_t)part * p.n_q_heads + h0 + h;
        // an empty chunk (a decode step's sequence with no GPU-pool
        // positions before the step) leaves a zero row of weight 0
        const bool any = den > 0.f;
        const float ov = any ? num / den : 0.f;
        const float lv = any ? (M + __log2f(den)) * 0.69314718055994530942f : -INFINITY;
        if constexpr (STEP) {
            // device-coherent stores: another XCD's workgroup reads them this launch
            __hip_atomic_store(p.part_o + row * kHeadDim + d, ov, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (d == 0) __hip_atomic_store(p.part_lse + row, lv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            p.part_o[row * kHeadDim + d] = ov;
            if (d == 0) p.part_lse[row] = lv;
        }
    }
}

// Arrival of a decode step's workgroup for sequence i, unit u, after its
// partial for them is stored.  The partials are stored device-coherent
// (written through the XCD's L2, which the other XCDs do not share); every
// wavefront waits until its stores are complete, and only then is the
// workgroup counted.  Returns whether it is the last arrival for the
// (sequence, unit), which then reads the partials with device-coherent
// loads and finishes pass 2.  No L2-wide writeback or invalidation: the
// other workgroups of the XCD keep streaming undisturbed.
__device__ __forceinline__ bool count_in(const AttendParams &p, const StepTail &t, int i, int u, int units) {
    __shared__ uint32_t s_last;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t *cnt = t.done + i * units + u;
        const uint32_t nc = p.chunk_begin[i + 1] - p.chunk_begin[i];
        const uint32_t prev = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const bool last = prev == nc - 1;
        // every arrival is in: reset for the next launch
        if (last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = last ? 1u : 0u;
    }
    __syncthreads();
    const bool last = s_last != 0u;
    __syncthreads();   // s_last is free again
    return last;
}

// Pass 2 for sequence i, unit u, by its last arrival (its inputs loaded in `in`).
template <int GH>
__device__ __forceinline__ void finish(const AttendParams &p, const StepTail &t, const TailIn<GH> &in, int i, int u) {
    const int g = u / p.head_groups;
    const int hg = u - g * p.head_groups;
    step_tail<GH>(p, t, in, i, g, hg, g * p.group + hg * GH, p.chunk_begin[i + 1] - p.chunk_begin[i],
                  p.chunk_begin[i]);
}

template <int GH>
__device__ __forceinline__ TailIn<GH> tail_inputs(const AttendParams &p, const StepTail &t, int i, int u) {
    const int g = u / p.head_groups;
    return tail_load<GH>(p, t, i, g, g * p.group + (u - g * p.head_groups) * GH);
}

// Tiles of launch-local sequence i's range.
__device__ __forceinline__ int seq_tiles(const AttendParams &p, int i) {
    return p.end[i] > p.start[i] ? ((p.end[i] - 1) >> 6) - (p.start[i] >> 6) + 1 : 0;
}

// One workgroup's work.  Per-sequence chunks (FLAT false): one segment,
// tiles [c tpc, (c + 1) tpc) of sequence i for unit u, partial
// chunk_begin[i] + c.  The flat split (FLAT true): workgroup w * units + u
// reads flat positions [lo, hi) of unit u, one segment per sequence they
// cross, in sequence order, each with its own partial
// chunk_begin[i] + w - wfirst[i]; an empty sequence of a decode step is an
// empty segment of the one workgroup wfirst names.  A decode step counts
// the workgroup in after each segment, so a workgroup that crosses into the
// next sequence has already arrived for the previous one.
template <int GH, bool STEP, bool FLAT>
__device__ __forceinline__ void attend(const AttendParams &p, const StepTail *st) {
    __shared__ float s_o[kWaves][GH][kHeadDim];
    __shared__ float s_m[kWaves][GH];
    __shared__ float s_l[kWaves][GH];
    const int units = p.n_kv_heads * p.head_groups;
    auto segment = [&](int i, int u, int a, int b, int part) {
        const int g = u / p.head_groups;
        const int h0 = g * p.group + (u - g * p.head_groups) * GH;
        const int first = p.start[i] >> 6;
        attend_segment<GH, STEP>(p, i, g, h0, first + a, first + b, part, s_o, s_m, s_l);
    };
    if constexpr (FLAT) {
        // Segments in sequence order; a decode step counts the workgroup in
        // after each, so a workgroup that crosses into the next sequence has
        // arrived for the previous one before it streams on.  Pass 2 of the
        // last segment's sequence follows at once when it is the last
        // arrival; that of an earlier one, after the last segment.
        __shared__ int s_fin[kMaxLaunchSeqs];
        int n_fin = 0;
        const int w = blockIdx.x / units;
        const int u = blockIdx.x - w * units;
        const int64_t total = p.flat_begin[p.n];
        const int lo = (int)(w * total / p.flat_wgs);
        const int hi = (int)((w + 1) * total / p.flat_wgs);
        auto has_segment = [&](int i, int &a, int &b) {
            const int fb = p.flat_begin[i];
            const int nt = seq_tiles(p, i);
            a = nt ? max(fb, lo) - fb : 0;
            b = nt ? min(fb + nt, hi) - fb : 0;
            return nt ? a < b : STEP && p.wfirst[i] == w;
        };
        // a decode step takes its last segment out of the loop, so that the
        // register-heavy pass 2 is not inside it
        int i_last = p.n;
        if constexpr (STEP) {
            for (int i = 0; i < p.n; ++i) {
                int a, b;
                if (has_segment(i, a, b)) i_last = i;
            }
        }
        for (int i = 0; i < i_last; ++i) {
            int a, b;
            if (!has_segment(i, a, b)) continue;
            segment(i, u, a, b, p.chunk_begin[i] + (w - p.wfirst[i]));
            __syncthreads();   // s_o, s_m, s_l are free again
            if constexpr (STEP) {
                if (count_in(p, *st, i, u, units)) {
                    if (threadIdx.x == 0) s_fin[n_fin] = i;
                    ++n_fin;
                }
            }
        }
        if constexpr (STEP) {
            if (i_last < p.n) {
                const int i = i_last;
                int a, b;
                has_segment(i, a, b);
                segment(i, u, a, b, p.chunk_begin[i] + (w - p.wfirst[i]));
                __syncthreads();
                // pass 2's inputs overlap the wait, as for per-sequence chunks
                const TailIn<GH> tin = tail_inputs<GH>(p, *st, i, u);
                if (count_in(p, *st, i, u, units)) finish<GH>(p, *st, tin, i, u);
                __syncthreads();
            }
        }
        if constexpr (STEP) {
            __syncthreads();
            for (int k = 0; k < n_fin; ++k) {
                const int i = s_fin[k];
                finish<GH>(p, *st, tail_inputs<GH>(p, *st, i, u), i, u);
                __syncthreads();   // the tail's LDS is free again
            }
        }
    } else {
        int i = 0;
        while ((int)blockIdx.x >= p.wg_begin[i + 1]) ++i;
        const int rel = blockIdx.x - p.wg_begin[i];
        const int c = rel / units;
        const int u = rel - c * units;
        const int nt = seq_tiles(p, i);
        const int a = min(c * p.tpc[i], nt);
        segment(i, u, a, min(a + p.tpc[i], nt), p.chunk_begin[i] + c);
        if constexpr (STEP) {
            // the loads pass 2 needs besides the partials overlap the wait in count_in
            const TailIn<GH> tin = tail_inputs<GH>(p, *st, i, u);
            if (count_in(p, *st, i, u, units)) finish<GH>(p, *st, tin, i, u);
        }
    }
}

template <int GH, bool FLAT>
__global__ __launch_bounds__(256, 2) void gqa_attend_kernel(const AttendParams p) {
    attend<GH, false, FLAT>(p, nullptr);
}

template <int GH, bool FLAT>
__global__ __launch_bounds__(256, 2) void gqa_step_kernel(const AttendParams p, const StepTail t) {
    attend<GH, true, FLAT>(p, &t);
}

}  // namespace

namespace {

template <bool FLAT>
hipError_t attend_launch(const AttendParams &p, int heads_per_wg, int n_wg, hipStream_t s) {
    const dim3 grid(n_wg), block(256);
    switch (heads_per_wg) {
        case 1: hipLaunchKernelGGL((gqa_attend_kernel<1, FLAT>), grid, block, 0, s, p); break;
        case 2: hipLaunchKernelGGL((gqa_attend_kernel<2, FLAT>), grid, block, 0, s, p); break;
        case 4: hipLaunchKernelGGL((gqa_attend_kernel<4, FLAT>), grid, block, 0, s, p); break;
        case 8: hipLaunchKernelGGL((gqa_attend_kernel<8, FLAT>), grid, block, 0, s, p); break;
        case 16: hipLaunchKernelGGL((gqa_attend_kernel<16, FLAT>), grid, block, 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <bool FLAT>
hipError_t step_launch(const AttendParams &p, const StepTail &t, int heads_per_wg, int n_wg, hipStream_t s) {
    const dim3 grid(n_wg), block(256);
    switch (heads_per_wg) {
        case 1: hipLaunchKernelGGL((gqa_step_kernel<1, FLAT>), grid, block, 0, s, p, t); break;
        case 2: hipLaunchKernelGGL((gqa_step_kernel<2, FLAT>), grid, block, 0, s, p, t); break;
        case 4: hipLaunchKernelGGL((gqa_step_kernel<4, FLAT>), grid, block, 0, s, p, t); break;
        case 8: hipLaunchKernelGGL((gqa_step_kernel<8, FLAT>), grid, block, 0, s, p, t); break;
        case 16: hipLaunchKernelGGL((gqa_step_kernel<16, FLAT>), grid, block, 0, s, p, t); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gqa_attend(const AttendParams &p, int heads_per_wg, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    return p.flat_wgs > 0 ? attend_launch<true>(p, heads_per_wg, n_wg, s) : attend_launch<false>(p, heads_per_wg, n_wg, s);
}

hipError_t launch_gqa_step(const AttendParams &p, const StepTail &t, int heads_per_wg, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    return p.flat_wgs > 0 ? step_launch<true>(p, t, heads_per_wg, n_wg, s)
                          : step_launch<false>(p, t, heads_per_wg, n_wg, s);
}

}  // namespace wsk
