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
// Work mapping: workgroup = (sequence, KV head, group of GH <= 16 query
// heads, chunk of 64-token tiles); its 4 wavefronts take every 4th tile of the
// chunk with their own online softmax and are merged through LDS at the end.
// Each wavefront issues the next tile's K loads as soon as QK has consumed
// the current ones, and the next V loads right after P.V.

#include "wsk_internal.h"

namespace wsk {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kWaves = 4;
constexpr int kTileBytes = 2 * kTile * kHeadDim * 2;   // K and V pieces of one 64-token tile: 32 KB

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Token (0..63) of row r (0..15) of QK M-tile mt (0..3).  Rows 4g..4g+3 of
// M-tiles 2k and 2k+1 are tokens 32k + 8g .. 32k + 8g + 7.
__device__ __forceinline__ int tile_token(int mt, int r) {
    return 32 * (mt >> 1) + 8 * (r >> 2) + 4 * (mt & 1) + (r & 3);
}

template <int GH>
__global__ __launch_bounds__(256, 2) void gqa_attend_kernel(const AttendParams p) {
    __shared__ float s_o[kWaves][GH][kHeadDim];
    __shared__ float s_m[kWaves][GH];
    __shared__ float s_l[kWaves][GH];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;     // MFMA column: query head (QK) / dim within an N-tile (P.V)
    const int grp = lane >> 4;   // MFMA k-group 0..3

    // ---- work item of this workgroup (uniform) ----
    const int wg = blockIdx.x;
    int i = 0;
    while (wg >= p.wg_begin[i + 1]) ++i;
    const int rel = wg - p.wg_begin[i];
    const int units = p.n_kv_heads * p.head_groups;
    const int c = rel / units;
    const int u = rel - c * units;
    const int g = u / p.head_groups;
    const int hg = u - g * p.head_groups;
    const int seq = p.seq[i];
    const int t_start = p.start[i];
    const int t_end = p.end[i];
    const int tpc = p.tpc[i];
    const int tile0 = (t_start >> 6) + c * tpc;
    const int tile_end = min(tile0 + tpc, ((t_end - 1) >> 6) + 1);
    const int h0 = g * p.group + hg * GH;
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

    const int part = p.chunk_begin[i] + c;
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
        p.part_o[row * kHeadDim + d] = num / den;
        if (d == 0) p.part_lse[row] = (M + __log2f(den)) * 0.69314718055994530942f;
    }
}

}  // namespace

hipError_t launch_gqa_attend(const AttendParams &p, int heads_per_wg, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    const dim3 grid(n_wg), block(256);
    switch (heads_per_wg) {
        case 1: hipLaunchKernelGGL(gqa_attend_kernel<1>, grid, block, 0, s, p); break;
        case 2: hipLaunchKernelGGL(gqa_attend_kernel<2>, grid, block, 0, s, p); break;
        case 4: hipLaunchKernelGGL(gqa_attend_kernel<4>, grid, block, 0, s, p); break;
        case 8: hipLaunchKernelGGL(gqa_attend_kernel<8>, grid, block, 0, s, p); break;
        case 16: hipLaunchKernelGGL(gqa_attend_kernel<16>, grid, block, 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace wsk
