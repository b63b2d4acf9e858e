// Split-KV decode attention over a GQA partition (pass 1), gfx950.
//
// Computes, for every query head of a KV head, the exact softmax attention
// over one chunk of the sequence range (the GPU engine of Sec. 5.1), and
// writes the normalised partial output and its natural-log LSE (the
// "partial output and normaliser" of Sec. 4.2).
//
// Work mapping (one workgroup = 4 wavefronts):
//   workgroup -> (sequence, KV head, group of GH query heads, chunk of tiles)
//   wavefront -> every 4th 64-token tile of the chunk, own online softmax
// Per tile and wavefront:
//   1. K tile (64 tokens x 128 bf16 = 16 KB) is read with coalesced 16-byte
//      loads (each instruction covers 4 full rows) and stored to LDS with the
//      16-byte chunk index XOR-ed by the row, so that reading one whole row
//      per lane hits distinct banks.
//   2. QK: lane j owns token j.  v_dot2 bf16 products with fp32 accumulation;
//      the query rows stay uniform across the wave (scalar registers).
//   3. Tile max per head with DPP row reductions + 4 readlanes; exp2-domain
//      online softmax (scale folded with log2 e).
//   4. P·V: lane (row group r, 16-byte chunk c) owns dims 8c..8c+7 for rows
//      r, r+4, ...; V comes straight from HBM in 16-byte loads; probabilities
//      are broadcast from LDS.  fp32 FMA, fp32 probabilities.
// The next tile's K and V loads are issued while the current tile computes.
// At the end the four wavefront states are merged through LDS.

#include "wsk_internal.h"

namespace wsk {
namespace {

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float lane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// DPP controls: quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror.
// Applied in this order they pair every lane of a 16-lane row with each other lane.
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f<0xB1>(v));
    v = fmaxf(v, dpp_f<0x4E>(v));
    v = fmaxf(v, dpp_f<0x141>(v));
    v = fmaxf(v, dpp_f<0x140>(v));
    return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x141>(v);
    v += dpp_f<0x140>(v);
    return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}

constexpr int kWaves = 4;
constexpr int kChunks = kHeadDim * 2 / 16;   // 16-byte chunks per row: 16

// Up to 4 heads per workgroup fit two workgroups per CU (<= 256 registers per
// lane); 5-8 heads need the whole register file (one workgroup per CU).
template <int GH>
__global__ __launch_bounds__(256, (GH <= 4 ? 2 : 1)) void gqa_attend_kernel(const AttendParams p) {
    __shared__ u32x4 s_k[kWaves][kTile * kChunks];   // 4 x 16 KB
    __shared__ float s_p[kWaves][kTile][8];           // 4 x 2 KB
    __shared__ float s_m[kWaves][8];
    __shared__ float s_l[kWaves][8];

    const int lane = threadIdx.x & 63;
    // uniform within a wavefront; readfirstlane tells the compiler so, which
    // keeps all tile addressing on the scalar unit
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

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
    const int tile0 = (t_start >> 6) + c * p.tiles_per_chunk;
    const int tile_end = min(tile0 + p.tiles_per_chunk, ((t_end - 1) >> 6) + 1);
    const int h0 = g * p.group + hg * GH;
    // The query rows are read-only for the whole kernel: read them through the
    // constant address space so they are fetched with scalar loads into SGPRs.
    typedef const __attribute__((address_space(4))) uint32_t cu32;
    cu32 *qw = (cu32 *)(p.q + (int64_t)i * p.q_row + (int64_t)h0 * kHeadDim);
    typedef const __attribute__((address_space(4))) int32_t ci32;
    ci32 *trow = (ci32 *)(p.table + (int64_t)seq * p.table_stride);   // read-only here
    const int bk = p.block_tokens;
    const int bshift = __builtin_ctz(bk);     // block_tokens is a power of two
    const int64_t head_off = (int64_t)g * 2 * bk * kHeadDim;

    // Buffer descriptor over the K and V rows of KV head g in the slot of
    // tile tt (2 * block_tokens rows of 256 bytes); soffset selects the tile's
    // first row.  Accesses past the descriptor's extent read zero.
    const int head_bytes = 2 * bk * kHeadDim * 2;
    auto tile_rsrc = [&](int tt, int &row_bytes0) -> __amdgpu_buffer_rsrc_t {
        const int tok0 = tt * kTile;
        const int blk = tok0 >> bshift;
        row_bytes0 = (tok0 - (blk << bshift)) * (kHeadDim * 2);
        const int slot = __builtin_amdgcn_readfirstlane(trow[blk]);
        const uint16_t *base = p.pool + (int64_t)slot * p.slot_elems + head_off;
        return __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, head_bytes, 0x00020000);
    };

    float m_run[GH], l_lane[GH], o[GH][8];
#pragma unroll
    for (int h = 0; h < GH; ++h) {
        m_run[h] = -INFINITY;
        l_lane[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
    }

    const int rgrp = lane >> 4;   // row group 0..3 (rows rgrp, rgrp+4, ...)
    const int chk = lane & 15;    // 16-byte chunk within a row
    u32x4 vreg[16];
    u32x4 *sk = s_k[wave];
    typedef __attribute__((address_space(3))) void lds_void;
    // K tile -> LDS by DMA.  Instruction ii fills LDS slots ii*64 .. ii*64+63;
    // slot (row r, position pc) receives logical chunk pc ^ (r & 15) of row r,
    // so the 16 lanes of a row still read that row's 256 contiguous bytes.
    int koff[4];                                    // lane part of the K DMA source
#pragma unroll
    for (int j = 0; j < 4; ++j) koff[j] = rgrp * 256 + ((chk ^ (j * 4 + rgrp)) * 16);
    const int voff = lane * 16;
    auto issue_k = [&](int tt) {
        int rb0;
        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(tt, rb0);
#pragma unroll
        for (int ii = 0; ii < 16; ++ii)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(sk + ii * 64), 16, koff[ii & 3],
                                                     rb0 + ii * 1024, 0, 0);
    };
    // V rows outside [start, end) may hold anything (even NaN bit patterns);
    // they are read from an offset past the descriptor's extent, which the
    // hardware returns as zeros, so their zero probability adds exactly nothing.
    auto issue_v = [&](int tt) {
        int rb0;
        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(tt, rb0);
        const int vb0 = rb0 + bk * kHeadDim * 2;
        const int tok_l = tt * kTile + rgrp;
#pragma unroll
        for (int ii = 0; ii < 16; ++ii) {
            const int tok = tok_l + ii * 4;
            const int off = (tok >= t_start && tok < t_end) ? voff : 0x40000000;
            vreg[ii] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, vb0 + ii * 1024, 0);
        }
    };

    int t = tile0 + wave;
    if (t < tile_end) {
        issue_k(t);
        issue_v(t);
    }
    for (; t < tile_end; t += kWaves) {
        const int tn = t + kWaves;
        // 2. QK: lane = token.  The query pointer is made opaque per tile so the
        // compiler re-reads the (scalar-cache resident) query inside the loop
        // instead of hoisting GH*64 dwords into scalar registers.
        cu32 *qt = qw;
        asm volatile("" : "+s"(qt));
        float acc[GH];
#pragma unroll
        for (int h = 0; h < GH; ++h) acc[h] = 0.f;
#pragma unroll 2
        for (int ch = 0; ch < kChunks; ++ch) {
            const u32x4 kk = sk[lane * kChunks + (ch ^ (lane & 15))];
#pragma unroll
            for (int h = 0; h < GH; ++h) {
                cu32 *qh = qt + h * (kHeadDim / 2) + ch * 4;
                acc[h] = dot2_bf16(qh[0], kk.x, acc[h]);
                acc[h] = dot2_bf16(qh[1], kk.y, acc[h]);
                acc[h] = dot2_bf16(qh[2], kk.z, acc[h]);
                acc[h] = dot2_bf16(qh[3], kk.w, acc[h]);
            }
        }

        // every lane has read its K row: the buffer may be refilled
        __builtin_amdgcn_wave_barrier();
        if (tn < tile_end) issue_k(tn);

        // 3. online softmax in the exp2 domain
        const int tok = t * kTile + lane;
        const bool valid = tok >= t_start && tok < t_end;
        float pr[GH], alpha[GH];
#pragma unroll
        for (int h = 0; h < GH; ++h) {
            const float s = valid ? acc[h] * p.scale_log2 : -INFINITY;
            const float mn = fmaxf(m_run[h], wave_max(s));
            alpha[h] = __builtin_amdgcn_exp2f(m_run[h] - mn);
            pr[h] = __builtin_amdgcn_exp2f(s - mn);
            l_lane[h] = fmaf(l_lane[h], alpha[h], pr[h]);
            m_run[h] = mn;
        }
        float *prow = s_p[wave][lane];
#pragma unroll
        for (int h = 0; h < GH; ++h) prow[h] = pr[h];
        __builtin_amdgcn_wave_barrier();

        // 4. P·V
#pragma unroll
        for (int h = 0; h < GH; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) o[h][e] *= alpha[h];
#pragma unroll
        for (int ii = 0; ii < 16; ++ii) {
            const int r = ii * 4 + rgrp;
            float pv[GH];
            const float *pp = s_p[wave][r];
            if constexpr (GH == 8) {
                const f32x4 a = *reinterpret_cast<const f32x4 *>(pp);
                const f32x4 b = *reinterpret_cast<const f32x4 *>(pp + 4);
                pv[0] = a.x; pv[1] = a.y; pv[2] = a.z; pv[3] = a.w;
                pv[4] = b.x; pv[5] = b.y; pv[6] = b.z; pv[7] = b.w;
            } else {
#pragma unroll
                for (int h = 0; h < GH; ++h) pv[h] = pp[h];
            }
            const u32x4 w4 = vreg[ii];
            const float vf[8] = {bf16_lo(w4.x), bf16_hi(w4.x), bf16_lo(w4.y), bf16_hi(w4.y),
                                 bf16_lo(w4.z), bf16_hi(w4.z), bf16_lo(w4.w), bf16_hi(w4.w)};
#pragma unroll
            for (int h = 0; h < GH; ++h)
#pragma unroll
                for (int e = 0; e < 8; ++e) o[h][e] = fmaf(pv[h], vf[e], o[h][e]);
            // keep each row step's probability reads and conversions next to
            // their FMAs (hoisting them all needs > 100 extra registers)
            if constexpr (GH > 2) __builtin_amdgcn_sched_barrier(0);
        }
        if (tn < tile_end) issue_v(tn);
        __builtin_amdgcn_wave_barrier();
    }

    // ---- merge the four wavefront states ----
    float l_w[GH];
#pragma unroll
    for (int h = 0; h < GH; ++h) l_w[h] = wave_sum(l_lane[h]);
    float *red = reinterpret_cast<float *>(sk);   // [4 row groups][GH][128] fp32 <= 16 KB
#pragma unroll
    for (int h = 0; h < GH; ++h) {
        f32x4 *dst = reinterpret_cast<f32x4 *>(red + (rgrp * GH + h) * kHeadDim + chk * 8);
        dst[0] = f32x4{o[h][0], o[h][1], o[h][2], o[h][3]};
        dst[1] = f32x4{o[h][4], o[h][5], o[h][6], o[h][7]};
    }
    if (lane == 0) {
#pragma unroll
        for (int h = 0; h < GH; ++h) {
            s_m[wave][h] = m_run[h];
            s_l[wave][h] = l_w[h];
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
            const float *rw = reinterpret_cast<const float *>(s_k[w]);
            float sum = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) sum += rw[(r * GH + h) * kHeadDim + d];
            num = fmaf(a, sum, num);
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
        case 3: hipLaunchKernelGGL(gqa_attend_kernel<3>, grid, block, 0, s, p); break;
        case 4: hipLaunchKernelGGL(gqa_attend_kernel<4>, grid, block, 0, s, p); break;
        case 5: hipLaunchKernelGGL(gqa_attend_kernel<5>, grid, block, 0, s, p); break;
        case 6: hipLaunchKernelGGL(gqa_attend_kernel<6>, grid, block, 0, s, p); break;
        case 7: hipLaunchKernelGGL(gqa_attend_kernel<7>, grid, block, 0, s, p); break;
        case 8: hipLaunchKernelGGL(gqa_attend_kernel<8>, grid, block, 0, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace wsk
