// Split-KV decode attention over an MLA latent partition (pass 1), gfx950.
//
// MLA caches one compressed latent row per token: c (512) | r (64, decoupled
// RoPE key).  With the query absorbed into the latent space (Sec. 6.1,
// compressed-MLA variant), every head attends the same rows:
//
//   s_h,j = scale * (q_lat[h] . c_j + q_rope[h] . r_j),   O_lat[h] = sum_j p_h,j c_j
//
// so heads x latent form a dense tile and both products run on the matrix
// cores (v_mfma_f32_16x16x32_bf16, up to 16 heads):
//
//   S^T [64 tokens x 16 heads] = C [64 x 576] . Q^T [576 x 16]
//   O   [16 heads x 512]      += P [16 x 64]  . c [64 x 512]
//
// Each latent row is read from HBM once and used by both products (the
// paper's CPU kernel makes the same point for its cache tiles).  A workgroup
// of 4 wavefronts walks one chunk of 64-token tiles together:
//   - wavefront w fetches the rows of its QK M-tile (16 tokens x 576) from
//     HBM straight into its A-operand registers, one tile ahead, computes
//     QK there (18 MFMAs in two independent chains), and stores the rows to
//     the double-buffered LDS tile (72 KB) that all wavefronts' P.V reads;
//   - the tile max per head is exchanged through LDS; probabilities go to
//     LDS as bf16 hi + lo parts in the P.V A-operand order;
//   - P.V: wavefront w computes output dims [128w, 128w + 128) for all 64
//     tokens; its B-operands (8 consecutive tokens of one dim) come from the
//     row-major tile through ds_read_b64_tr_b16, which transposes 16 lanes'
//     4-element rows into 4-token columns.
// LDS placement: row (token) t, 16-byte chunk c of the tile lives at slot
// t*72 + (c ^ x(t)); x(t) spreads the rows read together by one instruction
// over distinct banks for both the QK reads and the transposing reads.
// Tokens outside [start, end) are fetched from past the buffer descriptor's
// extent, which yields zeros, and their scores are masked to -inf.

#include "wsk_internal.h"

namespace wsk {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kRow = kLatent + kRope;        // 576 bf16 per cached token
constexpr int kChunksPerRow = kRow / 8;      // 72 16-byte chunks
constexpr int kTileSlots = kTile * kChunksPerRow;   // 4608 16-byte slots = 72 KB
constexpr int kKSteps = kRow / 32;           // 18 QK K-steps

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int tile_token(int mt, int r) {
    return 32 * (mt >> 1) + 8 * (r >> 2) + 4 * (mt & 1) + (r & 3);
}
// bank spread of row t (0..7): bit 1 of t -> bit 1, bit 3 -> bit 0, bit 4 -> bit 2
__device__ __forceinline__ int row_xor(int t) {
    return (((t >> 1) & 1) << 1) | ((t >> 3) & 1) | (((t >> 4) & 1) << 2);
}

__global__ __launch_bounds__(256, 1) void mla_attend_kernel(const AttendParams p) {
    __shared__ u32x4 s_tile[2][kTileSlots];           // 2 x 72 KB
    __shared__ u32x4 s_p[2][2][4][16];                // [hi/lo][ks][grp][head] 8 bf16 = 2 KB
    __shared__ float s_max[4][16];
    __shared__ float s_sum[4][16];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int grp = lane >> 4;

    // ---- work item (uniform): sequence i, chunk c ----
    const int wg = blockIdx.x;
    int i = 0;
    while (wg >= p.wg_begin[i + 1]) ++i;
    const int c = wg - p.wg_begin[i];
    const int seq = p.seq[i];
    const int t_start = p.start[i];
    const int t_end = p.end[i];
    const int tpc = p.tpc[i];
    const int tile0 = (t_start >> 6) + c * tpc;
    const int tile_end = min(tile0 + tpc, ((t_end - 1) >> 6) + 1);
    const int H = p.n_q_heads;
    typedef const __attribute__((address_space(4))) int32_t ci32;
    ci32 *trow = (ci32 *)(p.table + (int64_t)seq * p.table_stride);
    const int bk = p.block_tokens;
    const int bshift = __builtin_ctz(bk);
    const int slot_bytes = bk * kRow * 2;

    // Q^T operand: lane (grp, n) holds q[n][32ks + 8grp .. +8] for all 18 K-steps
    bf16x8 qop[kKSteps];
    {
        const u32x4 *qrow = reinterpret_cast<const u32x4 *>(p.q + (int64_t)i * p.q_row +
                                                            (int64_t)(n < H ? n : 0) * kRow);
#pragma unroll
        for (int ks = 0; ks < kKSteps; ++ks) {
            const u32x4 v = qrow[ks * 4 + grp];
            qop[ks] = as_bf16x8(n < H ? v : u32x4{0u, 0u, 0u, 0u});
        }
    }

    // Staging: lane (grp, n) of wavefront w fetches, for each K-step ks, the
    // 16 bytes its QK A-operand needs -- token tile_token(w, n), chunk
    // 4ks + grp -- straight into registers, multiplies them there, and also
    // stores them to the LDS tile (slot token*72 + (chunk ^ row_xor(token)))
    // for every wavefront's P.V.
    const int st_tok = tile_token(wave, n);
    const int st_x = row_xor(st_tok);
    u32x4 stX[kKSteps], stY[kKSteps];
    // Tiles past the chunk's end are "loaded" from past the descriptor's
    // extent (no memory traffic): loads stay unconditional so the compiler
    // waits for exactly the stage it needs.
    auto load_tile = [&](int t, u32x4 (&st)[kKSteps]) {
        const bool valid = t < tile_end;
        const int tt = valid ? t : tile0;
        const int tok0 = tt * kTile;
        const int blk = tok0 >> bshift;
        const int row0 = tok0 - (blk << bshift);
        const int slot = __builtin_amdgcn_readfirstlane(trow[blk]);
        const uint16_t *base = p.pool + (int64_t)slot * p.slot_elems;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, slot_bytes, 0x00020000);
        const int tk = tok0 + st_tok;
        // rows outside [start, end) are fetched from past the extent: zeros
        const bool ok = valid && tk >= t_start && tk < t_end;
        const int off0 = ok ? st_tok * (kRow * 2) + grp * 16 : 0x40000000;
#pragma unroll
        for (int ks = 0; ks < kKSteps; ++ks)
            st[ks] = __builtin_amdgcn_raw_buffer_load_b128(rs, off0 + (ok ? ks * 64 : 0), row0 * (kRow * 2),
                                                           kStreamLoad);
    };
    auto store_tile = [&](int buf, const u32x4 (&st)[kKSteps]) {
        u32x4 *dst = s_tile[buf] + st_tok * kChunksPerRow;
#pragma unroll
        for (int ks = 0; ks < kKSteps; ++ks) dst[(4 * ks + grp) ^ st_x] = st[ks];
    };

    // P.V transposing reads: lane (grp, i=n) points at token 32ks + 8grp + 4h + n/4,
    // dims 128*wave + 16nt + 4(n%4) .. +4, i.e. chunk 16*wave + 2nt + (n%4)/2, half (n%4)%2
    const int tr_tok_lo = 8 * grp + (n >> 2);
    const int tr_chunk = 16 * wave + ((n & 3) >> 1);
    const int tr_half = (n & 1) * 8;

    float m_run = -INFINITY;
    float l_lane = 0.f;
    f32x4 o[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // One tile: QK from the registers of `cur` (tile t, already in LDS buffer
    // buf), refill `cur` with tile t+2, softmax, P.V from LDS, then publish
    // `nxt` (tile t+1) into the other buffer.
    auto step = [&](int t, int buf, u32x4 (&cur)[kKSteps], u32x4 (&nxt)[kKSteps]) {
        f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = f32x4{0.f, 0.f, 0.f, 0.f};
        if (t < tile_end) {
            __syncthreads();   // tile t is in LDS for every wavefront; tile t-1 is no longer read
#pragma unroll
            for (int ks = 0; ks < kKSteps; ks += 2) {
                s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur[ks]), qop[ks], s0, 0, 0, 0);
                s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur[ks + 1]), qop[ks + 1], s1, 0, 0, 0);
            }
        }
        load_tile(t + 2, cur);
        if (t < tile_end) {
            const int tok0 = t * kTile;
            const u32x4 *tile = s_tile[buf];
            const f32x4 s = s0 + s1;
            // ---- softmax over the 64 tokens of the tile, per head n ----
            const bool partial = tok0 < t_start || tok0 + kTile > t_end;
            float sv[4];
            float mloc = -INFINITY;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tk = tok0 + tile_token(wave, 4 * grp + r);
                const bool ok = !partial || (tk >= t_start && tk < t_end);
                sv[r] = ok ? s[r] * p.scale_log2 : -INFINITY;
                mloc = fmaxf(mloc, sv[r]);
            }
            mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
            mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
            if (grp == 0) s_max[wave][n] = mloc;
            __syncthreads();
            const float mt = fmaxf(fmaxf(s_max[0][n], s_max[1][n]), fmaxf(s_max[2][n], s_max[3][n]));
            const float m_new = fmaxf(m_run, mt);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            float psum = 0.f;
            bf16x4 phi, plo;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float pv = __builtin_amdgcn_exp2f(sv[r] - m_new);
                psum += pv;
                const __bf16 hi = (__bf16)pv;
                phi[r] = hi;
                plo[r] = (__bf16)(pv - (float)hi);
            }
            l_lane = fmaf(l_lane, alpha, psum);
            // tokens 32(w>>1) + 8grp + 4(w&1) + r are elements 4(w&1) + r of the
            // P.V A-operand of (ks = w>>1, grp, head n)
            {
                u32x2 *dh = reinterpret_cast<u32x2 *>(&s_p[0][wave >> 1][grp][n]) + (wave & 1);
                u32x2 *dl = reinterpret_cast<u32x2 *>(&s_p[1][wave >> 1][grp][n]) + (wave & 1);
                *dh = __builtin_bit_cast(u32x2, phi);
                *dl = __builtin_bit_cast(u32x2, plo);
            }
            float alpha_r[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) alpha_r[r] = __shfl(alpha, 4 * grp + r);
#pragma unroll
            for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r) o[nt][r] *= alpha_r[r];
            __syncthreads();

            // ---- P.V: output dims [128 wave, 128 wave + 128) ----
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 ahi = as_bf16x8(s_p[0][ks][grp][n]);
                const bf16x8 alo = as_bf16x8(s_p[1][ks][grp][n]);
                s16x4 half[8][2];
#pragma unroll
                for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2) {
                        const int tk = 32 * ks + tr_tok_lo + 4 * h2;
                        const int ch = tr_chunk + 2 * nt;
                        const char *addr = reinterpret_cast<const char *>(tile) +
                                           (tk * kChunksPerRow + (ch ^ row_xor(tk))) * 16 + tr_half;
                        half[nt][h2] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (__attribute__((address_space(3))) s16x4 *)(addr));
                    }
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) {
                    const bf16x8 b = __builtin_bit_cast(
                        bf16x8, __builtin_shufflevector(half[nt][0], half[nt][1], 0, 1, 2, 3, 4, 5, 6, 7));
                    o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, b, o[nt], 0, 0, 0);
                    o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, b, o[nt], 0, 0, 0);
                }
            }
            if (t + 1 < tile_end) store_tile(buf ^ 1, nxt);   // nobody reads buf^1 until the next barrier
        }
    };

    if (tile0 < tile_end) {
        load_tile(tile0, stX);
        store_tile(0, stX);
        load_tile(tile0 + 1, stY);
    }
    for (int t = tile0; t < tile_end; t += 2) {
        step(t, 0, stX, stY);
        step(t + 1, 1, stY, stX);
    }

    // ---- normalise and write this chunk's partial ----
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (grp == 0) s_sum[wave][n] = l_tot;
    __syncthreads();
    const float den = s_sum[0][n] + s_sum[1][n] + s_sum[2][n] + s_sum[3][n];   // head n
    float inv_r[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) inv_r[r] = 1.f / __shfl(den, 4 * grp + r);
    const int part = p.chunk_begin[i] + c;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int h = 4 * grp + r;
        if (h < H) {
            float *dst = p.part_o + ((int64_t)part * H + h) * kLatent + 128 * wave + n;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) dst[16 * nt] = o[nt][r] * inv_r[r];
        }
    }
    if (wave == 0 && grp == 0 && n < H)
        p.part_lse[(int64_t)part * H + n] = (m_run + __log2f(den)) * 0.69314718055994530942f;
}

}  // namespace

hipError_t launch_mla_attend(const AttendParams &p, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    hipLaunchKernelGGL(mla_attend_kernel, dim3(n_wg), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace wsk
