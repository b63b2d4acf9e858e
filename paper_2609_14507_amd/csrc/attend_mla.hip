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
//   S^T [32 tokens x 16 heads] = C [32 x 576] . Q^T [576 x 16]     (2 M-tiles)
//   O   [16 heads x 512]      += P [16 x 32]  . c [32 x 512]       (32 N-tiles)
//
// Each latent row is read from HBM once and used by both products (the
// paper's CPU kernel makes the same point for its cache tiles).
//
// A workgroup is two teams of 4 wavefronts; the teams take alternate 32-token
// tiles of the workgroup's chunk and merge their results through LDS at the
// end (one partial per workgroup).  Within a team, the tile's 18 K-steps are
// split over the wavefronts by latent columns: wavefront w holds latent dims
// [128w, 128w + 128) (K-steps 4w .. 4w+3) and, for w < 2, the rope K-step
// 16 + w.  It computes a partial S^T over its K-steps and, after one exchange
// of partial scores through LDS, the P.V product for its own 128 output
// columns.
//   - The GPU pool stores each 32-token tile in the order of the QK
//     A-operand registers (WSK_LAYOUT_MLA32): load (ks, mt) is one fully
//     coalesced 1 KB read landing in the registers that feed the MFMA.
//   - P.V contracts over tokens, so its B-operand needs 8 consecutive tokens
//     of one latent dim per lane: the transpose of what was loaded.  After
//     QK each wavefront stores its 8 latent pieces, unchanged, in its own
//     8 KB of LDS and reads the operand back with ds_read_b64_tr_b16 (two
//     reads of 4 tokens per N-tile): no other wavefront touches that LDS,
//     so no barrier guards it.
//   - The token order inside an M-tile makes the QK accumulator of lane
//     (g, n) hold tokens 8g..8g+7 of head n, which is exactly the P.V
//     A-operand: probabilities never leave the registers.
//   - Each wavefront holds one tile's pieces in registers; once QK has
//     used them (and LDS has taken the latent ones) they take the team's
//     next tile, whose reads fly during the score exchange, softmax and P.V.
//     One tile in flight per wavefront streams faster here than two, three
//     or four: more outstanding reads lower the rate HBM delivers.
//   - The only synchronisation is the barrier of the score exchange (one
//     per round of two tiles, shared by both teams; partial scores are
//     double-buffered).
// Tokens outside [start, end) are fetched from past the buffer descriptor's
// extent, which yields zeros, and their scores are masked to -inf.

#include "wsk_internal.h"

namespace wsk {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(8))) short s16x8;

constexpr int kRow = kLatent + kRope;          // 576 bf16 per cached token
constexpr int kSub = 32;                       // tokens per tile
constexpr int kSubBytes = kSub * kRow * 2;     // 36864
constexpr int kWaveKS = 5;                     // K-steps per wavefront (4 latent + rope for w < 2)
constexpr int kWaveNT = 8;                     // P.V N-tiles (128 columns) per wavefront
constexpr int kDepth = 1;                      // tiles held per wavefront (in flight while one is used)
constexpr int kOOB = 0x40000000;               // offset past any descriptor extent

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// token (0..31) held by row r of M-tile mt
__device__ __forceinline__ int sub_token(int mt, int r) { return 8 * (r >> 2) + 4 * mt + (r & 3); }

__global__ __launch_bounds__(512, 1) void mla_attend_kernel(const AttendParams p) {
    __shared__ f32x4 s_part[2][2][4][2][64];       // 32 KB: partial S^T per team and wavefront, double-buffered
    __shared__ __attribute__((aligned(16))) uint8_t s_tr[8][8 * 1024];   // 64 KB: each wavefront's latent pieces
    __shared__ float s_mt[2][16], s_lt[2][16];      // per team: running max and normaliser of each head

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int team = wv >> 2;       // two teams of 4 wavefronts take alternate tiles
    const int wave = wv & 3;
    const int n = lane & 15;
    const int grp = lane >> 4;
    const bool rope = wave < 2;

    // ---- work item (uniform): sequence i, chunk c ----
    const int wg = blockIdx.x;
    int i = 0;
    while (wg >= p.wg_begin[i + 1]) ++i;
    const int c = wg - p.wg_begin[i];
    const int seq = p.seq[i];
    const int t_start = p.start[i];
    const int t_end = p.end[i];
    const int tile0 = (t_start >> 6) + c * p.tpc[i];   // a chunk is tpc 64-token tiles
    const int sub_begin = max(2 * tile0, t_start >> 5);
    const int sub_end = min(2 * (tile0 + p.tpc[i]), ((t_end - 1) >> 5) + 1);
    const int H = p.n_q_heads;
    typedef const __attribute__((address_space(4))) int32_t ci32;
    ci32 *trow = (ci32 *)(p.table + (int64_t)seq * p.table_stride);
    const int bk = p.block_tokens;
    const int bshift = __builtin_ctz(bk);
    const int slot_bytes = bk * kRow * 2;

    // K-step j of this wavefront: latent 4w + j (j < 4), rope 16 + w (j = 4)
    auto ks_of = [&](int j) { return j < 4 ? 4 * wave + j : 16 + wave; };

    // Q^T operands of those K-steps: lane (grp, n) holds q[n][32ks + 8grp .. +8]
    bf16x8 qop[kWaveKS];
    {
        const u32x4 *qrow = reinterpret_cast<const u32x4 *>(p.q + (int64_t)i * p.q_row +
                                                            (int64_t)(n < H ? n : 0) * kRow);
#pragma unroll
        for (int j = 0; j < kWaveKS; ++j) {
            const u32x4 v = qrow[ks_of(j) * 4 + grp];
            qop[j] = as_bf16x8((n < H && (j < 4 || rope)) ? v : u32x4{0u, 0u, 0u, 0u});
        }
    }
    // this wavefront's LDS copy of its latent pieces, and the address its
    // lane reads transposed: lane 16g + 4e + a reads token row 4g + e, dims
    // 4a .. 4a+3 of an N-tile (see the P.V loop)
    uint8_t *trbuf = &s_tr[wv][0];
    const int tr_off = 256 * ((lane & 3) >> 1) + 64 * grp + 16 * ((lane >> 2) & 3) + 8 * (lane & 1);

    // ---- tile addressing ----
    struct Src {
        __amdgpu_buffer_rsrc_t rs;
        int soff;       // byte offset of the tile in its slot
        int voff[2];    // per M-tile lane offset (kOOB for rows outside the range)
    };
    auto tile_src = [&](int sub) {
        Src s;
        const bool valid = sub < sub_end;
        const int su = valid ? sub : sub_begin;
        const int tok0 = su * kSub;
        const int blk = tok0 >> bshift;
        const int slot = __builtin_amdgcn_readfirstlane(trow[blk]);
        // a missing table entry (< 0) gets an empty extent: its loads read
        // zeros instead of memory outside the pool
        s.rs = __builtin_amdgcn_make_buffer_rsrc((void *)(p.pool + (slot < 0 ? 0 : (int64_t)slot * p.slot_elems)), 0,
                                                 slot < 0 ? 0 : slot_bytes, 0x00020000);
        s.soff = ((tok0 & (bk - 1)) >> 5) * kSubBytes;
        const bool partial = tok0 < t_start || tok0 + kSub > t_end;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            const int tk = tok0 + sub_token(mt, n);
            const bool ok = valid && (!partial || (tk >= t_start && tk < t_end));
            s.voff[mt] = ok ? lane * 16 : kOOB;
        }
        return s;
    };
    typedef u32x4 Stage[kWaveKS][2];
    // (wavefronts 2 and 3 have no rope K-step: their fifth piece is fetched
    // from past the extent, which costs no memory traffic and keeps every
    // wavefront's instruction stream, and its load counts, the same)
    auto load_j = [&](const Src &s, Stage &st, int j) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
            st[j][mt] = __builtin_amdgcn_raw_buffer_load_b128(s.rs, (j < 4 || rope) ? s.voff[mt] : kOOB,
                                                              s.soff + (2 * ks_of(j) + mt) * 1024, kStreamLoad);
    };
    auto load_tile = [&](int sub, Stage &st) {
        const Src s = tile_src(sub);
#pragma unroll
        for (int j = 4; j >= 0; --j) load_j(s, st, j);
    };

    f32x4 o[kWaveNT];
#pragma unroll
    for (int nt = 0; nt < kWaveNT; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;
    float l_lane = 0.f;

    // One tile t held in st: partial QK, score exchange, softmax, P.V; each
    // K-step of st is refilled with this team's tile kDepth rounds ahead as
    // soon as QK has used it.
    auto step = [&](int t, Stage &st) {
        const bool valid = t < sub_end;
        const Src nx = tile_src(t + 2 * kDepth);
        const int tok0 = t * kSub;
        f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = f32x4{0.f, 0.f, 0.f, 0.f};
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(st[4][0]), qop[4], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(st[4][1]), qop[4], s1, 0, 0, 0);
        load_j(nx, st, 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(st[j][0]), qop[j], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(st[j][1]), qop[j], s1, 0, 0, 0);
        }
        // the latent pieces go to LDS in the order they were loaded (piece
        // (j, mt) at 1 KB (2j + mt), lane l's 16 bytes at 16 l) for P.V's
        // transposed reads; their registers take the next tile at once
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
                *reinterpret_cast<u32x4 *>(trbuf + (2 * j + mt) * 1024 + lane * 16) = st[j][mt];
            load_j(nx, st, j);
        }
        // ---- exchange partial scores; every wavefront sums them in the same order ----
        const int b = (t >> 1) & 1;
        s_part[team][b][wave][0][lane] = s0;
        s_part[team][b][wave][1][lane] = s1;
        __syncthreads();
        if (!valid) return;   // this team has no tile in the last round
        f32x4 S0 = s_part[team][b][0][0][lane], S1 = s_part[team][b][0][1][lane];
#pragma unroll
        for (int w = 1; w < 4; ++w) {
            S0 += s_part[team][b][w][0][lane];
            S1 += s_part[team][b][w][1][lane];
        }

        // ---- online softmax: lane (grp, n) holds head n, tokens 8grp + e ----
        const bool partial = tok0 < t_start || tok0 + kSub > t_end;
        float sv[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            sv[r] = S0[r] * p.scale_log2;
            sv[4 + r] = S1[r] * p.scale_log2;
        }
        if (partial) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int tk = tok0 + 8 * grp + e;
                if (tk < t_start || tk >= t_end) sv[e] = -INFINITY;
            }
        }
        float mloc = sv[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mloc = fmaxf(mloc, sv[e]);
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        const float m_new = fmaxf(m_run, mloc);      // finite: every tile holds a token of the range
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        bf16x8 phi, plo;
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float pv = __builtin_amdgcn_exp2f(sv[e] - m_new);
            psum += pv;
            const __bf16 hi = (__bf16)pv;
            phi[e] = hi;
            plo[e] = (__bf16)(pv - (float)hi);
        }
        l_lane = fmaf(l_lane, alpha, psum);
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {   // some head's running max moved
            float alpha_r[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) alpha_r[r] = __shfl(alpha, 4 * grp + r);
#pragma unroll
            for (int nt = 0; nt < kWaveNT; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r) o[nt][r] *= alpha_r[r];
        }

        // ---- O[:, 128w + 16nt ..] += P . c ----
        // P.V contracts over tokens, so its B-operand is the transpose of the
        // loaded pieces: lane (grp, j) needs tokens 8grp .. 8grp+7 of dim
        // 128w + 16nt + j.  ds_read_b64_tr_b16 gives, within each 16-lane
        // group, element e of lane l from element l % 4 of the 8 bytes at the
        // address of lane 4e + l / 4; with tr_off, each read returns token
        // rows 4grp .. 4grp+3 of one M-tile, i.e. tokens 8grp + 4mt + e.
#pragma unroll
        for (int nt = 0; nt < kWaveNT; ++nt) {
            typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
            const uint8_t *src = trbuf + tr_off + 2048 * (nt >> 1) + 512 * (nt & 1);
            const s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)src);
            const s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(src + 1024));
            const bf16x8 bv = __builtin_bit_cast(bf16x8, s16x8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]});
            o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi, bv, o[nt], 0, 0, 0);
            o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo, bv, o[nt], 0, 0, 0);
        }
    };

    Stage st0;
    const int t0 = sub_begin + team;
    load_tile(t0, st0);
    const int rounds = (sub_end - sub_begin + 1) >> 1;   // same for both teams
    int r = 0;
    for (; r < rounds; ++r) step(t0 + 2 * r, st0);

    // ---- merge the two teams, normalise, write this wavefront's 128 columns ----
    // Each lane holds rows r = 0..3 (heads 4 grp + r) of 8 columns; team t
    // merges and stores rows 2t and 2t + 1, the other team's values of
    // those rows coming through LDS, so both teams share the stores.
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);                  // head n, in every lane of column n
    __syncthreads();                                 // s_part is free
    float *xs = reinterpret_cast<float *>(&s_part[0][0][0][0][0]);
    // rows of merging team mt, row rr (of its two), N-tile nt: 64 lanes contiguous
    auto slot = [&](int mt, int rr, int nt) { return xs + (((mt * 4 + wave) * 2 + rr) * kWaveNT + nt) * 64 + lane; };
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
#pragma unroll
        for (int nt = 0; nt < kWaveNT; ++nt) *slot(1 - team, rr, nt) = team == 0 ? o[nt][2 + rr] : o[nt][rr];
    if (wave == 0 && grp == 0) {
        s_mt[team][n] = m_run;
        s_lt[team][n] = l_tot;
    }
    __syncthreads();
    const int part = p.chunk_begin[i] + c;
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
        const int h = 4 * grp + 2 * team + rr;
        const float m0 = __shfl(m_run, h), l0 = __shfl(l_tot, h);   // this team's (-inf if it read no tile)
        const float m1 = s_mt[1 - team][h], l1 = s_lt[1 - team][h];
        const float M = fmaxf(m0, m1);                  // finite: team 0 reads at least one tile
        const float w0 = m0 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m0 - M);
        const float w1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
        const float den = w0 * l0 + w1 * l1;
        const float inv = 1.f / den;
        if (h < H) {
            float *dst = p.part_o + ((int64_t)part * H + h) * kLatent + 128 * wave + n;
#pragma unroll
            for (int nt = 0; nt < kWaveNT; ++nt) {
                const float own = team == 0 ? o[nt][rr] : o[nt][2 + rr];
                dst[16 * nt] = (w0 * own + w1 * *slot(team, rr, nt)) * inv;
            }
        }
    }
    if (team == 0 && wave == 0 && grp == 0 && n < H) {
        const float m1 = s_mt[1][n], l1 = s_lt[1][n];
        const float M = fmaxf(m_run, m1);
        const float den = __builtin_amdgcn_exp2f(m_run - M) * l_tot +
                          (m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M) * l1);
        p.part_lse[(int64_t)part * H + n] = (M + __log2f(den)) * 0.69314718055994530942f;
    }
}

}  // namespace

hipError_t launch_mla_attend(const AttendParams &p, int n_wg, hipStream_t s) {
    if (n_wg <= 0) return hipSuccess;
    hipLaunchKernelGGL(mla_attend_kernel, dim3(n_wg), dim3(512), 0, s, p);
    return hipGetLastError();
}

}  // namespace wsk
