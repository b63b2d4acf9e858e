// Device helpers of the small kernels: vector types, bf16 widening,
// and the placement of one K/V (GQA) or latent (MLA) row into the GPU
// pool's tile formats.  Device code only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wsk_internal.h"

namespace wsk {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Places 16-byte piece k (dims 8k..8k+7) of the K (which = 0) or V row of
// token `row` of one KV head into the GPU pool's TILED64 format; `head`
// points at the head's first tile in the slot.  A tile is 1024 K pieces then
// 1024 V pieces of 8 bf16, in the order the attention kernel's matrix-core
// lanes read them (see attend_gqa.hip).
__device__ __forceinline__ void put_tiled(uint16_t *head, int row, int which, int k, u32x4 v) {
    uint16_t *tile = head + (int64_t)(row >> 6) * (2 * 64 * 128);
    const int t = row & 63;
    if (which == 0) {
        const int mt = 2 * (t >> 5) + ((t & 7) >> 2);
        const int nk = 4 * ((t & 31) >> 3) + (t & 3);
        const int piece = (4 * mt + (k >> 2)) * 64 + 16 * (k & 3) + nk;
        *reinterpret_cast<u32x4 *>(tile + piece * 8) = v;
    } else {
        uint16_t *vt = tile + 1024 * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int d = 8 * k + e;
            const int piece = (2 * (d >> 4) + (t >> 5)) * 64 + 16 * ((t & 31) >> 3) + (d & 15);
            vt[piece * 8 + (t & 7)] = (uint16_t)((e & 1) ? (v[e >> 1] >> 16) : (v[e >> 1] & 0xffffu));
        }
    }
}

// Places 16-byte piece c (dims 8c..8c+7) of the MLA row of token `row` into
// a GPU-pool slot in the MLA32 format: 32-token tiles of 2304 pieces, piece
// (ks, mt, lane) being what matrix-core lane (lane / 16, lane % 16) of M-tile
// mt loads for K-step ks (see attend_mla.hip).
__device__ __forceinline__ void put_mla32(uint16_t *slot, int row, int c, u32x4 v) {
    uint16_t *tile = slot + (int64_t)(row >> 5) * (32 * (kLatent + kRope));
    const int u = row & 31;
    const int piece = (2 * (c >> 2) + ((u >> 2) & 1)) * 64 + 16 * (c & 3) + 4 * (u >> 3) + (u & 3);
    *reinterpret_cast<u32x4 *>(tile + piece * 8) = v;
}

// The inverse placements: 16-byte piece k (dims 8k..8k+7) of the K
// (which = 0) or V row of token `row` of one KV head, read from the TILED64
// format; V is stored transposed (8 tokens of one dim per piece), so its row
// piece gathers one element from each of 8 pieces.
__device__ __forceinline__ u32x4 get_tiled(const uint16_t *head, int row, int which, int k) {
    const uint16_t *tile = head + (int64_t)(row >> 6) * (2 * 64 * 128);
    const int t = row & 63;
    if (which == 0) {
        const int mt = 2 * (t >> 5) + ((t & 7) >> 2);
        const int nk = 4 * ((t & 31) >> 3) + (t & 3);
        const int piece = (4 * mt + (k >> 2)) * 64 + 16 * (k & 3) + nk;
        return *reinterpret_cast<const u32x4 *>(tile + piece * 8);
    }
    const uint16_t *vt = tile + 1024 * 8;
    uint32_t w[4];
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
        uint32_t lohi[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int d = 8 * k + 2 * e2 + h;
            const int piece = (2 * (d >> 4) + (t >> 5)) * 64 + 16 * ((t & 31) >> 3) + (d & 15);
            lohi[h] = vt[piece * 8 + (t & 7)];
        }
        w[e2] = lohi[0] | (lohi[1] << 16);
    }
    return u32x4{w[0], w[1], w[2], w[3]};
}

// Piece c (dims 8c..8c+7) of the MLA row of token `row` of an MLA32 slot.
__device__ __forceinline__ u32x4 get_mla32(const uint16_t *slot, int row, int c) {
    const uint16_t *tile = slot + (int64_t)(row >> 5) * (32 * (kLatent + kRope));
    const int u = row & 31;
    const int piece = (2 * (c >> 2) + ((u >> 2) & 1)) * 64 + 16 * (c & 3) + 4 * (u >> 3) + (u & 3);
    return *reinterpret_cast<const u32x4 *>(tile + piece * 8);
}

}  // namespace wsk
