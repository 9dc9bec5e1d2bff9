// LDS staging of 64-key tiles shared by the attention kernels.
//
// A "key tile" is 64 key rows of one KV head: either a 64 x 64 block of the
// grid (rows kb*64 .. kb*64 + 63) or up to 64 gathered vertical columns.  It
// is staged two ways:
//   row-major  X[key][d]        (operand whose contraction runs over d)
//   transposed Xt[d][pos(key)]  (operand whose contraction runs over keys)
// The transposed copy stores each 16-key group in the order
//   keys 0-3, 8-11, 4-7, 12-15
// because a 32x32 MFMA accumulator gives lane half h the rows
// 8*(r/4) + 4*h + r%4; reading 8 consecutive positions at offset 8*h of a
// 16-group then yields exactly the keys that the same lane holds in its
// accumulator, so P (or dS) feeds the next MFMA straight from registers.
#pragma once

#include "common.h"

namespace msparse {

template <int D>
struct TileLds {
    static constexpr int kRowStride = D + 8;    // bf16 elements, row-major rows
    static constexpr int kTStride = 64 + 8;     // bf16 elements, transposed rows
    static constexpr int kRowElems = 64 * kRowStride;
    static constexpr int kTElems = D * kTStride;
};

// position of key k (0..63) inside a transposed row
__device__ __forceinline__ int tpos(int k) {
    const int a = (k >> 2) & 3;
    const int sw = ((a & 1) << 1) | (a >> 1);
    return (k & ~15) | (sw << 2) | (k & 3);
}

// Row-major staging: 64 rows x D bf16 from `src` rows kidx[r] (row length D).
template <int D, int NT>
__device__ __forceinline__ void stage_rows(uint16_t* lds, const uint16_t* __restrict__ src, const int32_t* kidx,
                                           int tid) {
    constexpr int kChunks = D / 8;              // 16-byte chunks per row
    constexpr int kRowsPerPass = NT / kChunks;
#pragma unroll
    for (int p = 0; p < 64 / kRowsPerPass; ++p) {
        const int r = p * kRowsPerPass + tid / kChunks;
        const int c = tid % kChunks;
        const u32x4 v = *reinterpret_cast<const u32x4*>(src + int64_t(kidx[r]) * D + c * 8);
        *reinterpret_cast<u32x4*>(lds + r * TileLds<D>::kRowStride + c * 8) = v;
    }
}

// Transposed staging: Xt[d][tpos(key)] for 64 rows kidx[r] of `src`.
template <int D, int NT>
__device__ __forceinline__ void stage_transposed(uint16_t* lds, const uint16_t* __restrict__ src,
                                                 const int32_t* kidx, int tid) {
    constexpr int kItems = 16 * (D / 8);  // (4-key quad) x (8-wide d chunk)
#pragma unroll
    for (int p = 0; p < (kItems + NT - 1) / NT; ++p) {
        const int item = p * NT + tid;
        if (kItems % NT != 0 && item >= kItems) break;
        const int q4 = item & 15;
        const int dc = item >> 4;
        u32x4 r[4];
#pragma unroll
        for (int b = 0; b < 4; ++b)
            r[b] = *reinterpret_cast<const u32x4*>(src + int64_t(kidx[4 * q4 + b]) * D + dc * 8);
        const int pos = tpos(4 * q4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t w0 = r[0][e], w1 = r[1][e], w2 = r[2][e], w3 = r[3][e];
            u32x2 even, odd;
            even.x = (w0 & 0xffffu) | (w1 << 16);
            even.y = (w2 & 0xffffu) | (w3 << 16);
            odd.x = (w0 >> 16) | (w1 & 0xffff0000u);
            odd.y = (w2 >> 16) | (w3 & 0xffff0000u);
            const int d0 = dc * 8 + 2 * e;
            *reinterpret_cast<u32x2*>(lds + d0 * TileLds<D>::kTStride + pos) = even;
            *reinterpret_cast<u32x2*>(lds + (d0 + 1) * TileLds<D>::kTStride + pos) = odd;
        }
    }
}

// 16-byte LDS read
__device__ __forceinline__ u32x4 lds_read16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// pack 8 consecutive accumulator values (regs base .. base+7) to bf16 x 8
__device__ __forceinline__ u32x4 pack8(const f32x16& acc, int base) {
    u32x4 r;
    r.x = pack_bf16x2(acc[base + 0], acc[base + 1]);
    r.y = pack_bf16x2(acc[base + 2], acc[base + 3]);
    r.z = pack_bf16x2(acc[base + 4], acc[base + 5]);
    r.w = pack_bf16x2(acc[base + 6], acc[base + 7]);
    return r;
}

}  // namespace msparse
