// LDS staging of 64-row tiles shared by the attention kernels.
//
// A tile is 64 rows of one head: a 64 x 64 block of the grid, or up to 64
// gathered vertical columns (key rows named by an index list).  It is staged
// two ways:
//   row-major  X[row][d]        (operand whose contraction runs over d)
//   transposed Xt[d][pos(row)]  (operand whose contraction runs over rows)
// The transposed copy stores each 16-row group in the order
//   rows 0-3, 8-11, 4-7, 12-15
// because a 32x32 MFMA accumulator gives lane half h the rows
// 8*(r/4) + 4*h + r%4; reading 8 consecutive positions at offset 8*h of a
// 16-group then yields exactly the rows that the same lane holds in its
// accumulator, so P (or dZ) feeds the next MFMA straight from registers.
//
// The transposed copy is converted to fp16 (times a power-of-two factor) for
// the second GEMM of each pair (P V, P^T dO, dZ K, dZ^T Q): fp16 holds 3 more
// significand bits than bf16, which keeps the rounding of P and dZ far below
// the gradient tolerance at the same MFMA rate.
#pragma once

#include "common.h"

namespace msparse {

template <int D>
struct TileLds {
    static constexpr int kRowStride = D + 8;    // 16-bit elements per row-major row
    static constexpr int kTStride = 64 + 8;     // 16-bit elements per transposed row
    static constexpr int kRowElems = 64 * kRowStride;
    static constexpr int kTElems = D * kTStride;
};

// fp16 row-major tiles read through transposing loads: row stride D + 16
// elements, so the reads of a 16-lane group (4 rows x 32 bytes) hit distinct
// banks.
template <int D>
struct F16Tile {
    static constexpr int kStride = D + 16;
    static constexpr int kElems = 64 * kStride;
};

// position of row k (0..63) inside a transposed row
__device__ __forceinline__ int tpos(int k) {
    const int a = (k >> 2) & 3;
    const int sw = ((a & 1) << 1) | (a >> 1);
    return (k & ~15) | (sw << 2) | (k & 3);
}

// Row sources: rows named by an LDS index list, or a contiguous run.
struct IndexedRows {
    const int32_t* idx;
    __device__ __forceinline__ int64_t operator()(int r) const { return idx[r]; }
};
struct ContiguousRows {
    int64_t base;
    __device__ __forceinline__ int64_t operator()(int r) const { return base + r; }
};

// Row-major staging of 64 rows x D bf16 (row length D in `src`).
template <int D, int NT, class Rows, int RS = TileLds<D>::kRowStride>
__device__ __forceinline__ void stage_rows(uint16_t* lds, const uint16_t* __restrict__ src, Rows rows, int tid) {
    constexpr int kChunks = D / 8;              // 16-byte chunks per row
    constexpr int kRowsPerPass = NT / kChunks;
#pragma unroll
    for (int p = 0; p < 64 / kRowsPerPass; ++p) {
        const int r = p * kRowsPerPass + tid / kChunks;
        const int c = tid % kChunks;
        const u32x4 v = *reinterpret_cast<const u32x4*>(src + rows(r) * D + c * 8);
        *reinterpret_cast<u32x4*>(lds + r * RS + c * 8) = v;
    }
}

// Transposed staging Xt[d][tpos(row)] (row stride TS elements), converted to
// fp16 after multiplying by `mul` (a power of two).
template <int D, int NT, class Rows, int TS = TileLds<D>::kTStride>
__device__ __forceinline__ void stage_transposed_f16(uint16_t* lds, const uint16_t* __restrict__ src, Rows rows,
                                                     float mul, int tid) {
    constexpr int kItems = 16 * (D / 8);  // (4-row quad) x (8-wide d chunk)
#pragma unroll
    for (int p = 0; p < (kItems + NT - 1) / NT; ++p) {
        const int item = p * NT + tid;
        if (kItems % NT != 0 && item >= kItems) break;
        const int q4 = item & 15;
        const int dc = item >> 4;
        u32x4 r[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) r[b] = *reinterpret_cast<const u32x4*>(src + rows(4 * q4 + b) * D + dc * 8);
        const int pos = tpos(4 * q4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            u32x2 even, odd;
            even.x = bf16_to_f16_bits(r[0][e] & 0xffffu, mul) | (bf16_to_f16_bits(r[1][e] & 0xffffu, mul) << 16);
            even.y = bf16_to_f16_bits(r[2][e] & 0xffffu, mul) | (bf16_to_f16_bits(r[3][e] & 0xffffu, mul) << 16);
            odd.x = bf16_to_f16_bits(r[0][e] >> 16, mul) | (bf16_to_f16_bits(r[1][e] >> 16, mul) << 16);
            odd.y = bf16_to_f16_bits(r[2][e] >> 16, mul) | (bf16_to_f16_bits(r[3][e] >> 16, mul) << 16);
            const int d0 = dc * 8 + 2 * e;
            *reinterpret_cast<u32x2*>(lds + d0 * TS + pos) = even;
            *reinterpret_cast<u32x2*>(lds + (d0 + 1) * TS + pos) = odd;
        }
    }
}

// Two-phase staging for software pipelining: the global loads of a tile go to
// registers first (issued before the current tile's compute), the LDS stores
// (with the fp16 conversion of the transposed copy) follow after it.
template <int D, int NT>
struct RowRegs {
    static constexpr int kChunks = D / 8;
    static constexpr int kRowsPerPass = NT / kChunks;
    static constexpr int kPasses = 64 / kRowsPerPass;
    u32x4 r[kPasses];
};
template <int D, int NT, class Rows>
__device__ __forceinline__ void load_rows(RowRegs<D, NT>& g, const uint16_t* __restrict__ src, Rows rows, int tid) {
    using R = RowRegs<D, NT>;
#pragma unroll
    for (int p = 0; p < R::kPasses; ++p) {
        const int r = p * R::kRowsPerPass + tid / R::kChunks;
        g.r[p] = *reinterpret_cast<const u32x4*>(src + rows(r) * D + (tid % R::kChunks) * 8);
    }
}
template <int D, int NT, int RS = TileLds<D>::kRowStride>
__device__ __forceinline__ void store_rows(uint16_t* lds, const RowRegs<D, NT>& g, int tid) {
    using R = RowRegs<D, NT>;
#pragma unroll
    for (int p = 0; p < R::kPasses; ++p) {
        const int r = p * R::kRowsPerPass + tid / R::kChunks;
        *reinterpret_cast<u32x4*>(lds + r * RS + (tid % R::kChunks) * 8) = g.r[p];
    }
}
// transposed staging: item = (4-row quad, 8-wide d chunk), 16 * D / 8 items
template <int D, int NT>
struct TransRegs {
    static constexpr int kItems = 16 * (D / 8);
    static constexpr int kPasses = (kItems + NT - 1) / NT;
    u32x4 r[kPasses][4];
};
template <int D, int NT, class Rows>
__device__ __forceinline__ void load_trans(TransRegs<D, NT>& g, const uint16_t* __restrict__ src, Rows rows, int tid) {
    using R = TransRegs<D, NT>;
#pragma unroll
    for (int p = 0; p < R::kPasses; ++p) {
        const int item = p * NT + tid;
        if (R::kItems % NT != 0 && item >= R::kItems) break;
        const int q4 = item & 15, dc = item >> 4;
#pragma unroll
        for (int b = 0; b < 4; ++b) g.r[p][b] = *reinterpret_cast<const u32x4*>(src + rows(4 * q4 + b) * D + dc * 8);
    }
}
template <int D, int NT, int TS = TileLds<D>::kTStride>
__device__ __forceinline__ void store_trans_f16(uint16_t* lds, const TransRegs<D, NT>& g, float mul, int tid) {
    using R = TransRegs<D, NT>;
#pragma unroll
    for (int p = 0; p < R::kPasses; ++p) {
        const int item = p * NT + tid;
        if (R::kItems % NT != 0 && item >= R::kItems) break;
        const int q4 = item & 15, dc = item >> 4;
        const int pos = tpos(4 * q4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const u32x4* r = g.r[p];
            u32x2 even, odd;
            even.x = bf16_to_f16_bits(r[0][e] & 0xffffu, mul) | (bf16_to_f16_bits(r[1][e] & 0xffffu, mul) << 16);
            even.y = bf16_to_f16_bits(r[2][e] & 0xffffu, mul) | (bf16_to_f16_bits(r[3][e] & 0xffffu, mul) << 16);
            odd.x = bf16_to_f16_bits(r[0][e] >> 16, mul) | (bf16_to_f16_bits(r[1][e] >> 16, mul) << 16);
            odd.y = bf16_to_f16_bits(r[2][e] >> 16, mul) | (bf16_to_f16_bits(r[3][e] >> 16, mul) << 16);
            const int d0 = dc * 8 + 2 * e;
            *reinterpret_cast<u32x2*>(lds + d0 * TS + pos) = even;
            *reinterpret_cast<u32x2*>(lds + (d0 + 1) * TS + pos) = odd;
        }
    }
}

// ---------------------------------------------------------------- DMA tiles
// 64 rows x D 16-bit elements filled by direct global->LDS loads.  One wave
// instruction writes 64 lanes x 16 bytes contiguously (the lanes free to
// gather any rows), i.e. RPI = 1024 / (2 D) whole rows.  Instruction g of a
// tile carries rows g, g + NG, g + 2 NG, ... (NG = 64 / RPI groups) and the
// groups lie 1024 + P bytes apart:
//   byte offset of (row r, chunk c) = (r % NG) (1024 + P) + (r / NG) 2 D + 16 c.
// Every operand read is then a per-lane base plus immediate offsets.  P = 16
// spreads the 16 rows of a row-wise operand read over distinct banks; P = 64
// does the same for the 4 rows x 32 bytes of each 16-lane group of a
// transposing read (and for two such groups served together).
template <int D, int P>
struct DmaTile {
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kRowsPerInst = 1024 / kRowBytes;   // 4 (D = 128) or 8 (D = 64)
    static constexpr int kGroups = 64 / kRowsPerInst;       // 16 or 8
    static constexpr int kGroupBytes = 1024 + P;
    static constexpr int kBytes = kGroups * kGroupBytes;
    static constexpr int kElems = kBytes / 2;
    __device__ static constexpr int off(int r, int c) {      // element offset of chunk c of row r
        return ((r % kGroups) * kGroupBytes + (r / kGroups) * kRowBytes + 16 * c) / 2;
    }
};
constexpr int kRowPad = 16;   // tiles read row-wise
constexpr int kTrPad = 64;    // tiles read through transposing loads

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// LDS byte address of a pointer into a __shared__ object
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return uint32_t(reinterpret_cast<uintptr_t>((lds_void_ptr)(const_cast<void*>(p))));
}

// One global->LDS DMA instruction: each lane loads 16 bytes from its own
// `src`; lane l's bytes land at LDS byte address `lds` + 16 l (`lds` uniform
// across the wave).  Written as inline assembly so that the compiler adds no
// waits of its own before LDS reads of other buffers; the consumer waits with
// wait_vmem() and publishes the tile with a barrier.
__device__ __forceinline__ void dma16(const void* src, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory", "m0");
}

// Issue the loads of one tile (rows(r), r = 0..63, row length D) into `tile`:
// wave `wave` of NW issues instructions wave, wave + NW, ... < NG.  The data
// lands asynchronously: wait_vmem() before the barrier that publishes it.
template <int D, int P, int NW, class Rows>
__device__ __forceinline__ void dma_rows(uint16_t* tile, const uint16_t* __restrict__ src, Rows rows, int wave,
                                         int lane) {
    using T = DmaTile<D, P>;
    constexpr int NC = D / 8;
#pragma unroll
    for (int j = 0; j < (T::kGroups + NW - 1) / NW; ++j) {
        const int g = wave + NW * j;
        if (T::kGroups % NW != 0 && g >= T::kGroups) break;
        const int r = g + T::kGroups * (lane / NC);
        const int c = lane % NC;
        dma16(src + rows(r) * D + c * 8, lds_addr(tile + g * (T::kGroupBytes / 2)));
    }
}

// wait until this wave's outstanding vector-memory loads (tile DMA included) are done
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// 16 bytes of row r, chunk c of a DMA tile (row-wise MFMA operand)
template <int D, int P>
__device__ __forceinline__ u32x4 dma_read16(const uint16_t* tile, int r, int c) {
    return *reinterpret_cast<const u32x4*>(tile + DmaTile<D, P>::off(r, c));
}

// A operand of a 32x32x16 fp16 MFMA read transposed from a DMA tile of fp16
// rows (same operand as lds_read_tr_a: A[m][k] = X[k0 + kperm(k)][m0 + m]).
template <int D, int P>
__device__ __forceinline__ u32x4 dma_read_tr(const uint16_t* x, int k0, int m0, int lane) {
    typedef short v4s __attribute__((ext_vector_type(4)));
    using T = DmaTile<D, P>;
    const int r0 = k0 + 4 * (lane >> 5) + ((lane & 15) >> 2);
    const int e = m0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);   // element column
    const uint16_t* p0 = x + T::off(r0, 0) + e;
    const uint16_t* p1 = x + T::off(r0 + 8, 0) + e;
    const v4s a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p0));
    const v4s a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p1));
    const u32x2 a = __builtin_bit_cast(u32x2, a0), b = __builtin_bit_cast(u32x2, a1);
    u32x4 o;
    o.x = a.x;
    o.y = a.y;
    o.z = b.x;
    o.w = b.y;
    return o;
}

#ifndef MS_XCHUNK
#define MS_XCHUNK 64   // logical items per XCD run
#endif
// Workgroup ids are dispatched round-robin over the 8 XCDs, each with its own
// L2.  xcd_chunk maps id t to a logical index so that each XCD receives runs
// of C consecutive logical items (the tail past the last full round of 8 runs
// keeps its identity mapping); a bijection on [0, total).
__device__ __forceinline__ int64_t xcd_chunk(int64_t t, int64_t total) {
    constexpr int64_t C = MS_XCHUNK;
    const int64_t full = total / (8 * C) * (8 * C);
    if (t >= full) return t;
    const int64_t n = t >> 3, x = t & 7;
    return (n / C) * 8 * C + x * C + (n % C);
}

// (head, query block) of workgroup t in a B*Hq*nqb grid: KV-group-major
// (the group's heads at one block are neighbours), latest blocks first.
__device__ __forceinline__ void query_tile_of(int64_t t, int B, int Hq, int Hkv, int nqb, int& bh, int& qb) {
    const int64_t u = xcd_chunk(t, int64_t(B) * Hq * nqb);
    const int G = Hq / Hkv;
    const int64_t per = int64_t(nqb) * G;
    const int bg = int(u / per);
    const int64_t r = u % per;
    qb = nqb - 1 - int(r / G);
    bh = (bg / Hkv) * Hq + (bg % Hkv) * G + int(r % G);
}

// A operand of a 32x32x16 fp16 MFMA taken transposed from a row-major fp16
// tile X[row][col] (row stride RS elements): A[m][k] = X[k0 + kperm(k)][m0 + m]
// with kperm the key order of an accumulator-resident B operand (lane half h
// supplies rows k0 + 4h + {0..3} and k0 + 8 + 4h + {0..3}).  Two
// ds_read_b64_tr_b16: in each group of 16 lanes, lane s names 4 consecutive
// elements of row (s / 4) and receives element s % 4 of the rows named by
// lanes s / 4 + 4j, j = 0..3.
template <int RS>
__device__ __forceinline__ u32x4 lds_read_tr_a(const uint16_t* x, int k0, int m0, int lane) {
    typedef short v4s __attribute__((ext_vector_type(4)));
    const int row = k0 + 4 * (lane >> 5) + ((lane & 15) >> 2);
    const int col = m0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const uint16_t* p = x + row * RS + col;
    const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p));
    const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p + 8 * RS));
    const u32x2 a = __builtin_bit_cast(u32x2, r0), b = __builtin_bit_cast(u32x2, r1);
    u32x4 o;
    o.x = a.x;
    o.y = a.y;
    o.z = b.x;
    o.w = b.y;
    return o;
}

// 16-byte LDS read
__device__ __forceinline__ u32x4 lds_read16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// pack 8 consecutive accumulator values (regs base .. base+7) to fp16 x 8
template <int BASE>
__device__ __forceinline__ u32x4 pack8_f16(const f32x16& acc) {
    u32x4 r;
    r.x = pack_f16x2(acc[BASE + 0], acc[BASE + 1]);
    r.y = pack_f16x2(acc[BASE + 2], acc[BASE + 3]);
    r.z = pack_f16x2(acc[BASE + 4], acc[BASE + 5]);
    r.w = pack_f16x2(acc[BASE + 6], acc[BASE + 7]);
    return r;
}

}  // namespace msparse
