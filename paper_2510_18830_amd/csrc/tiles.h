// LDS tiles shared by the attention kernels.
//
// A tile is 64 rows of one head: a 64 x 64 block of the grid, or up to 64
// gathered vertical columns (key rows named by an index list).  The attention
// kernels fill tiles with direct global->LDS loads (DMA tiles below) and read
// them two ways:
//   row-wise      16 bytes of one row per lane: an MFMA operand whose
//                 contraction runs over d (K in S = Q K^T, Q and dO rows)
//   transposed    ds_read_b64_tr_b16 over 16 rows x 32 columns: an MFMA A
//                 operand whose contraction runs over the rows (V^T, K^T, Q^T,
//                 dO^T), from fp16 copies of those tensors
// A 32x32 MFMA accumulator gives lane half h the rows 8(r/4) + 4h + r%4; the
// transposed reads fetch exactly that row order, so P (or dZ) feeds the next
// MFMA straight from registers.  The second GEMM of each pair runs in fp16: 3
// more significand bits than bf16 keep the rounding of P and dZ far below the
// gradient tolerance at the same MFMA rate.
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

// Row sources: rows named by an LDS index list, or a contiguous run.
struct IndexedRows {
    const int32_t* idx;
    __device__ __forceinline__ int64_t operator()(int r) const { return idx[r]; }
};
struct ContiguousRows {
    int64_t base;
    __device__ __forceinline__ int64_t operator()(int r) const { return base + r; }
};

// Row-major staging of 64 rows x D bf16 through registers (row length D in
// `src`), padded rows of RS elements.
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

// ---------------------------------------------------------------- DMA tiles
// 64 rows x D 16-bit elements filled by direct global->LDS loads.  One wave
// instruction writes 64 lanes x 16 bytes contiguously (the lanes free to
// gather any rows), i.e. RPI = 1024 / (2 D) whole rows.  Instruction g of a
// tile carries rows g, g + NG, g + 2 NG, ... (NG = 64 / RPI groups) and the
// groups start at goff(g):
//   byte offset of (row r, chunk c) = goff(r % NG) + (r / NG) 2 D + 16 c.
// Every operand read is then a per-lane base plus immediate offsets.  The LDS
// serves 256 bytes (64 banks x 4 bytes) per cycle: 16 lanes of a row-wise
// 16-byte read, or 32 lanes of a transposing 8-byte read.  With uniform
// spacing goff(g) = g (1024 + P), P = 16 puts the 16 rows of a row-wise
// operand read in distinct banks and P = 64 the 4 rows x 64 bytes of a
// transposing read; no uniform P serves both, hence the placement of the
// tiles read both ways.
template <int D, int P>
struct DmaTile {
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kRowsPerInst = 1024 / kRowBytes;   // 4 (D = 128) or 8 (D = 64)
    static constexpr int kGroups = 64 / kRowsPerInst;       // 16 or 8
    // byte offset of group g: uniform pad P, or (P < 0, tiles read both ways,
    // D = 128) groups placed so that, modulo the 256 bytes one LDS cycle
    // serves, the 16 groups start at distinct multiples of 16 (a row-wise
    // read: 16 lanes, one 16-byte chunk per group) and each quad of groups
    // 4j .. 4j + 3 starts 64 bytes apart (a transposing read: 32 lanes, 64
    // contiguous bytes of each of four groups of one quad); P < 0 at D = 64
    // is a uniform 48-byte pad
    __host__ __device__ static constexpr int goff(int g) {
        return P >= 0 ? g * (1024 + P)
                      : (D == 128 ? 1024 * g + 272 * (g >> 2) + 64 * (g & 3) : g * (1024 + 48));
    }
    static constexpr int kBytes = goff(kGroups - 1) + 1024 + (P >= 0 ? P : (D == 128 ? 0 : 48));
    static constexpr int kElems = kBytes / 2;
    __device__ static constexpr int off(int r, int c) {      // element offset of chunk c of row r
        return (goff(r % kGroups) + (r / kGroups) * kRowBytes + 16 * c) / 2;
    }
};
constexpr int kRowPad = 16;   // tiles read row-wise
constexpr int kTrPad = 64;    // tiles read through transposing loads
constexpr int kDualPad = -1;  // tiles read both ways (group placement above)

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
        dma16(src + rows(r) * D + c * 8, lds_addr(tile + T::goff(g) / 2));
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
#define MS_XCHUNK 8    // longest run of logical items per XCD
#endif
// Workgroup ids are dispatched round-robin over the 8 XCDs, each with its own
// L2.  xcd_chunk maps id t to a logical index so that each XCD receives runs
// of C consecutive logical items, C = MS_XCHUNK halved until every XCD gets
// at least 16 runs (a small grid would otherwise give each XCD one
// contiguous stretch of the sequence, and the causal work falls along it),
// with the XCD order reversed every other round (each XCD gets early and late
// runs alike).  The tail past the last full round keeps its identity mapping;
// a bijection on [0, total).
__device__ __forceinline__ int64_t xcd_chunk(int64_t t, int64_t total) {
    int64_t C = MS_XCHUNK;
    while (C > 1 && total < 8 * 16 * C) C >>= 1;
    const int64_t full = total / (8 * C) * (8 * C);
    if (t >= full) return t;
    const int64_t n = t >> 3, k = n / C;
    const int64_t x = (k & 1) ? 7 - (t & 7) : (t & 7);
    return k * 8 * C + x * C + (n % C);
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

// Sum over a row of the fp16 weights in four packed B operands (32 values per
// lane) plus the partner lane l ^ 32 (the other half of the row's keys), in
// fp32: one v_dot2 per pair, two chains.
__device__ __forceinline__ float row_sum_f16(const u32x4* pb) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const h2 one = {(_Float16)1.f, (_Float16)1.f};
    float a = 0.f, b = 0.f;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        // elements copied out first: a bit cast of an ext_vector element
        // expression reads element 0 under this compiler
        const uint32_t w0 = pb[g].x, w1 = pb[g].y, w2 = pb[g].z, w3 = pb[g].w;
        a = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w0), one, a, false);
        b = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w1), one, b, false);
        a = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w2), one, a, false);
        b = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, w3), one, b, false);
    }
    return half_swap_sum(a + b);
}

}  // namespace msparse
