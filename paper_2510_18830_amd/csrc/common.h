// Shared device helpers for the gfx950 kernels: bf16 packing, MFMA wrappers,
// wavefront reductions, ring-layout block maps and the launch-error plumbing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/msparse.h"

namespace msparse {

constexpr int kBlock = 64;   // token block edge (Section 4.1 (ii))
constexpr int kWave = 64;    // CDNA wavefront width

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(4))) int32_t i32x4;

// ---------------------------------------------------------------- bf16 <-> fp32
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;

// fp32 pair -> packed bf16 / fp16, round to nearest even (one v_cvt_pk_* each)
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2 v;
    v.x = (__bf16)lo;
    v.y = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    f16x2 v;
    v.x = (_Float16)lo;
    v.y = (_Float16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// Read-only index data (lists, maps) through the constant address space: a
// wave-uniform address then compiles to a scalar load, which does not share
// the vector-memory counter with in-flight tile loads.
template <class T>
__device__ __forceinline__ T ldc(const T* p, int64_t i) {
    return ((const __attribute__((address_space(4))) T*)(p))[i];
}

// True when the index build that produced the lists ran out of capacity
// (flag may be NULL): the lists are then incomplete and are not walked.
__device__ __forceinline__ bool index_overflowed(const int32_t* flag) { return flag && ldc(flag, 0) != 0; }

// Marks a rarely taken branch as having a side effect, so the compiler keeps
// it a branch instead of turning its body into unconditional selects.
__device__ __forceinline__ void keep_branch() { asm volatile(""); }

// ---------------------------------------------------------------- MFMA
// D(32x32) += A(32x16) * B(16x32), bf16 inputs, fp32 accumulate.
// Lane l supplies A[l%32][8*(l/32) .. +8] and B[8*(l/32) .. +8][l%32];
// accumulator element r of lane l is D[8*(r/4) + 4*(l/32) + r%4][l%32].
__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                  0, 0, 0);
}

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
// Same layout as mfma32, fp16 inputs.
__device__ __forceinline__ f32x16 mfma32h(const u32x4& a, const u32x4& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                 0, 0);
}

// ---------------------------------------------------------------- math
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// x combined with the value of lane l ^ 32 (the other half of the wave) by a
// symmetric operation, through v_permlane32_swap: a VALU exchange of the two
// halves, where __shfl_xor(x, 32) would be an LDS permute with its round trip.
// The swap of x with itself leaves {x[l], x[l ^ 32]} in the two results (in
// lane-dependent order), so max and sum come out the same in both halves.
__device__ __forceinline__ float half_swap_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Power-of-two factor s with max |s x| in [8, 16) given max |x| as fp32 bits;
// 1 for zero or non-finite input.
// Power of two s with max * s in [2^(E-1), 2^E), from the fp32 bits of a
// non-negative max (1 when it is 0 or not finite).  Multiplying by s is exact.
template <int E>
__device__ __forceinline__ float pow2_scale_to(const uint32_t* maxbits) {
    const float mx = __uint_as_float(*maxbits);
    if (!(mx > 0.f) || !isfinite(mx)) return 1.f;
    int e;
    frexpf(mx, &e);           // mx = f 2^e, f in [0.5, 1)
    return ldexpf(1.f, max(-100, min(100, E - e)));
}
// dO: max |s dO| in [8, 16), so s dP, s Delta and s dZ stay inside fp16
__device__ __forceinline__ float pow2_scale(const uint32_t* maxbits) { return pow2_scale_to<4>(maxbits); }
// dZ scale of the backward: the power of two t with t d max|V| in
// [2^9, 2^10).  The fp16 operand t s dZ then satisfies |t s dZ| = t P
// |s dP - s Delta| <= t 2 max|s dO| d max|V| < 2^15 (P <= 1, max|s dO| < 16,
// and |dP|, |Delta| <= max|dO| d max|V|, O being a convex combination of V
// rows): inside the fp16 range whatever the scale of V, and the same fp16
// values for V times any power of two (t = 1 for unit-normal V at d = 128).
// vmaxbits: max |V| as fp32 bits; 1 when it is 0 or not finite.
__device__ __forceinline__ float dz_scale(const uint32_t* vmaxbits, int d) {
    const float mx = __uint_as_float(*vmaxbits) * float(d);
    if (!(mx > 0.f) || !isfinite(mx)) return 1.f;
    int e;
    frexpf(mx, &e);           // mx in [2^(e-1), 2^e)
    return ldexpf(1.f, max(-100, min(100, 10 - e)));
}
// fp16 copies of Q, K, V: max in [2^14, 2^15) (exact conversion of every bf16
// value down to 2^-29 of the max; products stay far inside fp32)
constexpr int kOperandExp = 15;
__device__ __forceinline__ float operand_scale(const uint32_t* maxbits) { return pow2_scale_to<kOperandExp>(maxbits); }

// ---------------------------------------------------------------- ring layout
// Global 64-token blocks are dealt to `world` workers (Section 4.2).
struct Layout {
    int32_t world, nb, layout;  // nb = global block count

    __host__ __device__ int32_t owner(int32_t g) const {
        if (world == 1) return 0;
        if (layout == MSPARSE_LAYOUT_STRIPED) return g % world;
        int32_t c = g / (nb / (2 * world));
        return c < world ? c : 2 * world - 1 - c;
    }
    // local block number of global block g inside its owner
    __host__ __device__ int32_t local(int32_t g) const {
        if (world == 1) return g;
        if (layout == MSPARSE_LAYOUT_STRIPED) return g / world;
        int32_t chunk = nb / (2 * world);
        int32_t c = g / chunk;
        return c < world ? g - c * chunk : chunk + (g - c * chunk);
    }
    // global block number of local block l of worker w
    __host__ __device__ int32_t global(int32_t w, int32_t l) const {
        if (world == 1) return l;
        if (layout == MSPARSE_LAYOUT_STRIPED) return l * world + w;
        int32_t chunk = nb / (2 * world);
        return l < chunk ? w * chunk + l : (2 * world - 1 - w) * chunk + (l - chunk);
    }
};

}  // namespace msparse
