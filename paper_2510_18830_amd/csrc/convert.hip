// bf16 -> fp16 copies of the attention operands, each times a power of two
// chosen from the tensor's max magnitude (V for the forward; Q, K, V and s dO
// for the backward).  The attention kernels stage every tile as a plain row
// copy, read row-wise or transposed from LDS, and fold the scales back in
// exactly.  Exact for |x| * mul in [2^-14, 65504]; smaller magnitudes round as
// fp16 subnormals.
#include "common.h"
#include "kernels.h"
#include "trace.h"

namespace msparse {

namespace {

constexpr int kCvtThreads = 256;
constexpr int kCvtBlocks = 4096;

// max |x| over n8 chunks of 8 bf16 values into *maxbits (fp32 bits, atomic
// max; the caller zeroes it first).  NaN compares above inf: the scale is then 1.
__global__ void __launch_bounds__(kCvtThreads) absmax_kernel(const uint16_t* __restrict__ src, int64_t n8,
                                                             uint32_t* maxbits) {
    __shared__ uint32_t wmax[kCvtThreads / 64];
    uint32_t m = 0;
    for (int64_t i = int64_t(blockIdx.x) * kCvtThreads + threadIdx.x; i < n8; i += int64_t(gridDim.x) * kCvtThreads) {
        const u32x4 x = reinterpret_cast<const u32x4*>(src)[i];
        m = max(m, max(max(x.x & 0x7fffu, (x.x >> 16) & 0x7fffu), max(x.y & 0x7fffu, (x.y >> 16) & 0x7fffu)));
        m = max(m, max(max(x.z & 0x7fffu, (x.z >> 16) & 0x7fffu), max(x.w & 0x7fffu, (x.w >> 16) & 0x7fffu)));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = max(m, uint32_t(__shfl_xor(int(m), o)));
    if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t b = 0;
        for (int w = 0; w < kCvtThreads / 64; ++w) b = max(b, wmax[w]);
        atomicMax(maxbits, b << 16);   // bf16 magnitude bits -> fp32 bits
    }
}

// 8 elements (16 bytes) per thread and step, grid-stride; `maxbits` (may be
// NULL: factor 1) selects the power-of-two factor, max |x| * mul in
// [2^(E-1), 2^E).
template <int E>
__global__ void __launch_bounds__(kCvtThreads) to_f16_kernel(const uint16_t* __restrict__ src,
                                                             uint16_t* __restrict__ dst, int64_t n8,
                                                             const uint32_t* maxbits) {
    const float mul = maxbits ? pow2_scale_to<E>(maxbits) : 1.f;
    for (int64_t i = int64_t(blockIdx.x) * kCvtThreads + threadIdx.x; i < n8; i += int64_t(gridDim.x) * kCvtThreads) {
        const u32x4 x = reinterpret_cast<const u32x4*>(src)[i];
        u32x4 y;
        y.x = pack_f16x2(bf16_lo(x.x) * mul, bf16_hi(x.x) * mul);
        y.y = pack_f16x2(bf16_lo(x.y) * mul, bf16_hi(x.y) * mul);
        y.z = pack_f16x2(bf16_lo(x.z) * mul, bf16_hi(x.z) * mul);
        y.w = pack_f16x2(bf16_lo(x.w) * mul, bf16_hi(x.w) * mul);
        reinterpret_cast<u32x4*>(dst)[i] = y;
    }
}

}  // namespace

static unsigned cvt_grid(int64_t n8) {
    const int64_t want = (n8 + kCvtThreads - 1) / kCvtThreads;
    return unsigned(want < kCvtBlocks ? want : kCvtBlocks);
}

hipError_t launch_absmax(const uint16_t* src, int64_t n, uint32_t* maxbits, hipStream_t s) {
    const int64_t n8 = n / 8;   // callers pass multiples of 64 elements
    if (n8 <= 0) return hipSuccess;
    TraceScope _t("absmax", s);
    hipLaunchKernelGGL(absmax_kernel, dim3(cvt_grid(n8)), dim3(kCvtThreads), 0, s, src, n8, maxbits);
    return hipGetLastError();
}

hipError_t launch_to_f16(const uint16_t* src, uint16_t* dst, int64_t n, const uint32_t* maxbits, int exp,
                         hipStream_t s) {
    const int64_t n8 = n / 8;
    if (n8 <= 0) return hipSuccess;
    TraceScope _t("to_f16", s);
    if (exp == kOperandExp)
        hipLaunchKernelGGL(to_f16_kernel<kOperandExp>, dim3(cvt_grid(n8)), dim3(kCvtThreads), 0, s, src, dst, n8,
                           maxbits);
    else
        hipLaunchKernelGGL(to_f16_kernel<4>, dim3(cvt_grid(n8)), dim3(kCvtThreads), 0, s, src, dst, n8, maxbits);
    return hipGetLastError();
}

}  // namespace msparse
