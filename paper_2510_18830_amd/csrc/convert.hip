// bf16 -> fp16 copies of the operands that enter the fp16 second GEMMs (V for
// the forward; K for dQ; Q and s dO for dK / dV).  The attention kernels then
// stage every tile as a plain row copy and take the transposed operand with a
// transposing LDS read.  Exact for |x| * mul in [2^-14, 65504]; smaller
// magnitudes round as fp16 subnormals.
#include "common.h"
#include "kernels.h"
#include "trace.h"

namespace msparse {

namespace {

constexpr int kCvtThreads = 256;
constexpr int kCvtBlocks = 4096;

// 8 elements (16 bytes) per thread and step, grid-stride; `maxbits` (may be
// NULL) selects the power-of-two factor of pow2_scale.
__global__ void __launch_bounds__(kCvtThreads) to_f16_kernel(const uint16_t* __restrict__ src,
                                                             uint16_t* __restrict__ dst, int64_t n8,
                                                             const uint32_t* maxbits) {
    const float mul = maxbits ? pow2_scale(maxbits) : 1.f;
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

hipError_t launch_to_f16(const uint16_t* src, uint16_t* dst, int64_t n, const uint32_t* maxbits, hipStream_t s) {
    const int64_t n8 = n / 8;   // callers pass multiples of 64 elements
    if (n8 <= 0) return hipSuccess;
    const int64_t want = (n8 + kCvtThreads - 1) / kCvtThreads;
    const unsigned grid = unsigned(want < kCvtBlocks ? want : kCvtBlocks);
    TraceScope _t("to_f16", s);
    hipLaunchKernelGGL(to_f16_kernel, dim3(grid), dim3(kCvtThreads), 0, s, src, dst, n8, maxbits);
    return hipGetLastError();
}

}  // namespace msparse
