// Achievable MFMA rate (measurement): independent chains of the 32x32x16 fp16
// MFMA that the attention kernels use, with no memory traffic in the loop and
// no VALU work between the MFMAs, on constant or on random operands (the
// matrix cores' power, and so the clock under the power limit, depends on how
// much the operand bits switch).  The caller times one launch with HIP events
// and divides 4 * 2 * 32 * 32 * 16 * iters FLOPs per wave by the duration.
#include "../../include/msparse.h"
#include "common.h"

namespace msparse {

namespace {

// counter-based hash (lowbias32 constants) for the random operands
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// random: eight operand pairs of random fp16 values (random sign and
// mantissa, magnitude in [0.5, 1)), cycled from MFMA to MFMA, so that the
// matrix cores switch as they do on real data; otherwise one constant pair
constexpr int kSets = 8;

__global__ void __launch_bounds__(256) mfma_peak_kernel(float* out, int32_t iters, int32_t random) {
    f32x16 acc[4] = {};
    u32x4 a[kSets], b[kSets];
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
#pragma unroll
    for (int s = 0; s < kSets; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a[s][i] = random ? (mix32(t * 97u + 13u * s + i) & 0x83FF83FFu) | 0x38003800u
                             : 0x3C003C00u ^ (threadIdx.x << 3);   // finite fp16 pairs
            b[s][i] = random ? (mix32(t * 89u + 7u * s + i + 1000u) & 0x83FF83FFu) | 0x38003800u : 0x38003800u + i;
        }
    for (int32_t it = 0; it < iters; it += kSets) {
#pragma unroll
        for (int s = 0; s < kSets; ++s)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[c] = mfma32h(a[s], b[(s + c) % kSets], acc[c]);
    }
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += acc[c][r];
    out[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = sum;
}

}  // namespace

}  // namespace msparse

extern "C" {

int32_t msparse_mfma_peak_probe(int32_t waves_per_simd, int32_t iters, int32_t random_operands, float* out,
                                void* stream) {
    if (waves_per_simd < 1 || waves_per_simd > 8 || iters < 1 || iters % 8 != 0 || !out) return MSPARSE_ERR_INVALID;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return MSPARSE_ERR_HIP;
    // 256 threads = one wave per SIMD of a CU; waves_per_simd workgroups per CU
    hipLaunchKernelGGL(msparse::mfma_peak_kernel, dim3(unsigned(cus * waves_per_simd)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), out, iters, random_operands ? 1 : 0);
    return hipGetLastError() == hipSuccess ? MSPARSE_OK : MSPARSE_ERR_HIP;
}

}  // extern "C"
