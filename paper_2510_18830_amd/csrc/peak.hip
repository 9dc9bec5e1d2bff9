// Achievable MFMA rate (measurement): independent chains of the 32x32x16 fp16
// MFMA that the attention kernels use, with no memory traffic in the loop and
// no VALU work between the MFMAs.  The caller times one launch with HIP events
// and divides 4 * 2 * 32 * 32 * 16 * iters FLOPs per wave by the duration.
#include "../../include/msparse.h"
#include "common.h"

namespace msparse {

namespace {

__global__ void __launch_bounds__(256) mfma_peak_kernel(float* out, int32_t iters) {
    f32x16 acc[4] = {};
    u32x4 a, b;
    for (int i = 0; i < 4; ++i) {
        a[i] = 0x3C003C00u ^ (threadIdx.x << 3);   // finite fp16 pairs
        b[i] = 0x38003800u + i;
    }
    for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = mfma32h(a, b, acc[c]);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

}  // namespace

}  // namespace msparse

extern "C" {

int32_t msparse_mfma_peak_probe(int32_t waves_per_simd, int32_t iters, float* out, void* stream) {
    if (waves_per_simd < 1 || waves_per_simd > 8 || iters < 1 || !out) return MSPARSE_ERR_INVALID;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return MSPARSE_ERR_HIP;
    // 256 threads = one wave per SIMD of a CU; waves_per_simd workgroups per CU
    hipLaunchKernelGGL(msparse::mfma_peak_kernel, dim3(unsigned(cus * waves_per_simd)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), out, iters);
    return hipGetLastError() == hipSuccess ? MSPARSE_OK : MSPARSE_ERR_HIP;
}

}  // extern "C"
