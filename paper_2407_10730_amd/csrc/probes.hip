// probes.hip -- roofline probes of the conv2d library (measurement only).
//
// The roofline fractions the library reports divide by AMD's published peaks; these
// probes measure what the chip delivers on the same box, so that both can be reported
// side by side:
//  * an MFMA issue loop (fp32 32x32x2 or bf16 32x32x16) on register operands, four
//    independent accumulators per wave, two blocks of four waves per CU;
//  * a plain device copy with 16-byte accesses, which also serves to push the working
//    set of a timed call out of the caches (the 256 MiB memory-side cache included)
//    before a cold-cache run.
#include "device_common.h"

namespace cv {

template <bool BF16>
__global__ __launch_bounds__(256) void mfma_probe_kernel(float* sink, int64_t iters) {
    const int t = threadIdx.x;
    f32x16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.0f;
    // operands depend on the thread so the loop cannot be folded; values stay small
    const float fa = 1.0f + (float)(t & 7) * 0x1p-10f, fb = 1.0f - (float)(t & 3) * 0x1p-11f;
    if constexpr (BF16) {
        const uint32_t pa = (uint32_t)f32_to_bf16_rne(fa) * 0x10001u, pb = (uint32_t)f32_to_bf16_rne(fb) * 0x10001u;
        const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{pa, pa, pa, pa});
        const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{pb, pb, pb, pb});
        for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
        }
    } else {
        for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa, fb, acc[j], 0, 0, 0);
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) s += acc[j][v];
    sink[(int64_t)blockIdx.x * 256 + t] = s;
}

// dst[i] = src[i] for n 16-byte units, one unit per thread (measured faster on this chip
// than grid-stride loops with several loads in flight per thread)
__global__ __launch_bounds__(256) void copy_probe_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
                                                         int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = src[i];
}

}  // namespace cv

using namespace cv;

extern "C" int conv2d_probe_mfma(int dtype, int64_t iters, void* sink, int64_t sink_bytes, void* stream,
                                 double* flops) {
    if (!sink || !flops) return CONV2D_E_NULL;
    if ((dtype != CONV2D_F32 && dtype != CONV2D_BF16) || iters < 1) return CONV2D_E_INVALID;
    int dev = -1, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return CONV2D_E_HIP;
    const int blocks = 2 * cus;
    if (sink_bytes < (int64_t)blocks * 256 * 4) return CONV2D_E_INVALID;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == CONV2D_BF16)
        hipLaunchKernelGGL((mfma_probe_kernel<true>), dim3(blocks), dim3(256), 0, s, static_cast<float*>(sink), iters);
    else
        hipLaunchKernelGGL((mfma_probe_kernel<false>), dim3(blocks), dim3(256), 0, s, static_cast<float*>(sink), iters);
    if (hipGetLastError() != hipSuccess) return CONV2D_E_HIP;
    // 4 MFMAs per wave per iteration: 32x32x16 (bf16) or 32x32x2 (fp32) multiply-adds
    const double per_mfma = dtype == CONV2D_BF16 ? 2.0 * 32 * 32 * 16 : 2.0 * 32 * 32 * 2;
    *flops = (double)blocks * 4 /* waves */ * 4 /* MFMAs */ * (double)iters * per_mfma;
    return CONV2D_OK;
}

extern "C" int conv2d_probe_copy(void* dst, const void* src, int64_t bytes, void* stream) {
    if (!dst || !src) return CONV2D_E_NULL;
    if (bytes < 16 || bytes % 16 != 0) return CONV2D_E_INVALID;
    const int64_t n = bytes / 16;
    const int64_t blocks = (n + 255) / 256;
    if (blocks > 0x7fffffffLL) return CONV2D_E_INVALID;
    hipLaunchKernelGGL(copy_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<u32x4*>(dst), static_cast<const u32x4*>(src), n);
    return hipGetLastError() == hipSuccess ? CONV2D_OK : CONV2D_E_HIP;
}
