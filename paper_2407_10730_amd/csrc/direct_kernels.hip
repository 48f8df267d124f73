// direct_kernels.hip -- direct convolution on the vector ALUs for depthwise and
// small-group layers (NCHW).
//
// Grouped convolutions are the largest non-pointwise class of the paper's
// operation set (Sec. III-B); when C/g is small the reduction (C/g)*R*S is too
// short for matrix cores, so every output is summed with fp32 FMAs.  One block
// covers a band of output rows of one (n, k) plane: the input rows the band
// needs for one input channel are staged once in LDS with a zero halo, then
// each thread sums R*S taps per output from LDS.  Filter taps are
// block-uniform and come through the scalar cache.
#include "conv2d_internal.h"

namespace cv {

#define OOB_OFF 0x80000000u
#define RSRC_WORD3 0x00020000

__device__ __forceinline__ __amdgpu_buffer_rsrc_t dk_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, RSRC_WORD3);
}

// Element `idx` of x as fp32, or zero when !ok (the load then targets no record).
__device__ __forceinline__ float dk_load(__amdgpu_buffer_rsrc_t r, bool ok, int64_t idx, float*) {
    const uint32_t off = ok ? (uint32_t)(idx * 4) : OOB_OFF;
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ float dk_load(__amdgpu_buffer_rsrc_t r, bool ok, int64_t idx, uint16_t*) {
    const uint32_t off = ok ? (uint32_t)(idx * 2) : OOB_OFF;
    const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
    return __builtin_bit_cast(float, h << 16);
}

__device__ __forceinline__ uint16_t dk_f32_to_bf16(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

constexpr int DIRECT_THREADS = 256;
constexpr int DIRECT_LDS_FLOATS = 12288;  // 48 KiB staging buffer

// 1-D grid of nbands * N*K blocks (band fastest).  Band = `rows` output rows; the staged input window is
// in_rows = (rows-1)*sh + (R-1)*dh + 1 rows by in_cols = (Wo-1)*sw + (S-1)*dw + 1 columns.
template <typename TX, typename TY>
__global__ __launch_bounds__(DIRECT_THREADS) void direct_kernel(DirectArgs A, int rows, int in_rows,
                                                                int in_cols, int nbands) {
    __shared__ float tile[DIRECT_LDS_FLOATS];
    const int band = blockIdx.x % nbands;
    const int plane = blockIdx.x / nbands;  // n*K + k
    const int n = plane / A.K;
    const int k = plane - n * A.K;
    const int gi = k / A.Kg;
    const int ho0 = band * rows;
    const int ho_end = min(ho0 + rows, A.Ho);
    const int hi_base = ho0 * A.sh - A.ph;   // first staged input row
    const int wi_base = -A.pw;               // first staged input column
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const TX* wk = reinterpret_cast<const TX*>(A.w) + (int64_t)k * A.Cg * A.R * A.S;

    const int nout = (ho_end - ho0) * A.Wo;
    const int per_thread = (nout + DIRECT_THREADS - 1) / DIRECT_THREADS;
    float acc[4];
    const float b = A.bias ? A.bias[k] : 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = b;

    const int tile_elems = in_rows * in_cols;
    for (int c = 0; c < A.Cg; ++c) {
        const int64_t xplane = ((int64_t)n * A.C + (int64_t)gi * A.Cg + c) * A.H * A.W;
        __syncthreads();
        for (int i = threadIdx.x; i < tile_elems; i += DIRECT_THREADS) {
            const int rr = i / in_cols;
            const int cc = i - rr * in_cols;
            const int hi = hi_base + rr, wi = wi_base + cc;
            const bool ok = ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
            tile[i] = dk_load(rx, ok, xplane + (int64_t)hi * A.W + wi, (TX*)nullptr);
        }
        __syncthreads();
        const TX* wc = wk + c * A.R * A.S;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (q >= per_thread) break;
            const int o = threadIdx.x + q * DIRECT_THREADS;
            if (o >= nout) break;
            const int oh = o / A.Wo;
            const int ow = o - oh * A.Wo;
            const int base = (oh * A.sh) * in_cols + ow * A.sw;
            float s = 0.0f;
            for (int r = 0; r < A.R; ++r) {
                const float* trow = tile + base + r * A.dh * in_cols;
                for (int sx = 0; sx < A.S; ++sx) {
                    float wv;
                    if constexpr (sizeof(TX) == 4) wv = __builtin_bit_cast(float, wc[r * A.S + sx]);
                    else wv = __builtin_bit_cast(float, (uint32_t)wc[r * A.S + sx] << 16);
                    s = __builtin_fmaf(trow[sx * A.dw], wv, s);
                }
            }
            acc[q] += s;
        }
    }
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q >= per_thread) break;
        const int o = threadIdx.x + q * DIRECT_THREADS;
        if (o >= nout) break;
        const int oh = ho0 + o / A.Wo;
        const int ow = o % A.Wo;
        const int64_t off = ((int64_t)plane * A.Ho + oh) * A.Wo + ow;
        if constexpr (sizeof(TY) == 4)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, acc[q]), ry, (uint32_t)(off * 4), 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(acc[q]), ry, (uint32_t)(off * 2), 0, 0);
    }
}

// Output rows per block: as many as fit both the LDS window and 4 outputs per thread.
static int direct_rows(const DirectArgs& a, int* in_rows, int* in_cols) {
    const int ic = (a.Wo - 1) * a.sw + (a.S - 1) * a.dw + 1;
    int rows = (4 * DIRECT_THREADS) / a.Wo;
    if (rows > a.Ho) rows = a.Ho;
    while (rows > 1 && ((rows - 1) * a.sh + (a.R - 1) * a.dh + 1) * ic > DIRECT_LDS_FLOATS) --rows;
    *in_rows = (rows - 1) * a.sh + (a.R - 1) * a.dh + 1;
    *in_cols = ic;
    return rows;
}

hipError_t launch_direct(const DirectArgs& a, int xdt, int ydt, hipStream_t stream) {
    int in_rows = 0, in_cols = 0;
    const int rows = direct_rows(a, &in_rows, &in_cols);
    if (rows < 1 || a.Wo > 4 * DIRECT_THREADS || in_rows * in_cols > DIRECT_LDS_FLOATS)
        return hipErrorInvalidConfiguration;
    const int nbands = (a.Ho + rows - 1) / rows;
    const int64_t nblocks = (int64_t)nbands * a.N * a.K;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((direct_kernel<float, float>), grid, dim3(DIRECT_THREADS), 0, stream, a, rows,
                           in_rows, in_cols, nbands);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((direct_kernel<uint16_t, uint16_t>), grid, dim3(DIRECT_THREADS), 0, stream, a,
                           rows, in_rows, in_cols, nbands);
    else
        hipLaunchKernelGGL((direct_kernel<uint16_t, float>), grid, dim3(DIRECT_THREADS), 0, stream, a,
                           rows, in_rows, in_cols, nbands);
    return hipGetLastError();
}

}  // namespace cv
