// pack_kernels.hip -- packing, unpacking and layout kernels of the conv2d library.
//
//  im2col  : the explicit path's packing step (Sec. I: Im2col-GEMM needs a
//            reordering routine before the GEMM).  col[g][kr][pl] holds input
//            tap kr = (c, r, s) of output pixel p_begin + pl, zero outside.
//  unpack  : the explicit path's result unpacking (Sec. III-A, in-convolution
//            unpacking): the GEMM result C[g][m][pl] becomes y in NCHW, plus
//            bias, cast to the output type.
//  nhwc<->nchw : pre- and post-convolution reordering of x and y.
#include "conv2d_internal.h"

namespace cv {

#define OOB_OFF 0x80000000u
#define RSRC_WORD3 0x00020000

__device__ __forceinline__ __amdgpu_buffer_rsrc_t pk_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, RSRC_WORD3);
}

__device__ __forceinline__ uint16_t pk_f32_to_bf16(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ------------------------------------------------------------------ im2col
// grid (ceil(pc/256), ceil(Kred/KR_PER_BLOCK), G), 256 threads, one pixel per thread.
constexpr int KR_PER_BLOCK = 16;

template <typename T>
__global__ __launch_bounds__(256) void im2col_kernel(Im2colArgs A) {
    const int pl = blockIdx.x * 256 + threadIdx.x;
    const int gi = blockIdx.z;
    const int kr0 = blockIdx.y * KR_PER_BLOCK;
    if (pl >= A.pc) return;
    const int64_t p = A.p_begin + pl;
    const int64_t howo = (int64_t)A.Ho * A.Wo;
    const int64_t n = p / howo;
    const int hw = (int)(p - n * howo);
    const int ho = hw / A.Wo;
    const int wo = hw - ho * A.Wo;
    const int hi0 = ho * A.sh - A.ph;
    const int wi0 = wo * A.sw - A.pw;
    const T* xb = reinterpret_cast<const T*>(A.x) + n * A.x_nstride + gi * A.x_gstride +
                  (int64_t)hi0 * A.W + wi0;
    const __amdgpu_buffer_rsrc_t rc = pk_rsrc(A.col, A.col_bytes);
    const int kr_end = min(kr0 + KR_PER_BLOCK, A.Kred);
    for (int kr = kr0; kr < kr_end; ++kr) {
        const KTabEntry e = A.ktab[__builtin_amdgcn_readfirstlane(kr)];
        const int hi = hi0 + e.roff;
        const int wi = wi0 + e.soff;
        T v = T(0);
        if ((unsigned)hi < (unsigned)A.H && (unsigned)wi < (unsigned)A.W) v = xb[e.coff];
        const int64_t off = ((int64_t)gi * A.Kred + kr) * A.pc + pl;
        if constexpr (sizeof(T) == 4)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rc,
                                                  (uint32_t)(off * 4), 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, v), rc,
                                                  (uint32_t)(off * 2), 0, 0);
    }
}

hipError_t launch_im2col(const Im2colArgs& a, int xdt, int groups, hipStream_t stream) {
    dim3 grid((unsigned)((a.pc + 255) / 256), (unsigned)((a.Kred + KR_PER_BLOCK - 1) / KR_PER_BLOCK),
              (unsigned)groups);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL(im2col_kernel<float>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(im2col_kernel<uint16_t>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ unpack
// grid (ceil(pc/256), Kg, G): C[g][m][pl] -> y[n][g*Kg + m][hw] (+ bias[g*Kg + m]).
template <bool BF16OUT>
__global__ __launch_bounds__(256) void unpack_kernel(UnpackArgs A) {
    const int pl = blockIdx.x * 256 + threadIdx.x;
    const int m = blockIdx.y;
    const int gi = blockIdx.z;
    if (pl >= A.pc) return;
    const int64_t p = A.p_begin + pl;
    const int64_t n = p / A.HoWo;
    const int64_t hw = p - n * A.HoWo;
    const int ch = gi * A.Kg + m;
    float v = A.c[((int64_t)gi * A.Kg + m) * A.pc + pl];
    if (A.bias) v += A.bias[ch];
    const int64_t off = n * A.y_nstride + (int64_t)ch * A.HoWo + hw;
    const __amdgpu_buffer_rsrc_t ry = pk_rsrc(A.y, A.y_bytes);
    if (BF16OUT)
        __builtin_amdgcn_raw_buffer_store_b16(pk_f32_to_bf16(v), ry, (uint32_t)(off * 2), 0, 0);
    else
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), ry, (uint32_t)(off * 4), 0, 0);
}

hipError_t launch_unpack(const UnpackArgs& a, int ydt, int groups, hipStream_t stream) {
    dim3 grid((unsigned)((a.pc + 255) / 256), (unsigned)a.Kg, (unsigned)groups);
    if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL(unpack_kernel<true>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(unpack_kernel<false>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ weight repack
// w [K][C/g][R*S] -> wr [K][R*S][C/g]: the tap-major order of the implicit GEMM's
// reduction, so one stage's weights (one tap, consecutive channels) are contiguous.
template <typename T>
__global__ __launch_bounds__(256) void repack_tap_major_kernel(const T* __restrict__ w, T* __restrict__ wr,
                                                              int64_t total, int cg, int rs) {
    const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (o >= total) return;
    const int c = (int)(o % cg);
    const int64_t kt = o / cg;
    const int tap = (int)(kt % rs);
    const int64_t k = kt / rs;
    wr[o] = w[(k * cg + c) * rs + tap];
}

hipError_t launch_repack_tap_major(const void* w, void* wr, int64_t k, int64_t cg, int64_t rs, int elem_bytes,
                                   hipStream_t stream) {
    const int64_t total = k * cg * rs;
    dim3 grid((unsigned)((total + 255) / 256));
    if (elem_bytes == 4)
        hipLaunchKernelGGL(repack_tap_major_kernel<uint32_t>, grid, dim3(256), 0, stream, (const uint32_t*)w,
                           (uint32_t*)wr, total, (int)cg, (int)rs);
    else
        hipLaunchKernelGGL(repack_tap_major_kernel<uint16_t>, grid, dim3(256), 0, stream, (const uint16_t*)w,
                           (uint16_t*)wr, total, (int)cg, (int)rs);
    return hipGetLastError();
}

// ------------------------------------------------------------------ layout transforms
// One image is a rows x cols matrix; out[c][r] = in[r][c].  32x32 tiles through LDS,
// block 32 x 8.  grid (ceil(cols/32), ceil(rows/32), n).
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                        int64_t rows, int64_t cols) {
    __shared__ T tile[32][33];
    const int64_t img = blockIdx.z;
    const int64_t c0 = (int64_t)blockIdx.x * 32, r0 = (int64_t)blockIdx.y * 32;
    const T* src = in + img * rows * cols;
    T* dst = out + img * rows * cols;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int i = ty; i < 32; i += 8) {
        const int64_t r = r0 + i, c = c0 + tx;
        if (r < rows && c < cols) tile[i][tx] = src[r * cols + c];
    }
    __syncthreads();
    for (int i = ty; i < 32; i += 8) {
        const int64_t c = c0 + i, r = r0 + tx;
        if (r < rows && c < cols) dst[c * rows + r] = tile[tx][i];
    }
}

static hipError_t launch_transpose(const void* src, void* dst, int64_t n, int64_t rows, int64_t cols,
                                   int elem_bytes, hipStream_t stream) {
    dim3 grid((unsigned)((cols + 31) / 32), (unsigned)((rows + 31) / 32), (unsigned)n);
    if (elem_bytes == 4)
        hipLaunchKernelGGL(transpose_kernel<uint32_t>, grid, dim3(256), 0, stream,
                           (const uint32_t*)src, (uint32_t*)dst, rows, cols);
    else
        hipLaunchKernelGGL(transpose_kernel<uint16_t>, grid, dim3(256), 0, stream,
                           (const uint16_t*)src, (uint16_t*)dst, rows, cols);
    return hipGetLastError();
}

hipError_t launch_nhwc_to_nchw(const void* src, void* dst, int64_t n, int64_t c, int64_t hw,
                               int elem_bytes, hipStream_t stream) {
    return launch_transpose(src, dst, n, hw, c, elem_bytes, stream);
}

hipError_t launch_nchw_to_nhwc(const void* src, void* dst, int64_t n, int64_t c, int64_t hw,
                               int elem_bytes, hipStream_t stream) {
    return launch_transpose(src, dst, n, c, hw, elem_bytes, stream);
}

}  // namespace cv
