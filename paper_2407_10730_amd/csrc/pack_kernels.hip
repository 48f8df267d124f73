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
#include <algorithm>

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
// grid (ceil(pc / 1024), ceil(Kred / KR_PER_BLOCK), G), 256 threads.  A thread packs 4
// consecutive pixels for KR_PER_BLOCK reduction rows: all its gathers are issued first,
// then each row's 4 values go out as one 16-byte (fp32) or 8-byte (bf16) store when the
// column matrix rows are aligned (pc % 4 == 0).
constexpr int KR_PER_BLOCK = 8;
constexpr int PIX_PER_THREAD = 4;

template <typename T>
__global__ __launch_bounds__(256) void im2col_kernel(Im2colArgs A) {
    const int gi = blockIdx.z;
    const int kr0 = blockIdx.y * KR_PER_BLOCK;
    const int pl0 = (blockIdx.x * 256 + threadIdx.x) * PIX_PER_THREAD;
    if (pl0 >= A.pc) return;
    const __amdgpu_buffer_rsrc_t rc = pk_rsrc(A.col, A.col_bytes);
    // window origins of the 4 pixels (consecutive in (n, ho, wo) order)
    int hi0[PIX_PER_THREAD], wi0[PIX_PER_THREAD];
    int64_t xb[PIX_PER_THREAD];
    bool pv[PIX_PER_THREAD];
    {
        const int64_t p = A.p_begin + pl0;
        const int64_t howo = (int64_t)A.Ho * A.Wo;
        int64_t n = p / howo;
        int hw = (int)(p - n * howo);
        int ho = hw / A.Wo;
        int wo = hw - ho * A.Wo;
#pragma unroll
        for (int j = 0; j < PIX_PER_THREAD; ++j) {
            pv[j] = pl0 + j < A.pc;
            hi0[j] = ho * A.sh - A.ph;
            wi0[j] = wo * A.sw - A.pw;
            xb[j] = n * A.x_nstride + gi * A.x_gstride + (int64_t)hi0[j] * A.W + wi0[j];
            if (++wo == A.Wo) {
                wo = 0;
                if (++ho == A.Ho) {
                    ho = 0;
                    ++n;
                }
            }
        }
    }
    const T* x = reinterpret_cast<const T*>(A.x);
    KTabEntry e[KR_PER_BLOCK];
#pragma unroll
    for (int i = 0; i < KR_PER_BLOCK; ++i) e[i] = A.ktab[__builtin_amdgcn_readfirstlane(min(kr0 + i, A.Kred - 1))];
    T v[KR_PER_BLOCK][PIX_PER_THREAD];
    if (A.x_bytes != 0) {
        // x below 2 GiB: 32-bit element offsets into a range-checked buffer (a window position
        // outside the image takes the out-of-range offset and reads zero), instead of 64-bit
        // address arithmetic per gathered element
        const __amdgpu_buffer_rsrc_t rx = pk_rsrc(A.x, A.x_bytes);
        int32_t xb32[PIX_PER_THREAD];
#pragma unroll
        for (int j = 0; j < PIX_PER_THREAD; ++j) xb32[j] = (int32_t)xb[j];
#pragma unroll
        for (int i = 0; i < KR_PER_BLOCK; ++i)
#pragma unroll
            for (int j = 0; j < PIX_PER_THREAD; ++j) {
                const int hi = hi0[j] + e[i].roff;
                const int wi = wi0[j] + e[i].soff;
                const bool ok = pv[j] & ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
                const uint32_t off = ok ? (uint32_t)(xb32[j] + e[i].coff) * (uint32_t)sizeof(T) : OOB_OFF;
                if constexpr (sizeof(T) == 4)
                    v[i][j] = __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(rx, off, 0, 0));
                else
                    v[i][j] = (T)__builtin_amdgcn_raw_buffer_load_b16(rx, off, 0, 0);
            }
    } else {
#pragma unroll
        for (int i = 0; i < KR_PER_BLOCK; ++i)
#pragma unroll
            for (int j = 0; j < PIX_PER_THREAD; ++j) {
                const int hi = hi0[j] + e[i].roff;
                const int wi = wi0[j] + e[i].soff;
                const bool ok = pv[j] & ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
                v[i][j] = ok ? x[xb[j] + e[i].coff] : T(0);
            }
    }
    const bool vec = ((A.pc & 3) == 0) & (pl0 + PIX_PER_THREAD <= A.pc);
#pragma unroll
    for (int i = 0; i < KR_PER_BLOCK; ++i) {
        const int kr = kr0 + i;
        if (kr >= A.Kred) break;
        const int64_t off = ((int64_t)gi * A.Kred + kr) * A.pc + pl0;
        if constexpr (sizeof(T) == 4) {
            if (vec) {
                typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                const u32x4 q = {__builtin_bit_cast(uint32_t, v[i][0]), __builtin_bit_cast(uint32_t, v[i][1]),
                                 __builtin_bit_cast(uint32_t, v[i][2]), __builtin_bit_cast(uint32_t, v[i][3])};
                __builtin_amdgcn_raw_buffer_store_b128(q, rc, (uint32_t)(off * 4), 0, 0);
            } else {
#pragma unroll
                for (int j = 0; j < PIX_PER_THREAD; ++j)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[i][j]), rc,
                                                          pv[j] ? (uint32_t)((off + j) * 4) : OOB_OFF, 0, 0);
            }
        } else {
            if (vec) {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                const u32x2 q = {(uint32_t)v[i][0] | ((uint32_t)v[i][1] << 16),
                                 (uint32_t)v[i][2] | ((uint32_t)v[i][3] << 16)};
                __builtin_amdgcn_raw_buffer_store_b64(q, rc, (uint32_t)(off * 2), 0, 0);
            } else {
#pragma unroll
                for (int j = 0; j < PIX_PER_THREAD; ++j)
                    __builtin_amdgcn_raw_buffer_store_b16(v[i][j], rc, pv[j] ? (uint32_t)((off + j) * 2) : OOB_OFF, 0, 0);
            }
        }
    }
}

hipError_t launch_im2col(const Im2colArgs& a, int xdt, int groups, hipStream_t stream) {
    const int per_block = 256 * PIX_PER_THREAD;
    dim3 grid((unsigned)((a.pc + per_block - 1) / per_block),
              (unsigned)((a.Kred + KR_PER_BLOCK - 1) / KR_PER_BLOCK), (unsigned)groups);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL(im2col_kernel<float>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(im2col_kernel<uint16_t>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ unpack
// grid (ceil(pc / 1024), Kg, G): C[g][m][pl] -> y[n][g*Kg + m][hw] (+ bias[g*Kg + m]).
// A thread moves 4 consecutive pixels; with HoWo % 4 == 0 and pc % 4 == 0 they are one
// 16-byte load and one 16-byte (fp32) or 8-byte (bf16) store.
template <bool BF16OUT>
__global__ __launch_bounds__(256) void unpack_kernel(UnpackArgs A) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const int pl0 = (blockIdx.x * 256 + threadIdx.x) * 4;
    const int m = blockIdx.y;
    const int gi = blockIdx.z;
    if (pl0 >= A.pc) return;
    const int ch = gi * A.Kg + m;
    const float bias = A.bias ? A.bias[ch] : 0.0f;
    const float* crow = A.c + ((int64_t)gi * A.Kg + m) * A.pc;
    const int splits = A.splits > 1 ? A.splits : 1;
    const __amdgpu_buffer_rsrc_t ry = pk_rsrc(A.y, A.y_bytes);
    const int64_t p = A.p_begin + pl0;
    const int64_t n = p / A.HoWo;
    const int64_t hw = p - n * A.HoWo;
    const int64_t off = n * A.y_nstride + (int64_t)ch * A.HoWo + hw;
    const bool vec = ((A.HoWo & 3) == 0) & ((A.pc & 3) == 0) & ((A.p_begin & 3) == 0) & (pl0 + 4 <= A.pc) &
                     ((A.split_stride & 3) == 0);
    if (vec) {
        f32x4 c = *reinterpret_cast<const f32x4*>(crow + pl0);
        for (int sp = 1; sp < splits; ++sp) c += *reinterpret_cast<const f32x4*>(crow + sp * A.split_stride + pl0);
        if (BF16OUT) {
            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
            const u32x2 q = {(uint32_t)pk_f32_to_bf16(c[0] + bias) | ((uint32_t)pk_f32_to_bf16(c[1] + bias) << 16),
                             (uint32_t)pk_f32_to_bf16(c[2] + bias) | ((uint32_t)pk_f32_to_bf16(c[3] + bias) << 16)};
            __builtin_amdgcn_raw_buffer_store_b64(q, ry, (uint32_t)(off * 2), 0, 0);
        } else {
            typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
            const u32x4 q = {__builtin_bit_cast(uint32_t, c[0] + bias), __builtin_bit_cast(uint32_t, c[1] + bias),
                             __builtin_bit_cast(uint32_t, c[2] + bias), __builtin_bit_cast(uint32_t, c[3] + bias)};
            __builtin_amdgcn_raw_buffer_store_b128(q, ry, (uint32_t)(off * 4), 0, 0);
        }
        return;
    }
    for (int j = 0; j < 4 && pl0 + j < A.pc; ++j) {
        const int64_t pj = p + j;
        const int64_t nj = pj / A.HoWo;
        const int64_t o = nj * A.y_nstride + (int64_t)ch * A.HoWo + (pj - nj * A.HoWo);
        float c = crow[pl0 + j];
        for (int sp = 1; sp < splits; ++sp) c += crow[sp * A.split_stride + pl0 + j];
        const float v = c + bias;
        if (BF16OUT)
            __builtin_amdgcn_raw_buffer_store_b16(pk_f32_to_bf16(v), ry, (uint32_t)(o * 2), 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), ry, (uint32_t)(o * 4), 0, 0);
    }
}

// NHWC y: grid (ceil(pc / 256), ceil(Kg / 4), G).  A thread takes one pixel and 4 consecutive
// channels: 4 loads, each coalesced over the wave's consecutive pixels, and one 16-byte (fp32)
// or 8-byte (bf16) store of y[p][g*Kg + m .. +3] when Kg % 4 == 0, element stores otherwise.
template <bool BF16OUT>
__global__ __launch_bounds__(256) void unpack_nhwc_kernel(UnpackArgs A) {
    const int pl = blockIdx.x * 256 + threadIdx.x;
    const int m0 = blockIdx.y * 4;
    const int gi = blockIdx.z;
    if (pl >= A.pc) return;
    const int splits = A.splits > 1 ? A.splits : 1;
    const int kall = A.Kg * gridDim.z;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int m = m0 + j < A.Kg ? m0 + j : A.Kg - 1;  // rows past Kg are computed but not stored
        const float* crow = A.c + ((int64_t)gi * A.Kg + m) * A.pc + pl;
        float c = crow[0];
        for (int sp = 1; sp < splits; ++sp) c += crow[sp * A.split_stride];
        v[j] = c + (A.bias ? A.bias[gi * A.Kg + m] : 0.0f);
    }
    const __amdgpu_buffer_rsrc_t ry = pk_rsrc(A.y, A.y_bytes);
    const int64_t o = (A.p_begin + pl) * kall + (int64_t)gi * A.Kg + m0;
    if ((A.Kg & 3) == 0) {
        if (BF16OUT) {
            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
            const u32x2 q = {(uint32_t)pk_f32_to_bf16(v[0]) | ((uint32_t)pk_f32_to_bf16(v[1]) << 16),
                             (uint32_t)pk_f32_to_bf16(v[2]) | ((uint32_t)pk_f32_to_bf16(v[3]) << 16)};
            __builtin_amdgcn_raw_buffer_store_b64(q, ry, (uint32_t)(o * 2), 0, 0);
        } else {
            typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
            const u32x4 q = {__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                             __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])};
            __builtin_amdgcn_raw_buffer_store_b128(q, ry, (uint32_t)(o * 4), 0, 0);
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (m0 + j >= A.Kg) break;
        if (BF16OUT)
            __builtin_amdgcn_raw_buffer_store_b16(pk_f32_to_bf16(v[j]), ry, (uint32_t)((o + j) * 2), 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[j]), ry, (uint32_t)((o + j) * 4), 0, 0);
    }
}

hipError_t launch_unpack(const UnpackArgs& a, int ydt, int groups, hipStream_t stream) {
    if (a.nhwc) {
        dim3 grid((unsigned)((a.pc + 255) / 256), (unsigned)((a.Kg + 3) / 4), (unsigned)groups);
        if (ydt == CONV2D_BF16)
            hipLaunchKernelGGL(unpack_nhwc_kernel<true>, grid, dim3(256), 0, stream, a);
        else
            hipLaunchKernelGGL(unpack_nhwc_kernel<false>, grid, dim3(256), 0, stream, a);
        return hipGetLastError();
    }
    dim3 grid((unsigned)((a.pc + 1023) / 1024), (unsigned)a.Kg, (unsigned)groups);
    if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL(unpack_kernel<true>, grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(unpack_kernel<false>, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ weight repack
// w [K][C/g][R*S] -> wr [K][R*S][C/g]: the tap-major order of the implicit GEMM's
// reduction, so one stage's weights (one tap, consecutive channels) are contiguous.
// Block (x, k) moves channels [x*cc, x*cc + cc) of filter k: it reads their cc*R*S
// contiguous elements into LDS (one word each) with consecutive threads on consecutive
// elements, then writes every tap's run of channels, again consecutive threads on
// consecutive elements (the LDS reads of one tap are R*S words apart).
template <typename T>
__global__ __launch_bounds__(256) void repack_tap_major_kernel(const T* __restrict__ w, T* __restrict__ wr,
                                                              uint32_t cg, uint32_t rs, uint32_t cc) {
    extern __shared__ uint32_t rtile[];
    const uint32_t k = blockIdx.y;
    const uint32_t c0 = blockIdx.x * cc;
    const uint32_t nc = min(cc, cg - c0);
    const uint32_t n = nc * rs;
    const T* src = w + ((size_t)k * cg + c0) * rs;
    for (uint32_t i = threadIdx.x; i < n; i += 256) rtile[i] = (uint32_t)src[i];
    __syncthreads();
    T* dst = wr + (size_t)k * rs * cg + c0;
    for (uint32_t i = threadIdx.x; i < n; i += 256) {
        const uint32_t tap = i / nc;
        const uint32_t c = i - tap * nc;
        dst[(size_t)tap * cg + c] = (T)rtile[c * rs + tap];
    }
}

// One thread per destination element, read straight from the source (a gather within the
// filter row, which the caches hold): one memory round trip instead of two and no barrier, for
// filter sets small enough that the repack is latency-bound.
template <typename T>
__global__ __launch_bounds__(256) void repack_tap_major_direct_kernel(const T* __restrict__ w, T* __restrict__ wr,
                                                                     uint32_t cg, uint32_t rs, uint32_t total,
                                                                     FastDiv fd_cg, FastDiv fd_rscg) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;  // destination index (k, tap, c)
    if (i >= total) return;
    const uint32_t k = (__umulhi(i, fd_rscg.m) + i) >> fd_rscg.s;
    const uint32_t rem = i - k * rs * cg;
    const uint32_t tap = (__umulhi(rem, fd_cg.m) + rem) >> fd_cg.s;
    const uint32_t c = rem - tap * cg;
    wr[i] = w[((size_t)k * cg + c) * rs + tap];
}

hipError_t launch_repack_tap_major(const void* w, void* wr, int64_t k, int64_t cg, int64_t rs, int elem_bytes,
                                   hipStream_t stream) {
    const int64_t total = k * cg * rs;
    if (total <= 0 || total >= ((int64_t)1 << 31) || k > 65535 || rs > 4096) return hipErrorInvalidValue;
    if (total <= (1 << 20)) {
        const dim3 grid((unsigned)((total + 255) / 256));
        const FastDiv fcg = make_fastdiv((uint32_t)cg), frc = make_fastdiv((uint32_t)(rs * cg));
        if (elem_bytes == 4)
            hipLaunchKernelGGL(repack_tap_major_direct_kernel<uint32_t>, grid, dim3(256), 0, stream, (const uint32_t*)w,
                               (uint32_t*)wr, (uint32_t)cg, (uint32_t)rs, (uint32_t)total, fcg, frc);
        else
            hipLaunchKernelGGL(repack_tap_major_direct_kernel<uint16_t>, grid, dim3(256), 0, stream, (const uint16_t*)w,
                               (uint16_t*)wr, (uint32_t)cg, (uint32_t)rs, (uint32_t)total, fcg, frc);
        return hipGetLastError();
    }
    // channels per block: at most 4096 elements (16 KiB of LDS)
    const int64_t cc = std::max<int64_t>(1, std::min<int64_t>(cg, 4096 / rs));
    dim3 grid((unsigned)((cg + cc - 1) / cc), (unsigned)k);
    const size_t lds = (size_t)(cc * rs) * 4;
    if (elem_bytes == 4)
        hipLaunchKernelGGL(repack_tap_major_kernel<uint32_t>, grid, dim3(256), lds, stream, (const uint32_t*)w,
                           (uint32_t*)wr, (uint32_t)cg, (uint32_t)rs, (uint32_t)cc);
    else
        hipLaunchKernelGGL(repack_tap_major_kernel<uint16_t>, grid, dim3(256), lds, stream, (const uint16_t*)w,
                           (uint16_t*)wr, (uint32_t)cg, (uint32_t)rs, (uint32_t)cc);
    return hipGetLastError();
}

// ------------------------------------------------------------------ fills
// dst[0:n] = value.  Clears counters with a kernel rather than hipMemsetAsync, so that a
// caller may record the call into a HIP graph.
__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t* __restrict__ dst, uint32_t n, uint32_t value) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i < n) dst[i] = value;
}

hipError_t launch_fill_u32(uint32_t* dst, int64_t n, uint32_t value, hipStream_t stream) {
    if (n <= 0 || n >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, dst, (uint32_t)n,
                       value);
    return hipGetLastError();
}

// Tap table on the device: entry kr = (c, r, s) of the natural reduction order holds the
// element offset c*H*W + r*dh*W + s*dw of the tap from the window origin and the row / column
// shifts r*dh, s*dw; entries past Kred get the dead row shift, so every bounds test fails.
// The same table the planner builds on the host, for callers that cannot upload it.
__global__ __launch_bounds__(256) void ktab_fill_kernel(KTabEntry* __restrict__ t, int32_t len, int32_t kred,
                                                        int32_t rs, int32_t S, int32_t hw, int32_t W, int32_t dh,
                                                        int32_t dw) {
    const int32_t kr = (int32_t)(blockIdx.x * 256u + threadIdx.x);
    if (kr >= len) return;
    KTabEntry e{0, KTAB_DEAD, 0, 0};
    if (kr < kred) {
        const int32_t c = kr / rs;
        const int32_t q = kr - c * rs;
        const int32_t r = q / S;
        const int32_t s = q - r * S;
        e.roff = r * dh;
        e.soff = s * dw;
        e.coff = c * hw + e.roff * W + e.soff;
    }
    t[kr] = e;
}

hipError_t launch_ktab_fill(KTabEntry* t, int64_t len, int64_t kred, int64_t cg, int64_t r, int64_t s, int64_t h,
                            int64_t w, int dh, int dw, hipStream_t stream) {
    if (len <= 0 || len >= ((int64_t)1 << 31) || kred > len || cg * h * w >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(ktab_fill_kernel, dim3((unsigned)((len + 255) / 256)), dim3(256), 0, stream, t, (int32_t)len,
                       (int32_t)kred, (int32_t)(r * s), (int32_t)s, (int32_t)(h * w), (int32_t)w, dh, dw);
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

// The same transform with 64x64 tiles when rows and cols are multiples of 4: a thread moves
// 4 consecutive elements per global access (8 bytes in bf16, 16 in fp32: the 32x32 kernel's
// 2-byte accesses moved bf16 at about 3 TB/s).  The tile keeps one element per 4-byte LDS word
// with a row pitch of 65 words, so the column reads of the write phase spread over all banks.
// grid (ceil(cols/64), ceil(rows/64), n).
template <typename T>
__global__ __launch_bounds__(256) void transpose64_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                          int64_t rows, int64_t cols) {
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
    __shared__ uint32_t tile[64][65];
    const int64_t img = blockIdx.z;
    const int64_t c0 = (int64_t)blockIdx.x * 64, r0 = (int64_t)blockIdx.y * 64;
    const T* src = in + img * rows * cols;
    T* dst = out + img * rows * cols;
    const int tq = threadIdx.x & 15, tr = threadIdx.x >> 4;  // quad of 4 elements, row of 16
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int lr = tr + 16 * i;
        const int64_t r = r0 + lr, c = c0 + 4 * tq;
        uint32_t e[4] = {0, 0, 0, 0};
        if (r < rows && c < cols) {  // cols % 4 == 0: the whole quad is inside
            if constexpr (sizeof(T) == 2) {
                const u32x2_t v = *reinterpret_cast<const u32x2_t*>(src + r * cols + c);
                e[0] = v[0] & 0xFFFFu; e[1] = v[0] >> 16; e[2] = v[1] & 0xFFFFu; e[3] = v[1] >> 16;
            } else {
                const u32x4_t v = *reinterpret_cast<const u32x4_t*>(src + r * cols + c);
                e[0] = v[0]; e[1] = v[1]; e[2] = v[2]; e[3] = v[3];
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) tile[lr][4 * tq + k] = e[k];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int lc = tr + 16 * i;
        const int64_t c = c0 + lc, r = r0 + 4 * tq;
        if (c < cols && r < rows) {  // rows % 4 == 0
            const uint32_t e0 = tile[4 * tq][lc], e1 = tile[4 * tq + 1][lc], e2 = tile[4 * tq + 2][lc],
                           e3 = tile[4 * tq + 3][lc];
            if constexpr (sizeof(T) == 2)
                *reinterpret_cast<u32x2_t*>(dst + c * rows + r) = u32x2_t{e0 | (e1 << 16), e2 | (e3 << 16)};
            else
                *reinterpret_cast<u32x4_t*>(dst + c * rows + r) = u32x4_t{e0, e1, e2, e3};
        }
    }
}

// The same transform when one side has at most NARROW_MAX entries (an image with few channels):
// the 32x32 tiles would stay mostly empty, so a thread takes one index j of the long side and
// moves its short row (reads or writes of consecutive threads are adjacent for every short
// index).  grid (ceil(long / 256), n).
constexpr int64_t NARROW_MAX = 8;
template <typename T, bool NARROW_COLS>
__global__ __launch_bounds__(256) void narrow_transpose_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                               int64_t rows, int64_t cols) {
    const int64_t img = blockIdx.y;
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const T* src = in + img * rows * cols;
    T* dst = out + img * rows * cols;
    if (NARROW_COLS) {
        if (j >= rows) return;
        for (int64_t c = 0; c < cols; ++c) dst[c * rows + j] = src[j * cols + c];
    } else {
        if (j >= cols) return;
        for (int64_t r = 0; r < rows; ++r) dst[j * rows + r] = src[r * cols + j];
    }
}

template <typename T>
static void launch_narrow(const void* src, void* dst, int64_t n, int64_t rows, int64_t cols, hipStream_t stream) {
    const bool ncols = cols <= NARROW_MAX;
    dim3 grid((unsigned)(((ncols ? rows : cols) + 255) / 256), (unsigned)n);
    if (ncols)
        hipLaunchKernelGGL((narrow_transpose_kernel<T, true>), grid, dim3(256), 0, stream, (const T*)src, (T*)dst,
                           rows, cols);
    else
        hipLaunchKernelGGL((narrow_transpose_kernel<T, false>), grid, dim3(256), 0, stream, (const T*)src, (T*)dst,
                           rows, cols);
}

static hipError_t launch_transpose(const void* src, void* dst, int64_t n, int64_t rows, int64_t cols,
                                   int elem_bytes, hipStream_t stream) {
    if (n > 65535) return hipErrorInvalidValue;
    if (std::min(rows, cols) <= NARROW_MAX) {
        if (elem_bytes == 4) launch_narrow<uint32_t>(src, dst, n, rows, cols, stream);
        else launch_narrow<uint16_t>(src, dst, n, rows, cols, stream);
        return hipGetLastError();
    }
    // (CONV2D_TRANSPOSE32=1 keeps the 32x32 kernel: tests run both)
    const char* t32 = std::getenv("CONV2D_TRANSPOSE32");
    if (rows % 4 == 0 && cols % 4 == 0 && ((uintptr_t)src & 15) == 0 && ((uintptr_t)dst & 15) == 0 &&
        !(t32 && t32[0] == '1')) {
        dim3 grid64((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64), (unsigned)n);
        if (elem_bytes == 4)
            hipLaunchKernelGGL(transpose64_kernel<uint32_t>, grid64, dim3(256), 0, stream, (const uint32_t*)src,
                               (uint32_t*)dst, rows, cols);
        else
            hipLaunchKernelGGL(transpose64_kernel<uint16_t>, grid64, dim3(256), 0, stream, (const uint16_t*)src,
                               (uint16_t*)dst, rows, cols);
        return hipGetLastError();
    }
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
