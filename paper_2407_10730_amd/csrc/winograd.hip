// winograd.hip -- Winograd minimal-filtering convolution F(m x m, 3x3), m = 2 or 4 (Lavin and
// Gray, CVPR 2016), the transform-based algorithm family the paper names next to GEMM and
// direct methods (Sec. I), for 3x3 filters, stride 1, dilation 1, one group, fp32.
//
// Every m x m block of outputs (a tile) is computed from the (m+2) x (m+2) input patch under it:
//   Y = A^T [ (G g G^T) (.) (B^T d B) ] A
// with the element-wise product (.) summed over input channels, which turns the (m+2)^2
// positions of the transformed domain into independent GEMMs
//   M[xi][k][t] = sum_c U[xi][k][c] * V[xi][c][t]
// (U: transformed filters, V: transformed input patches, t: tile).  The phases map onto the
// timing tool's steps: the filter transform is a pre-convolution reordering of the weights,
// the input transform is the packing, the batched GEMM is the microkernel (the library's MFMA
// GEMM with dense operands, one "group" per position) and the output transform is the
// unpacking, which also adds the bias and writes NCHW y.  Tiles are processed in chunks that
// fit the workspace.
//
// F(2x2, 3x3), interpolation points 0, 1, -1 and infinity:
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1]
//   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1]
//   A^T = [1 1 1 0; 0 1 -1 -1]
// F(4x4, 3x3), points 0, 1, -1, 2, -2 and infinity (2.25x fewer multiplications than F(2x2),
// with larger transform constants and so larger rounding errors):
//   B^T = [4 0 -5 0 1 0; 0 -4 -4 1 1 0; 0 4 -4 -1 1 0; 0 -2 -1 2 1 0; 0 2 -1 -2 1 0; 0 4 0 -5 0 1]
//   G   = [1/4 0 0; -1/6 -1/6 -1/6; -1/6 1/6 -1/6; 1/24 1/12 1/6; 1/24 -1/12 1/6; 0 0 1]
//   A^T = [1 1 1 1 1 0; 0 1 -1 2 -2 0; 0 1 1 4 4 0; 0 1 -1 8 -8 1]
#include "device_common.h"

namespace cv {

// o = G g for one column g of the filter (length 3 -> MT+2)
template <int MT>
__device__ __forceinline__ void wino_g(float g0, float g1, float g2, float* o) {
    if constexpr (MT == 2) {
        o[0] = g0;
        o[1] = 0.5f * (g0 + g1 + g2);
        o[2] = 0.5f * (g0 - g1 + g2);
        o[3] = g2;
    } else {
        o[0] = 0.25f * g0;
        o[1] = (-1.0f / 6.0f) * (g0 + g1 + g2);
        o[2] = (-1.0f / 6.0f) * (g0 - g1 + g2);
        o[3] = (1.0f / 24.0f) * g0 + (1.0f / 12.0f) * g1 + (1.0f / 6.0f) * g2;
        o[4] = (1.0f / 24.0f) * g0 - (1.0f / 12.0f) * g1 + (1.0f / 6.0f) * g2;
        o[5] = g2;
    }
}

// o = B^T d for one column d of the input patch (length MT+2)
template <int MT>
__device__ __forceinline__ void wino_bt(const float* d, float* o) {
    if constexpr (MT == 2) {
        o[0] = d[0] - d[2];
        o[1] = d[1] + d[2];
        o[2] = d[2] - d[1];
        o[3] = d[1] - d[3];
    } else {
        o[0] = 4.0f * d[0] - 5.0f * d[2] + d[4];
        o[1] = (d[3] + d[4]) - 4.0f * (d[1] + d[2]);
        o[2] = (d[4] - d[3]) + 4.0f * (d[1] - d[2]);
        o[3] = (d[4] - d[2]) + 2.0f * (d[3] - d[1]);
        o[4] = (d[4] - d[2]) - 2.0f * (d[3] - d[1]);
        o[5] = 4.0f * d[1] - 5.0f * d[3] + d[5];
    }
}

// o = A^T m for one column m of the GEMM results (length MT+2 -> MT)
template <int MT>
__device__ __forceinline__ void wino_at(const float* m, float* o) {
    if constexpr (MT == 2) {
        o[0] = m[0] + m[1] + m[2];
        o[1] = m[1] - m[2] - m[3];
    } else {
        const float p12 = m[1] + m[2], d12 = m[1] - m[2];
        const float p34 = m[3] + m[4], d34 = m[3] - m[4];
        o[0] = m[0] + p12 + p34;
        o[1] = d12 + 2.0f * d34;
        o[2] = p12 + 4.0f * p34;
        o[3] = d12 + 8.0f * d34 + m[5];
    }
}

// element v of w (fp32, or bf16 widened) and a transformed value in the workspace's type (fp32,
// or bf16 rounded to nearest even)
__device__ __forceinline__ float wino_ld(const float* p, int64_t v) { return p[v]; }
__device__ __forceinline__ float wino_ld(const uint16_t* p, int64_t v) {
    return __builtin_bit_cast(float, (uint32_t)p[v] << 16);
}
__device__ __forceinline__ void wino_st(float* p, int64_t v, float f) { p[v] = f; }
__device__ __forceinline__ void wino_st(uint16_t* p, int64_t v, float f) { p[v] = f32_to_bf16_rne(f); }

// U[xi][k][c] = (G g_kc G^T)[xi]; one thread per (k, c), c fastest (coalesced writes).  The
// transform is computed in fp32 from the (fp32 or bf16) filters; bf16 U is rounded once.
template <int MT, typename T>
__global__ __launch_bounds__(256) void wino_filter_kernel(const T* __restrict__ w, T* __restrict__ u, int K, int C) {
    constexpr int AL = MT + 2;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)K * C) return;
    const T* g = w + i * 9;  // w[k][c][3][3], i = k*C + c
    float t[AL][3];          // G g
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        float col[AL];
        wino_g<MT>(wino_ld(g, j), wino_ld(g, 3 + j), wino_ld(g, 6 + j), col);
#pragma unroll
        for (int a = 0; a < AL; ++a) t[a][j] = col[a];
    }
    const int64_t plane = (int64_t)K * C;
#pragma unroll
    for (int a = 0; a < AL; ++a) {  // (G g) G^T
        float row[AL];
        wino_g<MT>(t[a][0], t[a][1], t[a][2], row);
#pragma unroll
        for (int b = 0; b < AL; ++b) wino_st(u, (a * AL + b) * plane + i, row[b]);
    }
}

// bf16: V[xi][t - t0][c] = (B^T d B)[xi] from the NHWC copy of x, one thread per (tile, c), c
// fastest: reads of x and writes of V both run along the channels (the GEMM then reads 8
// channels of a tile with one 16-byte load).  Computed in fp32, rounded to bf16 once.
template <int MT>
__global__ __launch_bounds__(256) void wino_input_nhwc_kernel(WinoArgs A, uint16_t* __restrict__ v) {
    constexpr int AL = MT + 2;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)A.C * A.tc) return;
    const int tl = (int)(i / A.C);
    const int c = (int)(i - (int64_t)tl * A.C);
    const int64_t t = A.t0 + tl;
    const int tiles_img = A.th * A.tw;
    const int n = (int)(t / tiles_img);
    const int r = (int)(t - (int64_t)n * tiles_img);
    const int ty = r / A.tw, tx = r - (r / A.tw) * A.tw;
    const int hi0 = MT * ty - A.ph, wi0 = MT * tx - A.pw;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(A.x, A.x_bytes);
    float d[AL][AL];
#pragma unroll
    for (int a = 0; a < AL; ++a) {
        const int hi = hi0 + a;
        const bool hok = (unsigned)hi < (unsigned)A.H;
#pragma unroll
        for (int b = 0; b < AL; ++b) {
            const int wi = wi0 + b;
            const bool ok = hok & ((unsigned)wi < (unsigned)A.W);
            const int64_t e = (((int64_t)n * A.H + hi) * A.W + wi) * A.C + c;
            const uint32_t h = ld_u16(rx, ok ? (uint32_t)(e * 2) : OOB_OFF);
            d[a][b] = __builtin_bit_cast(float, h << 16);
        }
    }
    float e[AL][AL];  // B^T d
#pragma unroll
    for (int b = 0; b < AL; ++b) {
        float col[AL], o[AL];
#pragma unroll
        for (int a = 0; a < AL; ++a) col[a] = d[a][b];
        wino_bt<MT>(col, o);
#pragma unroll
        for (int a = 0; a < AL; ++a) e[a][b] = o[a];
    }
    const int64_t plane = (int64_t)A.tc * A.C;
#pragma unroll
    for (int a = 0; a < AL; ++a) {  // (B^T d) B
        float o[AL];
        wino_bt<MT>(e[a], o);
#pragma unroll
        for (int b = 0; b < AL; ++b) v[(a * AL + b) * plane + i] = f32_to_bf16_rne(o[b]);
    }
}

// V[xi][c][t - t0] = (B^T d B)[xi] for the tiles t0 .. t0+tc-1 (tile t = (n, th, tw) row-major);
// one thread per (c, tile), tile fastest.  VPW = pw (0 or 1) for F(4x4) when W is a multiple
// of 4 and every tile's aligned columns 4*tx .. 4*tx+3 lie inside the row: the 6 columns of a
// patch row then hold those four, read with one 16-byte load (consecutive lanes read consecutive
// 16-byte words), and two single columns; VPW = -1 reads 6 single columns.
template <int MT, int VPW>
__global__ __launch_bounds__(256) void wino_input_kernel(WinoArgs A, float* __restrict__ v) {
    constexpr int AL = MT + 2;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)A.C * A.tc) return;
    const int c = (int)(i / A.tc);
    const int tl = (int)(i - (int64_t)c * A.tc);
    const int64_t t = A.t0 + tl;
    const int tiles_img = A.th * A.tw;
    const int n = (int)(t / tiles_img);
    const int r = (int)(t - (int64_t)n * tiles_img);
    const int ty = r / A.tw, tx = r - (r / A.tw) * A.tw;
    const int hi0 = MT * ty - A.ph, wi0 = MT * tx - A.pw;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(A.x, A.x_bytes);
    const int64_t plane0 = ((int64_t)n * A.C + c) * A.H;
    float d[AL][AL];
#pragma unroll
    for (int a = 0; a < AL; ++a) {
        const int hi = hi0 + a;
        const bool hok = (unsigned)hi < (unsigned)A.H;
        const int64_t row = (plane0 + hi) * A.W;
        if constexpr (VPW >= 0) {
            // the aligned columns MT*tx .. MT*tx+3 with one 16-byte load, the other two singly
            const f32x4 q = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(rx, hok ? (uint32_t)((row + MT * tx) * 4) : OOB_OFF, 0, 0));
#pragma unroll
            for (int b = 0; b < AL; ++b) {
                if (b >= VPW && b < VPW + 4) {
                    d[a][b] = q[b - VPW];
                } else {
                    const int wi = wi0 + b;
                    const bool ok = hok & ((unsigned)wi < (unsigned)A.W);
                    d[a][b] = ld_f32(rx, ok ? (uint32_t)((row + wi) * 4) : OOB_OFF);
                }
            }
        } else {
#pragma unroll
            for (int b = 0; b < AL; ++b) {
                const int wi = wi0 + b;
                const bool ok = hok & ((unsigned)wi < (unsigned)A.W);
                d[a][b] = ld_f32(rx, ok ? (uint32_t)((row + wi) * 4) : OOB_OFF);
            }
        }
    }
    float e[AL][AL];  // B^T d
#pragma unroll
    for (int b = 0; b < AL; ++b) {
        float col[AL], o[AL];
#pragma unroll
        for (int a = 0; a < AL; ++a) col[a] = d[a][b];
        wino_bt<MT>(col, o);
#pragma unroll
        for (int a = 0; a < AL; ++a) e[a][b] = o[a];
    }
    const int64_t plane = (int64_t)A.C * A.tc;
#pragma unroll
    for (int a = 0; a < AL; ++a) {  // (B^T d) B
        float o[AL];
        wino_bt<MT>(e[a], o);
#pragma unroll
        for (int b = 0; b < AL; ++b) v[(a * AL + b) * plane + i] = o[b];
    }
}

// y (the MT x MT block of tile t, clipped at the edges) = A^T M A + bias; one thread per
// (k, tile), tile fastest.
template <int MT, typename TY>
__global__ __launch_bounds__(256) void wino_output_kernel(WinoArgs A, const float* __restrict__ m) {
    constexpr int AL = MT + 2;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)A.K * A.tc) return;
    const int k = (int)(i / A.tc);
    const int tl = (int)(i - (int64_t)k * A.tc);
    const int64_t t = A.t0 + tl;
    const int tiles_img = A.th * A.tw;
    const int n = (int)(t / tiles_img);
    const int r = (int)(t - (int64_t)n * tiles_img);
    const int ty = r / A.tw, tx = r - (r / A.tw) * A.tw;
    const int64_t plane = (int64_t)A.K * A.tc;
    float q[AL][AL];
#pragma unroll
    for (int a = 0; a < AL; ++a)
#pragma unroll
        for (int b = 0; b < AL; ++b) q[a][b] = m[(a * AL + b) * plane + i];
    float s[MT][AL];  // A^T M
#pragma unroll
    for (int b = 0; b < AL; ++b) {
        float col[AL], o[MT];
#pragma unroll
        for (int a = 0; a < AL; ++a) col[a] = q[a][b];
        wino_at<MT>(col, o);
#pragma unroll
        for (int a = 0; a < MT; ++a) s[a][b] = o[a];
    }
    const float bias = A.bias ? A.bias[k] : 0.0f;
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
    // with Wo a multiple of MT every row of a tile starts MT-float aligned: one vector store
    // per row when it lies inside the plane
    const bool vec = sizeof(TY) == 4 && A.Wo % MT == 0;
#pragma unroll
    for (int a = 0; a < MT; ++a) {
        float o[MT];
        wino_at<MT>(s[a], o);  // (A^T M) A
        const int ho = MT * ty + a, wo = MT * tx;
        const bool rok = ho < A.Ho;
        const int64_t e = (((int64_t)n * A.K + k) * A.Ho + ho) * A.Wo + wo;
        if constexpr (sizeof(TY) == 2) {
#pragma unroll
            for (int b = 0; b < MT; ++b)
                st_u16(ry, rok & (wo + b < A.Wo) ? (uint32_t)((e + b) * 2) : OOB_OFF, f32_to_bf16_rne(o[b] + bias));
        } else if (vec) {
            if constexpr (MT == 4) {
                const u32x4 v = {__builtin_bit_cast(uint32_t, o[0] + bias), __builtin_bit_cast(uint32_t, o[1] + bias),
                                 __builtin_bit_cast(uint32_t, o[2] + bias), __builtin_bit_cast(uint32_t, o[3] + bias)};
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, rok ? (uint32_t)(e * 4) : OOB_OFF, 0, 0);
            } else {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                const u32x2 v = {__builtin_bit_cast(uint32_t, o[0] + bias), __builtin_bit_cast(uint32_t, o[1] + bias)};
                __builtin_amdgcn_raw_buffer_store_b64(v, ry, rok ? (uint32_t)(e * 4) : OOB_OFF, 0, 0);
            }
        } else {
#pragma unroll
            for (int b = 0; b < MT; ++b)
                st_f32(ry, rok & (wo + b < A.Wo) ? (uint32_t)((e + b) * 4) : OOB_OFF, o[b] + bias);
        }
    }
}

hipError_t launch_wino_filter(const void* w, void* u, int K, int C, int mt, int dt, hipStream_t stream) {
    const int64_t n = (int64_t)K * C;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL || (mt != 2 && mt != 4) || (dt == CONV2D_BF16 && mt != 2))
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (dt == CONV2D_BF16)
        hipLaunchKernelGGL((wino_filter_kernel<2, uint16_t>), grid, dim3(256), 0, stream,
                           static_cast<const uint16_t*>(w), static_cast<uint16_t*>(u), K, C);
    else if (mt == 2)
        hipLaunchKernelGGL((wino_filter_kernel<2, float>), grid, dim3(256), 0, stream, static_cast<const float*>(w),
                           static_cast<float*>(u), K, C);
    else
        hipLaunchKernelGGL((wino_filter_kernel<4, float>), grid, dim3(256), 0, stream, static_cast<const float*>(w),
                           static_cast<float*>(u), K, C);
    return hipGetLastError();
}

hipError_t launch_wino_input_nhwc(const WinoArgs& a, uint16_t* v, hipStream_t stream) {
    const int64_t n = (int64_t)a.C * a.tc;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL || a.mt != 2) return hipErrorInvalidValue;
    hipLaunchKernelGGL((wino_input_nhwc_kernel<2>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a, v);
    return hipGetLastError();
}

hipError_t launch_wino_input(const WinoArgs& a, float* v, hipStream_t stream) {
    const int64_t n = (int64_t)a.C * a.tc;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL || (a.mt != 2 && a.mt != 4)) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((n + 255) / 256));
    // (with W a multiple of 4 the condition holds for paddings 0 and 1, never for 2)
    const bool vec = a.mt == 4 && a.W % 4 == 0 && (a.pw == 0 || a.pw == 1) && 4 * (a.tw - 1) + 3 < a.W;
    if (a.mt == 2)
        hipLaunchKernelGGL((wino_input_kernel<2, -1>), grid, dim3(256), 0, stream, a, v);
    else if (!vec)
        hipLaunchKernelGGL((wino_input_kernel<4, -1>), grid, dim3(256), 0, stream, a, v);
    else if (a.pw == 0)
        hipLaunchKernelGGL((wino_input_kernel<4, 0>), grid, dim3(256), 0, stream, a, v);
    else
        hipLaunchKernelGGL((wino_input_kernel<4, 1>), grid, dim3(256), 0, stream, a, v);
    return hipGetLastError();
}

hipError_t launch_wino_output(const WinoArgs& a, const float* m, int ydt, hipStream_t stream) {
    const int64_t n = (int64_t)a.K * a.tc;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL || (a.mt != 2 && a.mt != 4)) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (ydt == CONV2D_BF16) {
        if (a.mt != 2) return hipErrorInvalidValue;
        hipLaunchKernelGGL((wino_output_kernel<2, uint16_t>), grid, dim3(256), 0, stream, a, m);
    } else if (a.mt == 2) {
        hipLaunchKernelGGL((wino_output_kernel<2, float>), grid, dim3(256), 0, stream, a, m);
    } else {
        hipLaunchKernelGGL((wino_output_kernel<4, float>), grid, dim3(256), 0, stream, a, m);
    }
    return hipGetLastError();
}

}  // namespace cv
