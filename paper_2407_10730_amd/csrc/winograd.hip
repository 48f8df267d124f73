// winograd.hip -- Winograd minimal-filtering convolution F(2x2, 3x3) (Lavin and Gray, CVPR
// 2016), the transform-based algorithm family the paper names next to GEMM and direct methods
// (Sec. I), for 3x3 filters, stride 1, dilation 1, one group, fp32.
//
// Every 2x2 block of outputs (a tile) is computed from the 4x4 input patch under it:
//   Y = A^T [ (G g G^T) (.) (B^T d B) ] A
// with the element-wise product (.) summed over input channels, which turns the 16 positions
// of the 4x4 transformed domain into 16 independent GEMMs
//   M[xi][k][t] = sum_c U[xi][k][c] * V[xi][c][t]
// (U: transformed filters, V: transformed input patches, t: tile).  The phases map onto the
// timing tool's steps: the filter transform is a pre-convolution reordering of the weights,
// the input transform is the packing, the batched GEMM is the microkernel (the library's MFMA
// GEMM with dense operands, one "group" per position) and the output transform is the
// unpacking, which also adds the bias and writes NCHW y.  Tiles are processed in chunks that
// fit the workspace.
//
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1]
//   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1]
//   A^T = [1 1 1 0; 0 1 -1 -1]
#include "device_common.h"

namespace cv {

// U[xi][k][c] = (G g_kc G^T)[xi]; one thread per (k, c), c fastest (coalesced writes).
__global__ __launch_bounds__(256) void wino_filter_kernel(const float* __restrict__ w, float* __restrict__ u, int K,
                                                          int C) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)K * C) return;
    const float* g = w + i * 9;  // w[k][c][3][3], i = k*C + c
    float t[4][3];               // G g
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const float g0 = g[j], g1 = g[3 + j], g2 = g[6 + j];
        t[0][j] = g0;
        t[1][j] = 0.5f * (g0 + g1 + g2);
        t[2][j] = 0.5f * (g0 - g1 + g2);
        t[3][j] = g2;
    }
    const int64_t plane = (int64_t)K * C;
#pragma unroll
    for (int a = 0; a < 4; ++a) {  // (G g) G^T
        const float h0 = t[a][0], h1 = t[a][1], h2 = t[a][2];
        u[(a * 4 + 0) * plane + i] = h0;
        u[(a * 4 + 1) * plane + i] = 0.5f * (h0 + h1 + h2);
        u[(a * 4 + 2) * plane + i] = 0.5f * (h0 - h1 + h2);
        u[(a * 4 + 3) * plane + i] = h2;
    }
}

// V[xi][c][t - t0] = (B^T d B)[xi] for the tiles t0 .. t0+tc-1 (tile t = (n, th, tw) row-major);
// one thread per (c, tile), tile fastest.
__global__ __launch_bounds__(256) void wino_input_kernel(WinoArgs A, float* __restrict__ v) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)A.C * A.tc) return;
    const int c = (int)(i / A.tc);
    const int tl = (int)(i - (int64_t)c * A.tc);
    const int64_t t = A.t0 + tl;
    const int tiles_img = A.th * A.tw;
    const int n = (int)(t / tiles_img);
    const int r = (int)(t - (int64_t)n * tiles_img);
    const int ty = r / A.tw, tx = r - (r / A.tw) * A.tw;
    const int hi0 = 2 * ty - A.ph, wi0 = 2 * tx - A.pw;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(A.x, A.x_bytes);
    const int64_t plane0 = ((int64_t)n * A.C + c) * A.H;
    float d[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int hi = hi0 + a;
        const bool hok = (unsigned)hi < (unsigned)A.H;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int wi = wi0 + b;
            const bool ok = hok & ((unsigned)wi < (unsigned)A.W);
            d[a][b] = ld_f32(rx, ok ? (uint32_t)(((plane0 + hi) * A.W + wi) * 4) : OOB_OFF);
        }
    }
    float e[4][4];  // B^T d
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        e[0][b] = d[0][b] - d[2][b];
        e[1][b] = d[1][b] + d[2][b];
        e[2][b] = d[2][b] - d[1][b];
        e[3][b] = d[1][b] - d[3][b];
    }
    const int64_t plane = (int64_t)A.C * A.tc;
#pragma unroll
    for (int a = 0; a < 4; ++a) {  // (B^T d) B
        v[(a * 4 + 0) * plane + i] = e[a][0] - e[a][2];
        v[(a * 4 + 1) * plane + i] = e[a][1] + e[a][2];
        v[(a * 4 + 2) * plane + i] = e[a][2] - e[a][1];
        v[(a * 4 + 3) * plane + i] = e[a][1] - e[a][3];
    }
}

// y (the 2x2 block of tile t, clipped at the edges) = A^T M A + bias; one thread per
// (k, tile), tile fastest.
__global__ __launch_bounds__(256) void wino_output_kernel(WinoArgs A, const float* __restrict__ m) {
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
    float q[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) q[a][b] = m[(a * 4 + b) * plane + i];
    float s[2][4];  // A^T M
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        s[0][b] = q[0][b] + q[1][b] + q[2][b];
        s[1][b] = q[1][b] - q[2][b] - q[3][b];
    }
    const float bias = A.bias ? A.bias[k] : 0.0f;
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const float o0 = s[a][0] + s[a][1] + s[a][2] + bias;  // (A^T M) A
        const float o1 = s[a][1] - s[a][2] - s[a][3] + bias;
        const int ho = 2 * ty + a, wo = 2 * tx;
        const bool rok = ho < A.Ho;
        const int64_t e = (((int64_t)n * A.K + k) * A.Ho + ho) * A.Wo + wo;
        st_f32(ry, rok ? (uint32_t)(e * 4) : OOB_OFF, o0);
        st_f32(ry, rok & (wo + 1 < A.Wo) ? (uint32_t)((e + 1) * 4) : OOB_OFF, o1);
    }
}

hipError_t launch_wino_filter(const float* w, float* u, int K, int C, hipStream_t stream) {
    const int64_t n = (int64_t)K * C;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(wino_filter_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, w, u, K, C);
    return hipGetLastError();
}

hipError_t launch_wino_input(const WinoArgs& a, float* v, hipStream_t stream) {
    const int64_t n = (int64_t)a.C * a.tc;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(wino_input_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a, v);
    return hipGetLastError();
}

hipError_t launch_wino_output(const WinoArgs& a, const float* m, hipStream_t stream) {
    const int64_t n = (int64_t)a.K * a.tc;
    if (n < 1 || (n + 255) / 256 > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(wino_output_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a, m);
    return hipGetLastError();
}

}  // namespace cv
