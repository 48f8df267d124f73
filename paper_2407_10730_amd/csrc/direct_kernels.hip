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
#include <algorithm>
#include <cstdlib>
#include <type_traits>

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

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

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

// ------------------------------------------------------------------ grouped (C/g > 1 or K/g > 1)
// One block per (image, GB consecutive groups, band of TR output rows, chunk of KG output
// channels per group).  The input window of the band -- every input row its outputs read,
// with a zero halo -- is staged in LDS next to the filters transposed to [c][tap][KG], so that
// a thread reads one input value per tap and pixel and uses it for all KG output channels,
// and reads the KG filter values of a tap as LDS broadcasts shared by its PX pixels.  Groups
// with few channels are batched GB to a block (their channels are consecutive in x, staged
// at once); a group with many channels is staged CC channels at a time.  Each x element is
// read from HBM once (halo rows of neighbouring bands hit L2); each output is written once.
constexpr int GRP_PX = 2;                 // output pixels per thread
constexpr int GRP_XF = 8192;              // LDS floats for the input window (32 KiB)
constexpr int GRP_WF = 2048;              // LDS floats for the filters (8 KiB)
constexpr int GRP_UNR = 16;               // window loads in flight per thread

template <int KG, typename TX, typename TY>
__global__ __launch_bounds__(DIRECT_THREADS) void grouped_kernel(DirectArgs A, GrpPlan P) {
    extern __shared__ __attribute__((aligned(16))) float glds[];
    float* xs = glds;                              // [channel][in_rows][in_cols]
    float* ws = glds + P.xfloats;                  // [channel][R*S][KG]
    const int G = A.C / A.Cg;
    int b = blockIdx.x;
    const int kc = b % P.kchunks;
    b /= P.kchunks;
    const int band = b % P.nbands;
    b /= P.nbands;
    const int ngb = (G + P.GB - 1) / P.GB;
    const int g0 = (b % ngb) * P.GB;
    const int n = b / ngb;
    const int gn = min(P.GB, G - g0);              // groups of this block
    const int kq0 = kc * KG;                       // first output channel of the chunk, within a group
    const int nk = min(KG, A.Kg - kq0);
    const int ho0 = band * P.TR;
    const int rows = min(P.TR, A.Ho - ho0);
    const int npx = rows * A.Wo;
    const int RS = A.R * A.S;
    const int plane = P.in_rows * P.in_cols;
    const int hi_base = ho0 * A.sh - A.ph;
    const int t = threadIdx.x;
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);
    const TX* wsrc = reinterpret_cast<const TX*>(A.w);

    // window offset of the thread's pixels (pixels past the band read a valid, discarded value)
    int base[GRP_PX];
#pragma unroll
    for (int q = 0; q < GRP_PX; ++q) {
        const int o = t + q * DIRECT_THREADS;
        const int oh = o < npx ? o / A.Wo : 0;
        const int ow = o < npx ? o - oh * A.Wo : 0;
        base[q] = oh * A.sh * P.in_cols + ow * A.sw;
    }

    // stage channels [ch0, ch0 + nch) of x (global channel index) and, for each, the filters
    // of the KG output channels of its group
    auto stage = [&](int ch0, int nch) {
        __syncthreads();  // nobody reads the previous contents any more
        const int total = nch * plane;
        int c = t / plane;  // incremental (channel, row, column) of element i
        int rem = t - c * plane;
        int rr = rem / P.in_cols;
        int cc = rem - rr * P.in_cols;
        const int dc = DIRECT_THREADS / plane, drem = DIRECT_THREADS - dc * plane;
        const int drr = drem / P.in_cols, dcc = drem - drr * P.in_cols;
        // GRP_UNR loads in flight per thread before their LDS stores
        for (int i0 = t; i0 < total; i0 += GRP_UNR * DIRECT_THREADS) {
            float v[GRP_UNR];
#pragma unroll
            for (int u = 0; u < GRP_UNR; ++u) {
                const int hi = hi_base + rr, wi = cc - A.pw;
                const bool ok = (i0 + u * DIRECT_THREADS < total) & ((unsigned)hi < (unsigned)A.H) &
                                ((unsigned)wi < (unsigned)A.W);
                const int64_t e = (((int64_t)n * A.C + ch0 + c) * A.H + hi) * A.W + wi;
                v[u] = dk_load(rx, ok, e, (TX*)nullptr);
                c += dc;
                rr += drr;
                cc += dcc;
                if (cc >= P.in_cols) {
                    cc -= P.in_cols;
                    ++rr;
                }
                if (rr >= P.in_rows) {
                    rr -= P.in_rows;
                    ++c;
                }
            }
#pragma unroll
            for (int u = 0; u < GRP_UNR; ++u)
                if (i0 + u * DIRECT_THREADS < total) xs[i0 + u * DIRECT_THREADS] = v[u];
        }
        for (int c2 = 0; c2 < nch; ++c2) {
            const int ch = ch0 + c2;
            const int gi = ch / A.Cg;
            const int64_t wbase = ((int64_t)gi * A.Kg + kq0) * A.Cg + (ch - gi * A.Cg);
            for (int j = t; j < RS * KG; j += DIRECT_THREADS) {
                const int k = j % KG;
                const int tap = j / KG;
                float v = 0.0f;
                if (k < nk) {
                    const TX raw = wsrc[(wbase + (int64_t)k * A.Cg) * RS + tap];
                    if constexpr (sizeof(TX) == 4) v = __builtin_bit_cast(float, raw);
                    else v = __builtin_bit_cast(float, (uint32_t)raw << 16);
                }
                ws[c2 * RS * KG + j] = v;
            }
        }
        __syncthreads();
    };

    float acc[GRP_PX][KG];
    // channels [c0, c0 + ccn) staged at LDS channel slot s0
    auto accumulate = [&](int s0, int ccn) {
        for (int c = 0; c < ccn; ++c) {
            const float* xc = xs + (s0 + c) * plane;
            const float* wc = ws + (s0 + c) * RS * KG;
            for (int r = 0; r < A.R; ++r) {
                const float* xr = xc + r * A.dh * P.in_cols;
                const float* wr = wc + r * A.S * KG;
                for (int sx = 0; sx < A.S; ++sx) {
                    float wv[KG];
                    if constexpr (KG % 4 == 0) {
#pragma unroll
                        for (int k4 = 0; k4 < KG / 4; ++k4) {
                            const f32x4 v = *reinterpret_cast<const f32x4*>(wr + sx * KG + 4 * k4);
                            wv[4 * k4] = v[0]; wv[4 * k4 + 1] = v[1]; wv[4 * k4 + 2] = v[2]; wv[4 * k4 + 3] = v[3];
                        }
                    } else {
#pragma unroll
                        for (int k = 0; k < KG; ++k) wv[k] = wr[sx * KG + k];
                    }
#pragma unroll
                    for (int q = 0; q < GRP_PX; ++q) {
                        const float xv = xr[base[q] + sx * A.dw];
#pragma unroll
                        for (int k = 0; k < KG; ++k) acc[q][k] = __builtin_fmaf(wv[k], xv, acc[q][k]);
                    }
                }
            }
        }
    };
    auto store = [&](int gi) {
        const int kglob0 = gi * A.Kg + kq0;
        float bv[KG];
#pragma unroll
        for (int k = 0; k < KG; ++k) bv[k] = (A.bias && k < nk) ? A.bias[kglob0 + k] : 0.0f;
#pragma unroll
        for (int q = 0; q < GRP_PX; ++q) {
            const int o = t + q * DIRECT_THREADS;
            if (o >= npx) continue;
            const int oh = ho0 + o / A.Wo;
            const int ow = o % A.Wo;
#pragma unroll
            for (int k = 0; k < KG; ++k) {
                if (k >= nk) break;
                const int64_t off = (((int64_t)n * A.K + kglob0 + k) * A.Ho + oh) * A.Wo + ow;
                if constexpr (sizeof(TY) == 4)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, acc[q][k] + bv[k]), ry,
                                                          (uint32_t)(off * 4), 0, 0);
                else
                    __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(acc[q][k] + bv[k]), ry,
                                                          (uint32_t)(off * 2), 0, 0);
            }
        }
    };
    auto zero = [&]() {
#pragma unroll
        for (int q = 0; q < GRP_PX; ++q)
#pragma unroll
            for (int k = 0; k < KG; ++k) acc[q][k] = 0.0f;
    };

    if (P.GB > 1) {
        // the block's groups are staged together (P.CC >= GB * Cg)
        stage(g0 * A.Cg, gn * A.Cg);
        for (int gg = 0; gg < gn; ++gg) {
            zero();
            accumulate(gg * A.Cg, A.Cg);
            store(g0 + gg);
        }
    } else {
        zero();
        for (int c0 = 0; c0 < A.Cg; c0 += P.CC) {
            const int ccn = min(P.CC, A.Cg - c0);
            stage(g0 * A.Cg + c0, ccn);
            accumulate(0, ccn);
        }
        store(g0);
    }
}

// ------------------------------------------------------------------ depthwise (C/g = 1)
// Every output plane (n, k) reads one input plane (n, k / (K/g)).  A block stages
// whole input rows of one or more planes into LDS with a zero halo (16-byte loads
// when W % 4 == 0), then each thread produces strips of 4 consecutive outputs of
// one row: for stride 1 / dilation 1 the S + 3 input values of a filter row are
// read once and reused by the 4 outputs.  HBM traffic is one read of x and one
// write of y; filter taps and bias of the block's planes sit in LDS.
constexpr int DW_LDS_FLOATS = 8192;   // 32 KiB input tile
constexpr int DW_MAX_PLANES = 64;

struct DwPlan {
    int32_t PB, TH, IR, LDW, LPAD, nbands, WS;
};

// One block per work item (a group of PB planes x a band of TH output rows).  The input
// tile lives in dynamic LDS sized to the item, so many blocks fit on a CU and their tile
// loads overlap (the kernel is bound by HBM bandwidth, which needs many bytes in flight).
// TILEF is the tile capacity in floats: 4096 (16 KiB) when a plane fits, 8192 (32 KiB) for
// tall planes cut into bands, where a larger band re-reads fewer halo rows.
constexpr int DWP_TILE_SMALL = 4096;
constexpr int DWP_TILE_LARGE = 8192;

template <int R, int S, int ST, int DL, int TILEF, typename TX, typename TY>
__global__ __launch_bounds__(DIRECT_THREADS) void dw_kernel(DirectArgs A, DwPlan P) {
    constexpr int DWP_VMAX = TILEF / 4 / DIRECT_THREADS;  // 16-byte loads per thread
    constexpr int DWP_SMAX = TILEF / DIRECT_THREADS;      // 4-byte loads per thread
    // With stride 2 and an even dilation (or a 1x1 filter) every window reads only the even
    // rows of the tile: only those are loaded and stored (tile row j holds input row
    // hi_base + 2j), which halves the tile and the loads.
    constexpr bool EVEN_ROWS = ST == 2 && (DL % 2 == 0 || R == 1);
    constexpr int RSTEP = EVEN_ROWS ? 2 : 1;  // input rows per tile row
    extern __shared__ __attribute__((aligned(16))) float tile[];  // PB * IR * LDW floats
    __shared__ float wsh[DW_MAX_PLANES * R * S];
    __shared__ float bsh[DW_MAX_PLANES];
    __shared__ int32_t pbase[DW_MAX_PLANES];  // element offset of the input plane of local plane lp
    const int t = threadIdx.x;
    const int planes_total = A.N * A.K;
    const int band = blockIdx.x % P.nbands;
    const int pl0 = (blockIdx.x / P.nbands) * P.PB;
    const int npl = min(P.PB, planes_total - pl0);
    const int oh0 = band * P.TH;
    const int nrows = min(P.TH, A.Ho - oh0);
    const int hi_base = oh0 * A.sh - A.ph;
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);
    const TX* wp = reinterpret_cast<const TX*>(A.w);

    for (int i = t; i < npl * R * S; i += DIRECT_THREADS) {
        const int k = (pl0 + i / (R * S)) % A.K;
        const TX v = wp[(int64_t)k * R * S + i % (R * S)];
        if constexpr (sizeof(TX) == 4) wsh[i] = __builtin_bit_cast(float, v);
        else wsh[i] = __builtin_bit_cast(float, (uint32_t)v << 16);
    }
    for (int i = t; i < npl; i += DIRECT_THREADS) {
        const int pl = pl0 + i;
        const int n = pl / A.K;
        const int k = pl - n * A.K;
        bsh[i] = A.bias ? A.bias[k] : 0.0f;
        pbase[i] = (int32_t)(((int64_t)n * A.C + k / A.Kg) * A.H * A.W);
    }
    __syncthreads();

    // input tile: row tr of local plane lp holds input row hi_base + tr, input column w sits at
    // w + LPAD.  All of a thread's loads are issued before any is written to LDS.
    {
        const int VW = (A.W & 3) == 0 ? 4 : 1;
        const int LDWV = P.LDW / VW;
        const int total = npl * P.IR * LDWV;
        const int srow = DIRECT_THREADS / LDWV, scol = DIRECT_THREADS - srow * LDWV;
        int row = t / LDWV;
        int cg = t - row * LDWV;
        int lp = row / P.IR;
        int tr = row - lp * P.IR;
        auto step = [&]() {
            cg += scol;
            int adv = srow;
            if (cg >= LDWV) {
                cg -= LDWV;
                ++adv;
            }
            tr += adv;
            while (tr >= P.IR) {
                tr -= P.IR;
                ++lp;
            }
        };
        if (VW == 4) {
            f32x4 vreg[DWP_VMAX];
#pragma unroll
            for (int u = 0; u < DWP_VMAX; ++u) {
                const int e = t + u * DIRECT_THREADS;
                const int hi = hi_base + RSTEP * tr;
                const int w0 = 4 * cg - P.LPAD;
                const bool ok = (e < total) & ((unsigned)hi < (unsigned)A.H) & ((unsigned)w0 < (unsigned)A.W);
                const int32_t idx = ok ? pbase[lp] + hi * A.W + w0 : 0;
                if constexpr (sizeof(TX) == 4) {
                    vreg[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                           rx, ok ? (uint32_t)idx * 4u : OOB_OFF, 0, 0));
                } else {
                    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                    const u32x2 h = __builtin_bit_cast(
                        u32x2, __builtin_amdgcn_raw_buffer_load_b64(rx, ok ? (uint32_t)idx * 2u : OOB_OFF, 0, 0));
                    vreg[u] = f32x4{__builtin_bit_cast(float, h[0] << 16), __builtin_bit_cast(float, h[0] & 0xFFFF0000u),
                                    __builtin_bit_cast(float, h[1] << 16), __builtin_bit_cast(float, h[1] & 0xFFFF0000u)};
                }
                step();
            }
#pragma unroll
            for (int u = 0; u < DWP_VMAX; ++u) {
                const int e = t + u * DIRECT_THREADS;
                if (e < total) *reinterpret_cast<f32x4*>(&tile[4 * e]) = vreg[u];
            }
        } else {
            float sreg[DWP_SMAX];
#pragma unroll
            for (int u = 0; u < DWP_SMAX; ++u) {
                const int e = t + u * DIRECT_THREADS;
                const int hi = hi_base + RSTEP * tr;
                const int w = cg - P.LPAD;
                const bool ok = (e < total) & ((unsigned)hi < (unsigned)A.H) & ((unsigned)w < (unsigned)A.W);
                sreg[u] = dk_load(rx, ok, ok ? pbase[lp] + hi * A.W + w : 0, (TX*)nullptr);
                step();
            }
#pragma unroll
            for (int u = 0; u < DWP_SMAX; ++u) {
                const int e = t + u * DIRECT_THREADS;
                if (e < total) tile[e] = sreg[u];
            }
        }
    }
    __syncthreads();

    // outputs: each thread computes a block of VR rows x HC columns.  It walks the NR input
    // rows under the block once; each row's RB values are read from LDS once and feed every
    // output row whose window contains it (which rows those are is known at compile time),
    // so a 3x3 stride-1 block reads 2.25 LDS values per output instead of 9.  Consecutive
    // lanes take consecutive column blocks; with Wo % 4 == 0 a row of the block is stored
    // with one 16-byte (fp32) or 8-byte (bf16) store.
    // HC shrinks for large filters, whose NR x RB input window would not fit the registers
    constexpr int VR = 4, HC = R <= 3 ? 4 : (R == 5 ? 2 : 1);
    constexpr int NR = (VR - 1) * ST + (R - 1) * DL + 1;
    constexpr int RB = (HC - 1) * ST + (S - 1) * DL + 1;
    auto compute = [&](auto uniform_w) {
        constexpr bool UW = decltype(uniform_w)::value;
        const int nrb = (nrows + VR - 1) / VR;
        const int ncb = (A.Wo + HC - 1) / HC;
        const int per_plane = nrb * ncb;
        const int items = npl * per_plane;
        const bool vec = HC == 4 && (A.Wo & 3) == 0;
        float wreg[R * S];
        if constexpr (UW) {
#pragma unroll
            for (int i = 0; i < R * S; ++i) wreg[i] = wsh[i];
        }
        for (int q = t; q < items; q += DIRECT_THREADS) {
            const int lp = q / per_plane;
            const int rem = q - lp * per_plane;
            const int rb = rem / ncb;
            const int cb = rem - rb * ncb;
            if constexpr (!UW) {
#pragma unroll
                for (int i = 0; i < R * S; ++i) wreg[i] = wsh[lp * R * S + i];
            }
            const float bias = bsh[lp];
            const int orow0 = rb * VR;
            const int ow0 = cb * HC;
            const float* rp = &tile[(lp * P.IR + orow0 * ST / RSTEP) * P.LDW + P.LPAD - A.pw + ow0 * ST];
            float acc[VR][HC];
#pragma unroll
            for (int v = 0; v < VR; ++v)
#pragma unroll
                for (int h = 0; h < HC; ++h) acc[v][h] = bias;
#pragma unroll
            for (int rr = 0; rr < NR; ++rr) {
                float xrow[RB];
#pragma unroll
                for (int c = 0; c < RB; ++c) xrow[c] = rp[(rr / RSTEP) * P.LDW + c];  // (odd rows unused)
#pragma unroll
                for (int v = 0; v < VR; ++v) {
                    // input row rr is filter row r of output row v when rr = v*ST + r*DL
                    const int d = rr - v * ST;
                    if (d < 0 || d % DL != 0 || d / DL >= R) continue;  // resolved at compile time
                    const int r = d / DL;
#pragma unroll
                    for (int h = 0; h < HC; ++h)
#pragma unroll
                        for (int sx = 0; sx < S; ++sx)
                            acc[v][h] = __builtin_fmaf(xrow[h * ST + sx * DL], wreg[r * S + sx], acc[v][h]);
                }
            }
            const int64_t o0 = ((int64_t)(pl0 + lp) * A.Ho + oh0 + orow0) * A.Wo + ow0;
#pragma unroll
            for (int v = 0; v < VR; ++v) {
                const bool rok = orow0 + v < nrows;
                const int64_t o = o0 + (int64_t)v * A.Wo;
                bool done = false;
                if constexpr (HC == 4) {
                    if (vec) {
                        if constexpr (sizeof(TY) == 4) {
                            const u32x4_t val = {__builtin_bit_cast(uint32_t, acc[v][0]), __builtin_bit_cast(uint32_t, acc[v][1]),
                                                 __builtin_bit_cast(uint32_t, acc[v][2]), __builtin_bit_cast(uint32_t, acc[v][3])};
                            __builtin_amdgcn_raw_buffer_store_b128(val, ry, rok ? (uint32_t)(o * 4) : OOB_OFF, 0, 0);
                        } else {
                            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                            const u32x2 val = {(uint32_t)dk_f32_to_bf16(acc[v][0]) | ((uint32_t)dk_f32_to_bf16(acc[v][1]) << 16),
                                               (uint32_t)dk_f32_to_bf16(acc[v][2]) | ((uint32_t)dk_f32_to_bf16(acc[v][3]) << 16)};
                            __builtin_amdgcn_raw_buffer_store_b64(val, ry, rok ? (uint32_t)(o * 2) : OOB_OFF, 0, 0);
                        }
                        done = true;
                    }
                }
                if (!done) {
#pragma unroll
                    for (int h = 0; h < HC; ++h) {
                        const bool ok = rok & (ow0 + h < A.Wo);
                        if constexpr (sizeof(TY) == 4)
                            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, acc[v][h]), ry,
                                                                  ok ? (uint32_t)((o + h) * 4) : OOB_OFF, 0, 0);
                        else
                            __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(acc[v][h]), ry,
                                                                  ok ? (uint32_t)((o + h) * 2) : OOB_OFF, 0, 0);
                    }
                }
            }
        }
    };
    if (npl == 1) compute(std::true_type{});
    else compute(std::false_type{});
}

// Host plan of the depthwise kernel; returns false when the shape needs the generic kernel.
static bool dw_plan(const DirectArgs& a, int sw_t, int dw_t, int tilef, DwPlan* p) {
    const int WS = (a.Wo + 3) / 4;
    const int LPAD = (a.pw + 3) / 4 * 4;
    // columns read by the last block of 4 outputs (ragged blocks read past Wo - 1)
    const int maxcol = LPAD - a.pw + (WS * 4 - 1) * sw_t + (a.S - 1) * dw_t;
    int LDW = (maxcol + 1 + 3) / 4 * 4;
    if (LDW < LPAD + a.W) LDW = (LPAD + a.W + 3) / 4 * 4;
    // rows of the tile: TH output rows rounded up to whole strips of 4; with stride 2 and an
    // even dilation or a 1x1 filter only the even input rows are kept
    const bool even = a.sh == 2 && (a.dh % 2 == 0 || a.R == 1);
    auto ir = [&](int th) {
        const int rows = (((th + 3) / 4) * 4 - 1) * a.sh + (a.R - 1) * a.dh + 1;
        return even ? (rows + 1) / 2 : rows;
    };
    int TH, PB;
    if (a.Ho * WS <= 1024) {
        TH = a.Ho;
        PB = 1024 / (a.Ho * WS);
        if (PB < 1) PB = 1;
        if (PB > DW_MAX_PLANES) PB = DW_MAX_PLANES;
        while (PB > 1 && PB * ir(TH) * LDW > tilef) --PB;
    } else {
        PB = 1;
        TH = 1024 / WS;
        if (TH < 1) TH = 1;
        if (TH > a.Ho) TH = a.Ho;
    }
    while (TH > 1 && PB * ir(TH) * LDW > tilef) --TH;
    if (PB * ir(TH) * LDW > tilef) return false;
    p->PB = PB;
    p->TH = TH;
    p->IR = ir(TH);
    p->LDW = LDW;
    p->LPAD = LPAD;
    p->nbands = (a.Ho + TH - 1) / TH;
    p->WS = WS;
    return true;
}

template <int R, int S, int ST, int DL, int TILEF>
static hipError_t launch_dw_t(const DirectArgs& a, const DwPlan& p, int xdt, int ydt, hipStream_t stream) {
    const int64_t planes = (int64_t)a.N * a.K;
    const int64_t nblocks = (planes + p.PB - 1) / p.PB * p.nbands;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
    const size_t lds = (size_t)p.PB * p.IR * p.LDW * sizeof(float);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((dw_kernel<R, S, ST, DL, TILEF, float, float>), grid, dim3(DIRECT_THREADS), lds, stream,
                           a, p);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((dw_kernel<R, S, ST, DL, TILEF, uint16_t, uint16_t>), grid, dim3(DIRECT_THREADS), lds,
                           stream, a, p);
    else
        hipLaunchKernelGGL((dw_kernel<R, S, ST, DL, TILEF, uint16_t, float>), grid, dim3(DIRECT_THREADS), lds,
                           stream, a, p);
    return hipGetLastError();
}

// Depthwise fast path: square 1/3/5/7 filters, equal strides of 1 or 2, equal dilations of 1 or 2.
static hipError_t try_launch_dw(const DirectArgs& a, int xdt, int ydt, hipStream_t stream, bool* launched) {
    *launched = false;
    if (a.Cg != 1 || a.R != a.S || (a.sw != 1 && a.sw != 2) || (a.dw != 1 && a.dw != 2)) return hipSuccess;
    if (a.sh != a.sw || a.dh != a.dw) return hipSuccess;
    if (a.R != 1 && a.R != 3 && a.R != 5 && a.R != 7) return hipSuccess;
    DwPlan p, pl;
    bool large = false;
    if (!dw_plan(a, a.sw, a.dw, DWP_TILE_SMALL, &p)) {
        if (!dw_plan(a, a.sw, a.dw, DWP_TILE_LARGE, &p)) return hipSuccess;
        large = true;
    } else if (p.nbands > 1 && dw_plan(a, a.sw, a.dw, DWP_TILE_LARGE, &pl) && pl.nbands < p.nbands) {
        p = pl;
        large = true;
    }
    *launched = true;
#define CV_DW(RV, SWV, DWV)                                                                   \
    if (a.R == RV && a.sw == SWV && a.dw == DWV)                                              \
        return large ? launch_dw_t<RV, RV, SWV, DWV, DWP_TILE_LARGE>(a, p, xdt, ydt, stream) \
                     : launch_dw_t<RV, RV, SWV, DWV, DWP_TILE_SMALL>(a, p, xdt, ydt, stream);
#define CV_DW4(RV) CV_DW(RV, 1, 1) CV_DW(RV, 1, 2) CV_DW(RV, 2, 1) CV_DW(RV, 2, 2)
    CV_DW4(1) CV_DW4(3) CV_DW4(5) CV_DW4(7)
#undef CV_DW4
#undef CV_DW
    *launched = false;
    return hipSuccess;
}

// ------------------------------------------------------------------ depthwise, streamed rows
// Stride-1 depthwise layers (C/g = 1) with 3x3 filters at dilation 1 or 2, or 5x5 and 7x7
// filters at dilation 1, on planes up to 256 output columns wide (bf16: an even number of
// input columns).  The block-per-plane kernel above spends far more vector
// instructions per output than its R*R FMAs (tile staging through registers and LDS, a
// barrier, a division pair per work item, a mostly idle last wave), so it is bound by
// instruction issue rather than by memory, worst in bf16.  Here a wave (a workgroup of its
// own) takes UPW units, a unit being a band of BR output rows of one (n, k) plane; lane l
// computes a strip of 4 consecutive outputs, column block l % ncb of unit l / ncb, walking
// down the band, and reads its inputs straight from memory (the L1 and L2 caches serve the
// columns that neighbouring strips share; no LDS, no barrier):
//   * per input row a lane loads the RB = 4 + (R-1)*DL values under its strip with 16-byte
//     (and 8- or 4-byte) loads, NS = (R-1)*DL + 1 rows ahead of the one it sums, into a
//     ring of registers, so each wave keeps NS rows of loads in flight;
//   * values left or right of the image are zeroed with one select (fp32) or one byte
//     permute (bf16, which also moves the 2-byte value into the top of an fp32 word) per
//     value, from per-lane selectors fixed at the start; rows above or below the image
//     are not loaded (their loads target no record and return zero);
//   * each input row feeds the R output rows whose windows hold it; the NS output rows in
//     progress rotate through as many accumulator sets, so the row that received its last
//     filter row is stored (4 outputs per 16-/8-byte store when Wo % 4 == 0) and its set
//     restarts from the bias while the walk goes on.
// Per output that is R*R FMAs plus about (RB/4)/R selects and one instruction of addressing
// and storing.  In bf16 at dilation 1 the products go through the packed 2-term dot product
// instead: the loaded words hold two neighbouring input values each, and one v_dot2 takes two
// taps of one output against a word of the filter row (weights prepacked as pairs for both
// alignments of a tap run), so a 3x3 output costs 6 instructions and no conversions.  bf16
// words start at an even column (ODD: the padding is odd, so the strip's first value is the
// top half of the first word).
struct DwrPlan {
    int32_t ncb, upw, br, ir, nbands, units;
    int32_t wpb;               // waves per block (independent; 1 or 4)
    uint32_t m_ncb;            // lane / ncb = (lane * m_ncb) >> 16 for lane < 64
    FastDiv fd_nb, fd_k, fd_kg;  // unit -> plane, plane -> image, channel -> input channel
};

__device__ __forceinline__ uint32_t dk_fdiv(uint32_t n, FastDiv f) { return (__umulhi(n, f.m) + n) >> f.s; }

// Words a lane loads per input row.
__host__ __device__ constexpr int dwr_words(int R, int DL, bool bf, bool odd) {
    return bf ? (4 + (R - 1) * DL + (odd ? 1 : 0) + 1) / 2 : 4 + (R - 1) * DL;
}

template <int R, int DL, bool ODD, int WPB, typename TX, typename TY>
__global__ __launch_bounds__(64 * WPB) void dw_rows_kernel(DirectArgs A, DwrPlan P) {
    constexpr int HALO = (R - 1) * DL;
    constexpr int NS = HALO + 1;  // output rows in progress
    constexpr int RB = 4 + HALO;  // input values under a strip of 4 outputs
    constexpr bool BF = sizeof(TX) == 2;
    constexpr bool DOT = BF && DL == 1;
    constexpr int NW = dwr_words(R, DL, BF, ODD);  // words loaded per row
    // rows of loads in flight per lane: one per output row in progress (deeper rings, with
    // the bands shortened to match, measured slower)
    constexpr int D = NS;
    constexpr int NP = (R + 1) / 2;                              // filter-row words per alignment
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    const int l = threadIdx.x & 63;
    const int U0 = (int)(blockIdx.x * WPB + (WPB > 1 ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) : 0)) * P.upw;
    if (WPB > 1 && U0 >= P.units) return;  // the whole wave: past the last unit
    const int nu = min(P.upw, P.units - U0);
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);

    const int ul = (int)(((uint32_t)l * P.m_ncb) >> 16);
    const int cb = l - ul * P.ncb;
    const bool lane_ok = ul < nu;
    const int U = U0 + (lane_ok ? ul : 0);
    const int plane = (int)dk_fdiv((uint32_t)U, P.fd_nb);
    const int band = U - plane * P.nbands;
    const int n = (int)dk_fdiv((uint32_t)plane, P.fd_k);
    const int k = plane - n * A.K;
    const int oh0 = band * P.br;
    const int nv = lane_ok ? min(P.br, A.Ho - oh0) : 0;  // output rows this lane stores
    const int hi0 = oh0 - A.ph;                          // input row of walk step 0
    const int ow0 = 4 * cb;
    const int c0 = ow0 - A.pw;                           // input column of the strip's value 0
    const int cw = BF ? c0 - (ODD ? 1 : 0) : c0;         // column of the first loaded word
    const int xplane = (n * A.C + (int)dk_fdiv((uint32_t)k, P.fd_kg)) * A.H * A.W;
    const int row0 = xplane + hi0 * A.W + cw;            // element offset of (hi0, cw), signed

    // per-word masks: the loaded values left or right of the image are zeroed (bf16: per
    // half-word); the non-dot bf16 path turns each value into fp32 with a byte permute whose
    // selector also zeroes it
    uint32_t msk[NW];
    uint32_t sel[BF && !DOT ? RB : 1];
#pragma unroll
    for (int c = 0; c < NW; ++c) {
        if constexpr (BF) {
            const int p0 = cw + 2 * c;
            msk[c] = ((unsigned)p0 < (unsigned)A.W ? 0x0000FFFFu : 0u) |
                     ((unsigned)(p0 + 1) < (unsigned)A.W ? 0xFFFF0000u : 0u);
        } else {
            msk[c] = (unsigned)(c0 + c) < (unsigned)A.W ? 0xFFFFFFFFu : 0u;
        }
    }
    if constexpr (BF && !DOT) {
#pragma unroll
        for (int t = 0; t < RB; ++t) {
            const int h = t + (ODD ? 1 : 0);
            const bool ok = (unsigned)(c0 + t) < (unsigned)A.W;
            sel[t] = ok ? ((h & 1) ? 0x03020C0Cu : 0x01000C0Cu) : 0x0C0C0C0Cu;
        }
    }

    const TX* wp = reinterpret_cast<const TX*>(A.w) + (int64_t)k * R * R;
    float wr[DOT ? 1 : R * R];
    uint32_t wpk[DOT ? R : 1][2][NP];  // [row][alignment][word]: bf16 weight pairs
    if constexpr (DOT) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            uint32_t h[R + 1];
#pragma unroll
            for (int q = 0; q < R; ++q) h[q] = (uint32_t)wp[r * R + q];
            h[R] = 0;
            // alignment 0: the run starts in a low half: (w0,w1) (w2,w3) ...
            // alignment 1: it starts in a high half: (0,w0) (w1,w2) ...
#pragma unroll
            for (int q = 0; q < NP; ++q) {
                wpk[r][0][q] = h[2 * q] | (h[2 * q + 1] << 16);
                wpk[r][1][q] = (q == 0 ? 0u : h[2 * q - 1]) | (h[2 * q] << 16);
            }
        }
    } else {
#pragma unroll
        for (int q = 0; q < R * R; ++q) {
            if constexpr (BF) wr[q] = __builtin_bit_cast(float, (uint32_t)wp[q] << 16);
            else wr[q] = __builtin_bit_cast(float, wp[q]);
        }
    }
    const float bias = A.bias ? A.bias[k] : 0.0f;
    const bool vec = (A.Wo & 3) == 0;
    const uint32_t yrow0 = (uint32_t)((plane * A.Ho + oh0) * A.Wo + ow0);

    // The wide loads of a strip at the left or right edge start before column 0 or end past
    // column W - 1 (those values are masked), which is still inside x except in the first
    // and the last input plane; a wave that holds one of those loads word by word, each word
    // checked against the ends of x.
    const int plane_lo = (int)dk_fdiv((uint32_t)U0, P.fd_nb);
    const int plane_hi = (int)dk_fdiv((uint32_t)(U0 + nu - 1), P.fd_nb);
    const int n_lo = (int)dk_fdiv((uint32_t)plane_lo, P.fd_k), n_hi = (int)dk_fdiv((uint32_t)plane_hi, P.fd_k);
    const int ip_lo = n_lo * A.C + (int)dk_fdiv((uint32_t)(plane_lo - n_lo * A.K), P.fd_kg);
    const int ip_hi = n_hi * A.C + (int)dk_fdiv((uint32_t)(plane_hi - n_hi * A.K), P.fd_kg);
    const bool edge_wave = ip_lo == 0 || ip_hi == A.N * A.C - 1;
    const int x_elems = A.N * A.C * A.H * A.W;
    constexpr int EPW = BF ? 2 : 1;  // elements per loaded word

    // the NW words of walk step i (input row hi0 + i), zero for rows outside the image
    auto load_row = [&](int i, uint32_t (&wv)[NW]) {
        const int hi = hi0 + i;
        const bool ok = (unsigned)hi < (unsigned)A.H;
        const int e0 = row0 + i * A.W;  // element offset of the first word
        if (edge_wave) {
#pragma unroll
            for (int c = 0; c < NW; ++c) {
                const int e = e0 + c * EPW;
                const bool in = ok & (e >= 0) & (e < x_elems);
                wv[c] = __builtin_amdgcn_raw_buffer_load_b32(rx, in ? (uint32_t)e * (uint32_t)sizeof(TX) : OOB_OFF,
                                                             0, 0);
            }
            return;
        }
        const uint32_t off = ok ? (uint32_t)e0 * (uint32_t)sizeof(TX) : OOB_OFF;
#pragma unroll
        for (int c = 0; c < NW; c += 4) {
            if (c + 4 <= NW) {
                const u32x4_t v =
                    __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 16 * (c / 4), 0));
#pragma unroll
                for (int q = 0; q < 4; ++q) wv[c + q] = v[q];
            } else if (NW - c == 3) {
                typedef uint32_t u32x3_t __attribute__((ext_vector_type(3)));
                const u32x3_t v =
                    __builtin_bit_cast(u32x3_t, __builtin_amdgcn_raw_buffer_load_b96(rx, off, 16 * (c / 4), 0));
                wv[c] = v[0];
                wv[c + 1] = v[1];
                wv[c + 2] = v[2];
            } else if (NW - c == 2) {
                const u32x2_t v =
                    __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rx, off, 16 * (c / 4), 0));
                wv[c] = v[0];
                wv[c + 1] = v[1];
            } else {
                wv[c] = __builtin_amdgcn_raw_buffer_load_b32(rx, off, 16 * (c / 4), 0);
            }
        }
    };

    auto store_row = [&](const float (&v)[4], int od) {
        const bool rok = od < nv;
        const uint32_t e = yrow0 + (uint32_t)(od * A.Wo);
        if (vec) {
            if constexpr (sizeof(TY) == 4) {
                const u32x4_t val = {__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                                     __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])};
                __builtin_amdgcn_raw_buffer_store_b128(val, ry, rok ? e * 4u : OOB_OFF, 0, 0);
            } else {
                const u32x2_t val = {
                    __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{v[0], v[1]}, bf16x2_t)),
                    __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{v[2], v[3]}, bf16x2_t))};
                __builtin_amdgcn_raw_buffer_store_b64(val, ry, rok ? e * 2u : OOB_OFF, 0, 0);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool ok = rok & (ow0 + j < A.Wo);
                if constexpr (sizeof(TY) == 4)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[j]), ry,
                                                          ok ? (e + j) * 4u : OOB_OFF, 0, 0);
                else
                    __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(v[j]), ry, ok ? (e + j) * 2u : OOB_OFF,
                                                          0, 0);
            }
        }
    };

    float acc[NS][4];
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[q][j] = bias;

    uint32_t ring[D][NW];
#pragma unroll
    for (int q = 0; q < D; ++q)
        if (q < P.ir) load_row(q, ring[q]);

    // walk: input row i feeds output rows i - r*DL (r = 0 .. R-1); after it, output row
    // i - HALO is complete.  Output row o accumulates in set o % NS and row i sits in ring
    // slot i % D (D a multiple of NS); the walk is unrolled by D so every index is a constant.
    for (int base = 0; base < P.ir; base += D) {
#pragma unroll
        for (int s = 0; s < D; ++s) {
            const int i = base + s;
            if (i < P.ir) {
                uint32_t wv[NW];
#pragma unroll
                for (int c = 0; c < NW; ++c) wv[c] = ring[s][c] & msk[c];
                if (i + D < P.ir) load_row(i + D, ring[s]);
                float xv[DOT ? 1 : RB];
                if constexpr (!DOT) {
#pragma unroll
                    for (int t = 0; t < RB; ++t) {
                        if constexpr (BF) {
                            const int h = t + (ODD ? 1 : 0);
                            xv[t] = __builtin_bit_cast(float, __builtin_amdgcn_perm(0u, wv[h >> 1], sel[t]));
                        } else {
                            xv[t] = __builtin_bit_cast(float, wv[t]);
                        }
                    }
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int o = i - r * DL;
                    const int q = ((s - r * DL) % NS + NS) % NS;  // = o mod NS (D % NS == 0)
                    if (o >= 0 && o < P.br) {
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            if constexpr (DOT) {
                                // taps of output j sit at half-words j + ODD ... j + ODD + R - 1
                                const int p0 = j + (ODD ? 1 : 0);
#pragma unroll
                                for (int m = 0; m < NP; ++m)
                                    acc[q][j] = __builtin_amdgcn_fdot2_f32_bf16(
                                        __builtin_bit_cast(bf16x2_t, wv[(p0 >> 1) + m]),
                                        __builtin_bit_cast(bf16x2_t, wpk[r][p0 & 1][m]), acc[q][j], false);
                            } else {
#pragma unroll
                                for (int sx = 0; sx < R; ++sx)
                                    acc[q][j] = __builtin_fmaf(xv[j + sx * DL], wr[r * R + sx], acc[q][j]);
                            }
                        }
                    }
                }
                const int od = i - HALO;
                if (od >= 0) {
                    const int q = (s + 1) % NS;  // = od mod NS
                    store_row(acc[q], od);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[q][j] = bias;
                }
            }
        }
    }
}

// Bands: enough units for about 4096 waves (16 per CU) where the planes allow, at least 8
// output rows each (the halo rows are loaded again by the next band).  Measured on 56x56
// planes: 2 bands 21.2 us (bf16), whole planes 30.4, 4 bands 22.3.
static bool dwr_plan(const DirectArgs& a, int xdt, DwrPlan* p) {
    if (a.Cg != 1 || a.R != a.S || a.sh != 1 || a.sw != 1 || a.dh != a.dw) return false;
    // 3x3 at dilation 1 or 2, 5x5 and 7x7 at dilation 1: the others' ring of rows in flight
    // ((R-1)*DL + 1 rows of 4 + (R-1)*DL values) would not fit the registers
    if (!(a.R == 3 && (a.dh == 1 || a.dh == 2)) && !((a.R == 5 || a.R == 7) && a.dh == 1)) return false;
    if (a.Ho < 1 || a.Wo < 1) return false;
    if (xdt == CONV2D_BF16 && a.W % 2 != 0) return false;  // bf16 rows are loaded as aligned words
    const int ncb = (a.Wo + 3) / 4;
    if (ncb > 64) return false;
    const int upw = 64 / ncb;
    if (4 * upw * ncb < 3 * 64) return false;  // fewer than three quarters of the lanes busy
    const int64_t planes = (int64_t)a.N * a.K;
    // target wave count: 3x3 filters at dilation 1 split planes into more bands (their 2 halo
    // rows cost less than the shorter row chains gain: N32 2048 28x28 bf16 51 -> 46 us); at
    // dilation 2 (4 halo rows: N1 1024 224x224 40 -> 43 us) and for 5x5 and 7x7 (more
    // arithmetic per row: N32 256 112x112 5x5 3 % slower) whole planes or long bands stay.
    // CONV2D_DWR_WAVES overrides it.
    // Many planes of up to 32 columns at 3x3 dilation 1 take blocks of 4 independent waves
    // and twice the waves (bf16, us, one-wave -> 4-wave blocks: N32 2048 28x28 45.3 -> 43.7,
    // N32 1024 14x14 15.5 either way; with fewer planes it loses: N32 256 28x28 8.07 -> 8.26,
    // N8 96 32x32 5.35 -> 5.71; the 56x56 and 112x112 layers 0.5-1.5 % slower).
    // CONV2D_DWR_WPB = 1 or 4 overrides the block size.
    const bool small = a.R == 3 && a.dh == 1 && a.Wo <= 32 && planes >= 32768;
    const char* tw = std::getenv("CONV2D_DWR_WAVES");
    const int64_t waves = tw && std::atoi(tw) > 0 ? std::atoi(tw)
                          : (a.R == 3 && a.dh == 1 ? (small ? 32768 : 16384) : 4096);
    const char* tb = std::getenv("CONV2D_DWR_WPB");
    p->wpb = tb && (tb[0] == '1' || tb[0] == '4') ? tb[0] - '0' : (small ? 4 : 1);
    if (p->wpb == 4 && !(a.R == 3 && a.dh == 1)) p->wpb = 1;  // (instantiated for 3x3 at dilation 1)
    int64_t nb = (waves * upw + planes - 1) / planes;
    const int nb_max = (a.Ho + 7) / 8;
    if (nb > nb_max) nb = nb_max;
    if (nb < 1) nb = 1;
    const int br = (a.Ho + (int)nb - 1) / (int)nb;
    const int nbands = (a.Ho + br - 1) / br;
    const int64_t units = planes * nbands;
    if (units > 0x7fffffffLL - upw) return false;
    p->ncb = ncb;
    p->upw = upw;
    p->br = br;
    p->ir = br + (a.R - 1) * a.dh;
    p->nbands = nbands;
    p->units = (int32_t)units;
    p->m_ncb = (65536u + (uint32_t)ncb - 1) / (uint32_t)ncb;
    p->fd_nb = make_fastdiv((uint32_t)nbands);
    p->fd_k = make_fastdiv((uint32_t)a.K);
    p->fd_kg = make_fastdiv((uint32_t)a.Kg);
    return true;
}

template <int R, int DL, int WPB>
static hipError_t launch_dwr_t(const DirectArgs& a, const DwrPlan& p, int xdt, int ydt, hipStream_t stream) {
    const int64_t wv = (p.units + p.upw - 1) / p.upw;
    dim3 grid((unsigned)((wv + WPB - 1) / WPB)), block(64 * WPB);
    const bool odd = a.pw & 1;
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((dw_rows_kernel<R, DL, false, WPB, float, float>), grid, block, 0, stream, a, p);
    else if (ydt == CONV2D_BF16) {
        if (odd) hipLaunchKernelGGL((dw_rows_kernel<R, DL, true, WPB, uint16_t, uint16_t>), grid, block, 0, stream, a, p);
        else hipLaunchKernelGGL((dw_rows_kernel<R, DL, false, WPB, uint16_t, uint16_t>), grid, block, 0, stream, a, p);
    } else {
        if (odd) hipLaunchKernelGGL((dw_rows_kernel<R, DL, true, WPB, uint16_t, float>), grid, block, 0, stream, a, p);
        else hipLaunchKernelGGL((dw_rows_kernel<R, DL, false, WPB, uint16_t, float>), grid, block, 0, stream, a, p);
    }
    return hipGetLastError();
}

// Taken for bf16 inputs: on the 56x56 depthwise layer it runs 21 us against the block
// kernel's 29 us, while in fp32 the block kernel's contiguous plane loads win (33 against
// 36 us).  CONV2D_DW_ROWS=1 takes it for fp32 inputs as well, 0 for none (the tests run
// every shape through both kernels).
static hipError_t try_launch_dw_rows(const DirectArgs& a, int xdt, int ydt, hipStream_t stream, bool* launched) {
    *launched = false;
    const char* env = std::getenv("CONV2D_DW_ROWS");
    if (env && env[0] == '0') return hipSuccess;
    if (xdt == CONV2D_F32 && !(env && env[0] == '1')) return hipSuccess;
    DwrPlan p;
    if (!dwr_plan(a, xdt, &p)) return hipSuccess;
    *launched = true;
    if (a.R == 3 && a.dh == 1)
        return p.wpb == 4 ? launch_dwr_t<3, 1, 4>(a, p, xdt, ydt, stream) : launch_dwr_t<3, 1, 1>(a, p, xdt, ydt, stream);
    if (a.R == 3 && a.dh == 2) return launch_dwr_t<3, 2, 1>(a, p, xdt, ydt, stream);
    if (a.R == 5 && a.dh == 1) return launch_dwr_t<5, 1, 1>(a, p, xdt, ydt, stream);
    if (a.R == 7 && a.dh == 1) return launch_dwr_t<7, 1, 1>(a, p, xdt, ydt, stream);
    *launched = false;
    return hipSuccess;
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

// ------------------------------------------------------------------ grouped, row strips
// Grouped layers with square filters, equal strides of 1 or 2 and no dilation: each thread
// owns a strip of GS_HC consecutive outputs of one row for KG output channels of its group.
// Per input channel and filter row it reads the RB input values under the strip once and
// uses every one for all the taps and pixels that need it, and it reads the KG weights of a
// tap with one broadcast, so a 3x3 stride-1 strip does 48 FMAs per 9 LDS reads (the
// per-pixel kernel above: 8 per 3).  A block holds GB groups x TR output rows x all column
// strips (one item per thread) and stages their input windows (16-byte loads when the row
// length allows) and filters; a group with more channels than fit is staged in chunks.
constexpr int GS_HC = 4;       // outputs per strip
constexpr int GS_XF = 8192;    // LDS floats for the windows (32 KiB)
constexpr int GS_WF = 2048;    // LDS floats for the filters

struct GsPlan {
    int32_t TR, GB, CC, IR, LDW, LPAD, ncb, nbands, kchunks, xfloats, lds_bytes;
    FastDiv fd_cpl, fd_ldw, fd_ir, fd_cg;  // staging: chunks per line, line width, rows, channels per group
    FastDiv fd_kch, fd_nb, fd_ngb, fd_ncb, fd_tr;  // block and thread decomposition
};

// Up to 4 output channels per strip the kernel fits in 73 registers, 7 blocks per CU; left to
// itself the compiler took 100 (5 blocks per CU, 20 % slower on C/g = 4).
// VW: rows of W % 4 == 0 columns, staged 16 bytes at a time (else element by element; the two
// staging loops are separate instances, so neither one's registers weigh on the other)
template <int R, int ST, int KG, bool VW, typename TX, typename TY>
__global__ __launch_bounds__(DIRECT_THREADS) __attribute__((amdgpu_waves_per_eu(KG <= 4 ? 7 : 1))) void
grouped_strip_kernel(DirectArgs A, GsPlan P) {
    constexpr int S = R;
    constexpr int RB = (GS_HC - 1) * ST + S;  // input columns under a strip
    extern __shared__ __attribute__((aligned(16))) float gsl[];
    float* xs = gsl;                // [CC][IR][LDW]
    float* ws = gsl + P.xfloats;    // [CC][R*S][KG]
    const int G = A.C / A.Cg;
    // block -> (image, group batch, band, channel chunk) and thread -> (group, row, strip)
    // with host-computed magic numbers (the compiler's divisions cost ~30 instructions each)
    uint32_t b = blockIdx.x;
    uint32_t b1 = dk_fdiv(b, P.fd_kch);
    const int kc = (int)(b - b1 * (uint32_t)P.kchunks);
    uint32_t b2 = dk_fdiv(b1, P.fd_nb);
    const int band = (int)(b1 - b2 * (uint32_t)P.nbands);
    const int ngb = (G + P.GB - 1) / P.GB;
    const uint32_t b3 = dk_fdiv(b2, P.fd_ngb);
    const int g0 = (int)(b2 - b3 * (uint32_t)ngb) * P.GB;
    const int n = (int)b3;
    const int gn = min(P.GB, G - g0);
    const int kq0 = kc * KG;
    const int nk = min(KG, A.Kg - kq0);
    const int ho0 = band * P.TR;
    const int rows = min(P.TR, A.Ho - ho0);
    const int hi_base = ho0 * ST - A.ph;
    const int plane = P.IR * P.LDW;
    const int t = threadIdx.x;
    // the thread's strip: column block cb, output row rv of the band, group gg of the block
    const uint32_t t1 = dk_fdiv((uint32_t)t, P.fd_ncb);
    const int cb = t - (int)t1 * P.ncb;
    const uint32_t t2 = dk_fdiv(t1, P.fd_tr);
    const int rv = (int)(t1 - t2 * (uint32_t)P.TR);
    const int gg = (int)t2;
    const bool act = gg < gn && rv < rows;
    const int ow0 = cb * GS_HC;
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);
    const __amdgpu_buffer_rsrc_t rw = dk_rsrc(A.w, A.w_bytes);

    // the bias goes in first: the FMAs add the products to it
    float acc[GS_HC][KG];
    {
        const int kb = (g0 + gg) * A.Kg + kq0;
#pragma unroll
        for (int k = 0; k < KG; ++k) {
            const float bv = A.bias && act && k < nk ? A.bias[kb + k] : 0.0f;
#pragma unroll
            for (int h = 0; h < GS_HC; ++h) acc[h][k] = bv;
        }
    }

    // the block's channels: all channels of its gn groups (staged at once when GB > 1), or the
    // Cg channels of its one group, CC at a time
    const int cper = P.GB > 1 ? gn * A.Cg : A.Cg;
    const int chb = g0 * A.Cg;  // first global input channel of the block
    for (int c0 = 0; c0 < cper; c0 += P.CC) {
        const int ccn = min(P.CC, cper - c0);
        __syncthreads();  // nobody reads the previous chunk any more
        // windows: line (lc, tr) holds input row hi_base + tr of channel chb + c0 + lc at
        // columns j = wi + LPAD
        // (element offsets fit 32 bits: x is below 2 GiB)
        const int cbase = (n * A.C + chb + c0) * A.H;  // row index of the chunk's first channel
        if constexpr (VW) {
            const int cpl = P.LDW / 4;  // 16-byte chunks per line (the odd last word is padding)
            const int total = ccn * P.IR * cpl;
            // up to 4 output channels per strip, two chunks per thread per trip: both loads go
            // out before the first LDS write waits (one load round trip per two chunks; g=64
            // 46.5 -> 44.9 us; four chunks spilled registers under the 7-wave cap, and the
            // 8-channel kernel measured 3 % slower with two)
            constexpr int UB = KG <= 4 ? 2 : 1;
            for (int i0 = t; i0 < total; i0 += UB * DIRECT_THREADS) {
                f32x4 v[UB];
                int dst[UB];
#pragma unroll
                for (int u = 0; u < UB; ++u) {
                    const int i = i0 + u * DIRECT_THREADS;
                    const int line = (int)dk_fdiv((uint32_t)i, P.fd_cpl);
                    const int q = i - line * cpl;
                    const int lc = (int)dk_fdiv((uint32_t)line, P.fd_ir);
                    const int tr = line - lc * P.IR;
                    const int hi = hi_base + tr, w0 = 4 * q - P.LPAD;
                    const bool ok = (i < total) & ((unsigned)hi < (unsigned)A.H) & ((unsigned)w0 < (unsigned)A.W);
                    const int e = (cbase + lc * A.H + hi) * A.W + w0;
                    if constexpr (sizeof(TX) == 4) {
                        v[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                             rx, ok ? (uint32_t)(e * 4) : OOB_OFF, 0, 0));
                    } else {
                        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                        const u32x2 hh = __builtin_bit_cast(
                            u32x2, __builtin_amdgcn_raw_buffer_load_b64(rx, ok ? (uint32_t)(e * 2) : OOB_OFF, 0, 0));
                        v[u] = f32x4{__builtin_bit_cast(float, hh[0] << 16), __builtin_bit_cast(float, hh[0] & 0xFFFF0000u),
                                     __builtin_bit_cast(float, hh[1] << 16), __builtin_bit_cast(float, hh[1] & 0xFFFF0000u)};
                    }
                    dst[u] = i < total ? line * P.LDW + 4 * q : -1;
                }
#pragma unroll
                for (int u = 0; u < UB; ++u) {
                    if (dst[u] >= 0) {
                        float* d = &xs[dst[u]];  // 4-byte aligned (odd line width)
                        d[0] = v[u][0];
                        d[1] = v[u][1];
                        d[2] = v[u][2];
                        d[3] = v[u][3];
                    }
                }
            }
        } else {
            const int total = ccn * P.IR * P.LDW;
            // (as above: EB elements per thread per trip, their loads issued together; N32
            // 1024 14x14 g=256 33.6 -> 24.4 us, 2048 7x7 g=512 27.9 -> 22.2 us)
            constexpr int EB = KG <= 4 ? 4 : 1;
            for (int i0 = t; i0 < total; i0 += EB * DIRECT_THREADS) {
                float v[EB];
#pragma unroll
                for (int u = 0; u < EB; ++u) {
                    const int i = i0 + u * DIRECT_THREADS;
                    const int line = (int)dk_fdiv((uint32_t)i, P.fd_ldw);
                    const int j = i - line * P.LDW;
                    const int lc = (int)dk_fdiv((uint32_t)line, P.fd_ir);
                    const int tr = line - lc * P.IR;
                    const int hi = hi_base + tr, wi = j - P.LPAD;
                    const bool ok = (i < total) & ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
                    v[u] = dk_load(rx, ok, ok ? (cbase + lc * A.H + hi) * A.W + wi : 0, (TX*)nullptr);
                }
#pragma unroll
                for (int u = 0; u < EB; ++u)
                    if (i0 + u * DIRECT_THREADS < total) xs[i0 + u * DIRECT_THREADS] = v[u];
            }
        }
        // filters: ws[lc][tap][k] = w[group's output channel kq0 + k][channel within group][tap]
        // (32-bit element index and a range-checked buffer load: the 64-bit address arithmetic
        // of a plain load cost about 45 vector instructions per element)
        for (int i = t; i < ccn * R * S * KG; i += DIRECT_THREADS) {
            const int k = i % KG;
            const int tap = (i / KG) % (R * S);
            const int lc = i / (KG * R * S);
            const int ch = chb + c0 + lc;
            const int gi = (int)dk_fdiv((uint32_t)ch, P.fd_cg);
            const int widx = ((gi * A.Kg + kq0 + k) * A.Cg + (ch - gi * A.Cg)) * (R * S) + tap;
            ws[i] = dk_load(rw, k < nk, widx, (TX*)nullptr);
        }
        __syncthreads();
        if (act) {
            const int lc0 = P.GB > 1 ? gg * A.Cg : 0;
            const int lcn = P.GB > 1 ? A.Cg : ccn;
            for (int lc = lc0; lc < lc0 + lcn; ++lc) {
                const float* xc = xs + lc * plane + rv * ST * P.LDW + P.LPAD - A.pw + ow0 * ST;
                const float* wc = ws + lc * (R * S * KG);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    float xr[RB];
#pragma unroll
                    for (int j = 0; j < RB; ++j) xr[j] = xc[r * P.LDW + j];
#pragma unroll
                    for (int sx = 0; sx < S; ++sx) {
                        float wv[KG];
                        if constexpr (KG % 4 == 0) {
#pragma unroll
                            for (int k4 = 0; k4 < KG / 4; ++k4) {
                                const f32x4 v = *reinterpret_cast<const f32x4*>(wc + (r * S + sx) * KG + 4 * k4);
                                wv[4 * k4] = v[0]; wv[4 * k4 + 1] = v[1]; wv[4 * k4 + 2] = v[2]; wv[4 * k4 + 3] = v[3];
                            }
                        } else {
#pragma unroll
                            for (int k = 0; k < KG; ++k) wv[k] = wc[(r * S + sx) * KG + k];
                        }
#pragma unroll
                        for (int h = 0; h < GS_HC; ++h)
#pragma unroll
                            for (int k = 0; k < KG; ++k) acc[h][k] = __builtin_fmaf(xr[h * ST + sx], wv[k], acc[h][k]);
                    }
                }
            }
        }
    }
    if (!act) return;
    const int kglob0 = (g0 + gg) * A.Kg + kq0;
    const int oh = ho0 + rv;
    const int howo = A.Ho * A.Wo;
    const int o0 = ((n * A.K + kglob0) * A.Ho + oh) * A.Wo + ow0;
    const bool vec = (A.Wo & 3) == 0;
#pragma unroll
    for (int k = 0; k < KG; ++k) {
        if (k >= nk) break;
        // (y holds fewer than 2^31 elements: 32-bit index arithmetic)
        const int o = o0 + k * howo;
        if (vec) {
            if constexpr (sizeof(TY) == 4) {
                const u32x4_t val = {__builtin_bit_cast(uint32_t, acc[0][k]), __builtin_bit_cast(uint32_t, acc[1][k]),
                                     __builtin_bit_cast(uint32_t, acc[2][k]), __builtin_bit_cast(uint32_t, acc[3][k])};
                __builtin_amdgcn_raw_buffer_store_b128(val, ry, (uint32_t)(o * 4), 0, 0);
            } else {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                const u32x2 val = {(uint32_t)dk_f32_to_bf16(acc[0][k]) | ((uint32_t)dk_f32_to_bf16(acc[1][k]) << 16),
                                   (uint32_t)dk_f32_to_bf16(acc[2][k]) | ((uint32_t)dk_f32_to_bf16(acc[3][k]) << 16)};
                __builtin_amdgcn_raw_buffer_store_b64(val, ry, (uint32_t)(o * 2), 0, 0);
            }
        } else {
#pragma unroll
            for (int h = 0; h < GS_HC; ++h) {
                const bool ok = ow0 + h < A.Wo;
                if constexpr (sizeof(TY) == 4)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, acc[h][k]), ry,
                                                          ok ? (uint32_t)((o + h) * 4) : OOB_OFF, 0, 0);
                else
                    __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(acc[h][k]), ry,
                                                          ok ? (uint32_t)((o + h) * 2) : OOB_OFF, 0, 0);
            }
        }
    }
}

// Row-strip plan: TR output rows x GB groups per block with one strip per thread; false when
// the shape does not fit (the per-pixel grouped kernel takes it then).
static bool gs_plan(const DirectArgs& a, int KG, GsPlan* p) {
    if (a.R != a.S || a.sh != a.sw || (a.sh != 1 && a.sh != 2) || a.dh != 1 || a.dw != 1) return false;
    if (a.R != 1 && a.R != 3 && a.R != 5 && a.R != 7) return false;
    const int ncb = (a.Wo + GS_HC - 1) / GS_HC;
    if (ncb > DIRECT_THREADS) return false;
    const int LPAD = (a.pw + 3) / 4 * 4;
    const int maxcol = LPAD - a.pw + (ncb * GS_HC - 1) * a.sw + a.S - 1;
    int LDW = std::max(maxcol + 1, LPAD + a.W);
    // an odd line width (4m + 1 words, the last one never read) moves each row one LDS bank
    // over: the lanes of a wave read 4 words apart within a row, so with a multiple-of-32
    // width the rows of one wave met in the same 8 banks (up to 5-way conflicts at 56 columns)
    LDW = (LDW + 3) / 4 * 4 + 1;
    const int RS = a.R * a.S;
    const int G = a.C / a.Cg;
    // rows per block: as many as the threads hold (one strip each), at most the plane
    int tr = std::max(1, std::min(a.Ho, DIRECT_THREADS / ncb));
    auto ir = [&](int r) { return (r - 1) * a.sh + a.R; };
    while (tr > 1 && (int64_t)ir(tr) * LDW > GS_XF) --tr;
    // equal bands (56 rows: 4 x 14 rather than 3 x 18 + 2)
    tr = (a.Ho + (a.Ho + tr - 1) / tr - 1) / ((a.Ho + tr - 1) / tr);
    const int64_t win = (int64_t)ir(tr) * LDW;
    if (win > GS_XF || RS * KG > GS_WF) return false;
    const int fit = (int)std::min<int64_t>(GS_XF / win, GS_WF / (RS * KG));
    // groups per block: the threads left over by the rows, and whole groups' channels in LDS
    // (filling the idle threads of 56-row planes with more groups in shorter bands measured
    // slower: C/g 4, bands of 8 with two groups 64 us against 54 with bands of 14)
    int gb = std::max(1, std::min({G, DIRECT_THREADS / (ncb * tr), fit / a.Cg}));
    p->TR = tr;
    p->GB = gb;
    p->CC = gb > 1 ? gb * a.Cg : std::min(a.Cg, fit);
    p->IR = ir(tr);
    p->LDW = LDW;
    p->LPAD = LPAD;
    p->ncb = ncb;
    p->nbands = (a.Ho + tr - 1) / tr;
    p->kchunks = (a.Kg + KG - 1) / KG;
    p->xfloats = (int)(p->CC * win);
    p->lds_bytes = (p->xfloats + p->CC * RS * KG) * 4;
    p->fd_cpl = make_fastdiv((uint32_t)(LDW / 4));
    p->fd_ldw = make_fastdiv((uint32_t)LDW);
    p->fd_ir = make_fastdiv((uint32_t)p->IR);
    p->fd_cg = make_fastdiv((uint32_t)a.Cg);
    p->fd_kch = make_fastdiv((uint32_t)p->kchunks);
    p->fd_nb = make_fastdiv((uint32_t)p->nbands);
    p->fd_ngb = make_fastdiv((uint32_t)((G + gb - 1) / gb));
    p->fd_ncb = make_fastdiv((uint32_t)ncb);
    p->fd_tr = make_fastdiv((uint32_t)tr);
    const int64_t blocks = (int64_t)a.N * ((G + gb - 1) / gb) * p->nbands * p->kchunks;
    return blocks <= 0x7fffffffLL && p->CC >= 1;
}

template <int R, int ST, int KG, bool VW>
static hipError_t launch_gs_v(const DirectArgs& a, const GsPlan& p, int xdt, int ydt, hipStream_t stream) {
    const int G = a.C / a.Cg;
    dim3 grid((unsigned)((int64_t)a.N * ((G + p.GB - 1) / p.GB) * p.nbands * p.kchunks));
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((grouped_strip_kernel<R, ST, KG, VW, float, float>), grid, dim3(DIRECT_THREADS),
                           p.lds_bytes, stream, a, p);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((grouped_strip_kernel<R, ST, KG, VW, uint16_t, uint16_t>), grid, dim3(DIRECT_THREADS),
                           p.lds_bytes, stream, a, p);
    else
        hipLaunchKernelGGL((grouped_strip_kernel<R, ST, KG, VW, uint16_t, float>), grid, dim3(DIRECT_THREADS),
                           p.lds_bytes, stream, a, p);
    return hipGetLastError();
}

template <int R, int ST, int KG>
static hipError_t launch_gs_t(const DirectArgs& a, const GsPlan& p, int xdt, int ydt, hipStream_t stream) {
    return (a.W & 3) == 0 ? launch_gs_v<R, ST, KG, true>(a, p, xdt, ydt, stream)
                          : launch_gs_v<R, ST, KG, false>(a, p, xdt, ydt, stream);
}

// Row-strip fast path for grouped layers (G > 1, C/g > 1 or K/g > 1): KG = 1, 2, 4 or 8 output
// channels per strip (chunks of 8 beyond).  CONV2D_GROUPED_STRIP=0 keeps the per-pixel kernel.
static hipError_t try_launch_grouped_strip(const DirectArgs& a, int xdt, int ydt, hipStream_t stream,
                                           bool* launched) {
    *launched = false;
    const char* env = std::getenv("CONV2D_GROUPED_STRIP");
    if ((env && env[0] == '0') || a.C == a.Cg) return hipSuccess;
    const int KG = a.Kg <= 1 ? 1 : a.Kg <= 2 ? 2 : a.Kg <= 4 ? 4 : 8;
    GsPlan p;
    if (!gs_plan(a, KG, &p)) return hipSuccess;
    *launched = true;
#define CV_GS(RV, STV, KGV) \
    if (a.R == RV && a.sh == STV && KG == KGV) return launch_gs_t<RV, STV, KGV>(a, p, xdt, ydt, stream);
#define CV_GS_K(RV, STV) CV_GS(RV, STV, 1) CV_GS(RV, STV, 2) CV_GS(RV, STV, 4) CV_GS(RV, STV, 8)
    CV_GS_K(1, 1) CV_GS_K(1, 2) CV_GS_K(3, 1) CV_GS_K(3, 2) CV_GS_K(5, 1) CV_GS_K(5, 2) CV_GS_K(7, 1) CV_GS_K(7, 2)
#undef CV_GS_K
#undef CV_GS
    *launched = false;
    return hipSuccess;
}

// Grouped kernel plan for KG output channels per block; false when the shape does not fit.
static bool grp_plan(const DirectArgs& a, int KG, GrpPlan* p) {
    const int in_cols = (a.Wo - 1) * a.sw + (a.S - 1) * a.dw + 1;
    auto in_rows = [&](int tr) { return (tr - 1) * a.sh + (a.R - 1) * a.dh + 1; };
    const int RS = a.R * a.S;
    if (a.Wo > GRP_PX * DIRECT_THREADS || RS * KG > GRP_WF) return false;
    int tr = std::max(1, std::min(a.Ho, GRP_PX * DIRECT_THREADS / a.Wo));
    while (tr > 1 && (int64_t)in_rows(tr) * in_cols > GRP_XF) --tr;
    const int64_t window = (int64_t)in_rows(tr) * in_cols;
    if (window > GRP_XF) return false;
    p->TR = tr;
    p->in_rows = in_rows(tr);
    p->in_cols = in_cols;
    // channels that fit: the window and the filters of each
    const int fit = (int)std::min<int64_t>(GRP_XF / window, (int64_t)(GRP_WF / (RS * KG)));
    if (fit < 1) return false;
    const int G = a.C / a.Cg;
    // groups with few channels go GB to a block, about 16 channels' worth
    p->GB = std::max(1, std::min({G, 16 / a.Cg, fit / a.Cg}));
    p->CC = p->GB > 1 ? p->GB * a.Cg : std::min(a.Cg, fit);
    p->xfloats = (int)(((int64_t)p->CC * window + 3) / 4 * 4);
    p->lds_bytes = (p->xfloats + p->CC * RS * KG) * 4;
    p->nbands = (a.Ho + tr - 1) / tr;
    p->kchunks = (a.Kg + KG - 1) / KG;
    const int64_t blocks = (int64_t)a.N * ((G + p->GB - 1) / p->GB) * p->nbands * p->kchunks;
    return blocks <= 0x7fffffffLL;
}

template <int KG>
static hipError_t launch_grp_t(const DirectArgs& a, const GrpPlan& p, int xdt, int ydt, hipStream_t stream) {
    const int G = a.C / a.Cg;
    dim3 grid((unsigned)((int64_t)a.N * ((G + p.GB - 1) / p.GB) * p.nbands * p.kchunks));
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((grouped_kernel<KG, float, float>), grid, dim3(DIRECT_THREADS), p.lds_bytes, stream, a, p);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((grouped_kernel<KG, uint16_t, uint16_t>), grid, dim3(DIRECT_THREADS), p.lds_bytes, stream,
                           a, p);
    else
        hipLaunchKernelGGL((grouped_kernel<KG, uint16_t, float>), grid, dim3(DIRECT_THREADS), p.lds_bytes, stream,
                           a, p);
    return hipGetLastError();
}

// Grouped fast path: KG = the smallest of 1, 2, 4, 8, 16 that covers K/g (chunks of 16 beyond).
static hipError_t try_launch_grouped(const DirectArgs& a, int xdt, int ydt, hipStream_t stream, bool* launched) {
    *launched = false;
    const int KG = a.Kg <= 1 ? 1 : a.Kg <= 2 ? 2 : a.Kg <= 4 ? 4 : a.Kg <= 8 ? 8 : 16;
    GrpPlan p;
    if (!grp_plan(a, KG, &p)) return hipSuccess;
    *launched = true;
    switch (KG) {
        case 1: return launch_grp_t<1>(a, p, xdt, ydt, stream);
        case 2: return launch_grp_t<2>(a, p, xdt, ydt, stream);
        case 4: return launch_grp_t<4>(a, p, xdt, ydt, stream);
        case 8: return launch_grp_t<8>(a, p, xdt, ydt, stream);
        default: return launch_grp_t<16>(a, p, xdt, ydt, stream);
    }
}

int64_t grouped_blocks(const DirectArgs& a) {
    const int KG = a.Kg <= 1 ? 1 : a.Kg <= 2 ? 2 : a.Kg <= 4 ? 4 : a.Kg <= 8 ? 8 : 16;
    GrpPlan p;
    if (!grp_plan(a, KG, &p)) return 0;
    return (int64_t)a.N * ((a.C / a.Cg + p.GB - 1) / p.GB) * p.nbands * p.kchunks;
}

// ------------------------------------------------------------------ few output channels
// Ungrouped layers with at most 4 output channels (image-to-image heads and the like): a GEMM
// tile of 32 rows would leave 7/8 or more of every MFMA idle, so the vector ALUs compute them.
// A thread owns one output pixel and walks a range of input channels (the reduction is split
// over blockIdx.y into ranges so that the grid fills the chip) and all R x S taps: it reads each
// input value once through the caches (neighbouring pixels share their windows there) and does
// K FMAs with it.  The weights of a chunk of SK_CW channels sit in LDS and are read at
// wave-uniform addresses (broadcast).  With one range the thread adds the bias and writes y;
// otherwise it writes fp32 partial sums [range][K][P] and the unpack kernel adds the ranges in
// order, then the bias (deterministic).
constexpr int SK_CW = 16;

template <int KK, int RR, typename TX, typename TY>
__global__ __launch_bounds__(256) void smallk_kernel(DirectArgs A, SmallKArgs S) {
    constexpr int RS = RR * RR;
    __shared__ float wl[KK * SK_CW * RS];
    const int t = threadIdx.x;
    const int HoWo = A.Ho * A.Wo;
    const int64_t P = (int64_t)A.N * HoWo;
    const int64_t p = (int64_t)blockIdx.x * 256 + t;
    const bool pok = p < P;
    const int n = pok ? (int)(p / HoWo) : 0;
    const int hw = pok ? (int)(p - (int64_t)n * HoWo) : 0;
    const int ho = hw / A.Wo, wo = hw - (hw / A.Wo) * A.Wo;
    const int hi0 = ho * A.sh - A.ph, wi0 = wo * A.sw - A.pw;
    const int c_begin = blockIdx.y * S.cper;
    const int c_end = min(A.C, c_begin + S.cper);
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const TX* wp = reinterpret_cast<const TX*>(A.w);
    float acc[KK];
#pragma unroll
    for (int k = 0; k < KK; ++k) acc[k] = 0.0f;
    for (int cc = c_begin; cc < c_end; cc += SK_CW) {
        const int cn = min(SK_CW, c_end - cc);
        __syncthreads();  // the previous chunk's weights are no longer read
        for (int i = t; i < KK * cn * RS; i += 256) {
            const int k = i / (cn * RS);
            const int rem = i - k * (cn * RS);
            const TX v = wp[((int64_t)k * A.C + cc) * RS + rem];  // w[k][c][r][s]
            float f;
            if constexpr (sizeof(TX) == 4) f = __builtin_bit_cast(float, v);
            else f = __builtin_bit_cast(float, (uint32_t)v << 16);
            wl[k * SK_CW * RS + rem] = f;
        }
        __syncthreads();
        for (int c = 0; c < cn; ++c) {
            const int64_t plane = ((int64_t)n * A.C + cc + c) * A.H;
#pragma unroll
            for (int r = 0; r < RR; ++r) {
                const int hi = hi0 + r * A.dh;
                const bool hok = pok & ((unsigned)hi < (unsigned)A.H);
                const int64_t row = (plane + hi) * A.W;
                float xv[RR];
#pragma unroll
                for (int sx = 0; sx < RR; ++sx) {
                    const int wi = wi0 + sx * A.dw;
                    xv[sx] = dk_load(rx, hok & ((unsigned)wi < (unsigned)A.W), row + wi, (TX*)nullptr);
                }
#pragma unroll
                for (int sx = 0; sx < RR; ++sx)
#pragma unroll
                    for (int k = 0; k < KK; ++k)
                        acc[k] = __builtin_fmaf(xv[sx], wl[(k * SK_CW + c) * RS + r * RR + sx], acc[k]);
            }
        }
    }
    if (!pok) return;
    if (S.part) {
#pragma unroll
        for (int k = 0; k < KK; ++k) S.part[((int64_t)blockIdx.y * KK + k) * P + p] = acc[k];
        return;
    }
    const __amdgpu_buffer_rsrc_t ry = dk_rsrc(A.y, A.y_bytes);
#pragma unroll
    for (int k = 0; k < KK; ++k) {
        const float v = acc[k] + (A.bias ? A.bias[k] : 0.0f);
        const int64_t o = ((int64_t)n * KK + k) * HoWo + hw;
        if constexpr (sizeof(TY) == 4)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), ry, (uint32_t)(o * 4), 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b16(dk_f32_to_bf16(v), ry, (uint32_t)(o * 2), 0, 0);
    }
}

bool smallk_supported(const DirectArgs& a) {
    return a.Cg == a.C && a.Kg == a.K && a.K >= 1 && a.K <= 4 && a.R == a.S &&
           (a.R == 1 || a.R == 3 || a.R == 5 || a.R == 7);
}

// Channel ranges for a grid of about 2048 blocks (at least SK_CW channels each); 1 = no split.
int smallk_ranges(const DirectArgs& a) {
    const int64_t P = (int64_t)a.N * a.Ho * a.Wo;
    const int64_t pblocks = (P + 255) / 256;
    int64_t ranges = (2048 + pblocks - 1) / pblocks;
    ranges = std::min<int64_t>(ranges, (a.C + SK_CW - 1) / SK_CW);
    while (ranges > 1 && ranges * a.K * P * 4 > ((int64_t)256 << 20)) --ranges;
    return (int)std::max<int64_t>(ranges, 1);
}

template <int KK, int RR>
static hipError_t launch_smallk_t(const DirectArgs& a, const SmallKArgs& sk, int ranges, int xdt, int ydt,
                                  hipStream_t stream) {
    const int64_t P = (int64_t)a.N * a.Ho * a.Wo;
    const dim3 grid((unsigned)((P + 255) / 256), (unsigned)ranges);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((smallk_kernel<KK, RR, float, float>), grid, dim3(256), 0, stream, a, sk);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((smallk_kernel<KK, RR, uint16_t, uint16_t>), grid, dim3(256), 0, stream, a, sk);
    else
        hipLaunchKernelGGL((smallk_kernel<KK, RR, uint16_t, float>), grid, dim3(256), 0, stream, a, sk);
    return hipGetLastError();
}

hipError_t launch_smallk(const DirectArgs& a, float* part, int ranges, int xdt, int ydt, hipStream_t stream) {
    const int64_t P = (int64_t)a.N * a.Ho * a.Wo;
    if (!smallk_supported(a) || ranges < 1 || ranges > 65535 || (ranges > 1) != (part != nullptr) ||
        (P + 255) / 256 > 0x7fffffffLL)
        return hipErrorInvalidValue;
    SmallKArgs sk{};
    sk.cper = (a.C + ranges - 1) / ranges;
    sk.part = part;
#define CV_SK(KV, RV) \
    if (a.K == KV && a.R == RV) return launch_smallk_t<KV, RV>(a, sk, ranges, xdt, ydt, stream);
#define CV_SK4(RV) CV_SK(1, RV) CV_SK(2, RV) CV_SK(3, RV) CV_SK(4, RV)
    CV_SK4(1) CV_SK4(3) CV_SK4(5) CV_SK4(7)
#undef CV_SK4
#undef CV_SK
    return hipErrorInvalidValue;
}

// ------------------------------------------------------------------ NHWC depthwise
// Depthwise layers (one input and one output channel per group, C a multiple of 4) with NHWC x
// and y: a thread takes 4 adjacent channels (8 in bf16 when C is a multiple of 8, one 16-byte
// load) of dwn_px() consecutive output pixels of one row.
// Per filter tap it loads the 4 channels' weights from the [R*S][C] copy once and one x run
// per pixel (16 bytes fp32, 8 bytes bf16); a tap in the padding reads zero through the buffer
// bounds.  Consecutive threads take consecutive channel quads, so each load and store of a
// wave covers a contiguous channel run.
// Stride 1, dilation 1 and S <= DWN_SMAX (the common depthwise layers): DWN_PX1 pixels per thread,
// and per filter row the DWN_PX1 + S - 1 input columns they share are loaded once and reused
// for every tap of the row.
constexpr int DWN_PX = 4;
constexpr int DWN_PX1 = 8;
constexpr int DWN_SMAX = 7;

// CH = 4 or 8 adjacent channels as CH/4 fp32 quads: fp32 16 bytes (CH = 4), bf16 8 or 16 bytes.
template <typename T, int CH>
__device__ __forceinline__ void dwn_load(__amdgpu_buffer_rsrc_t r, bool ok, int64_t e, f32x4 (&v)[CH / 4]) {
    if constexpr (sizeof(T) == 4) {
        static_assert(CH == 4, "fp32 takes 4 channels per load");
        v[0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? (uint32_t)(e * 4) : OOB_OFF,
                                                                               0, 0));
    } else if constexpr (CH == 4) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 h = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, ok ? (uint32_t)(e * 2) : OOB_OFF, 0, 0));
        v[0] = f32x4{__builtin_bit_cast(float, h[0] << 16), __builtin_bit_cast(float, h[0] & 0xFFFF0000u),
                     __builtin_bit_cast(float, h[1] << 16), __builtin_bit_cast(float, h[1] & 0xFFFF0000u)};
    } else {
        const u32x4_t h = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? (uint32_t)(e * 2) : OOB_OFF, 0, 0));
#pragma unroll
        for (int u = 0; u < 2; ++u)
            v[u] = f32x4{__builtin_bit_cast(float, h[2 * u] << 16), __builtin_bit_cast(float, h[2 * u] & 0xFFFF0000u),
                         __builtin_bit_cast(float, h[2 * u + 1] << 16),
                         __builtin_bit_cast(float, h[2 * u + 1] & 0xFFFF0000u)};
    }
}

// Workgroups go to the 8 XCDs round-robin and each XCD has its own L2: block b computes the
// work item range of logical block dwn_remap(b), so that each XCD takes one contiguous eighth of
// the output rows and the input rows that neighbouring output rows share stay in one L2
// (without it each input row was fetched from HBM by up to three XCDs).
__device__ __forceinline__ int64_t dwn_remap(int64_t bid, int64_t nb) {
    const int64_t per = nb >> 3, rem = nb & 7;
    const int64_t xcd = bid & 7, slot = bid >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Output pixels per thread: DWN_PX, or at stride 1 DWN_PX1 (4 with 8 channels, which hold
// twice the registers per pixel).
template <bool S1, int CH>
constexpr int dwn_px() { return S1 ? (CH == 8 ? 4 : DWN_PX1) : DWN_PX; }

template <typename TX, typename TY, bool S1, int CH>
__global__ __launch_bounds__(256) void dw_nhwc_kernel(DirectArgs A, const TX* __restrict__ wt, int64_t total) {
    constexpr int PX = dwn_px<S1, CH>();
    constexpr int NQ = CH / 4;
    const int64_t idx = dwn_remap(blockIdx.x, gridDim.x) * 256 + threadIdx.x;
    if (idx >= total) return;
    const int cq = A.C / CH;
    const int wgroups = (A.Wo + PX - 1) / PX;
    const int q = (int)(idx % cq);
    int64_t t = idx / cq;
    const int wg = (int)(t % wgroups);
    t /= wgroups;
    const int ho = (int)(t % A.Ho);
    const int n = (int)(t / A.Ho);
    const int c0 = CH * q;
    const int wo0 = wg * PX;
    f32x4 acc[PX][NQ];
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
        const int c = c0 + 4 * u;
        const f32x4 b = A.bias ? f32x4{A.bias[c], A.bias[c + 1], A.bias[c + 2], A.bias[c + 3]} : f32x4{0, 0, 0, 0};
#pragma unroll
        for (int p = 0; p < PX; ++p) acc[p][u] = b;
    }
    const __amdgpu_buffer_rsrc_t rx = dk_rsrc(A.x, A.x_bytes);
    const __amdgpu_buffer_rsrc_t rw = dk_rsrc(wt, (uint32_t)(A.R * A.S * A.C * (int)sizeof(TX)));
    for (int r = 0; r < A.R; ++r) {
        const int hi = ho * A.sh - A.ph + r * A.dh;
        const bool hok = (unsigned)hi < (unsigned)A.H;
        const int64_t rowbase = ((int64_t)n * A.H + hi) * A.W;
        if constexpr (S1) {
            // columns wo0 - pw + j, j < PX + S - 1
            f32x4 xc[PX + DWN_SMAX - 1][NQ];
#pragma unroll
            for (int j = 0; j < PX + DWN_SMAX - 1; ++j) {
                const int wi = wo0 - A.pw + j;
                const bool ok = hok & (j < PX + A.S - 1) & ((unsigned)wi < (unsigned)A.W);
                dwn_load<TX, CH>(rx, ok, (rowbase + wi) * A.C + c0, xc[j]);
            }
#pragma unroll
            for (int s = 0; s < DWN_SMAX; ++s) {
                if (s < A.S) {
                    f32x4 wv[NQ];
                    dwn_load<TX, CH>(rw, true, (int64_t)(r * A.S + s) * A.C + c0, wv);
#pragma unroll
                    for (int p = 0; p < PX; ++p)
#pragma unroll
                        for (int u = 0; u < NQ; ++u)
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                acc[p][u][j] = __builtin_fmaf(xc[p + s][u][j], wv[u][j], acc[p][u][j]);
                }
            }
        } else {
            for (int s = 0; s < A.S; ++s) {
                f32x4 wv[NQ];
                dwn_load<TX, CH>(rw, true, (int64_t)(r * A.S + s) * A.C + c0, wv);
#pragma unroll
                for (int p = 0; p < PX; ++p) {
                    const int wi = (wo0 + p) * A.sw - A.pw + s * A.dw;
                    const bool ok = hok & ((unsigned)wi < (unsigned)A.W);
                    f32x4 xv[NQ];
                    dwn_load<TX, CH>(rx, ok, (rowbase + wi) * A.C + c0, xv);
#pragma unroll
                    for (int u = 0; u < NQ; ++u)
#pragma unroll
                        for (int j = 0; j < 4; ++j) acc[p][u][j] = __builtin_fmaf(xv[u][j], wv[u][j], acc[p][u][j]);
                }
            }
        }
    }
    const int64_t ybase = (((int64_t)n * A.Ho + ho) * A.Wo + wo0) * A.K + c0;
#pragma unroll
    for (int p = 0; p < PX; ++p) {
        if (wo0 + p >= A.Wo) break;
        const int64_t e = ybase + (int64_t)p * A.K;
#pragma unroll
        for (int u = 0; u < NQ; ++u) {
            if constexpr (sizeof(TY) == 4) {
                *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(A.y) + e + 4 * u) = acc[p][u];
            } else {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                const u32x2 h = {
                    (uint32_t)dk_f32_to_bf16(acc[p][u][0]) | ((uint32_t)dk_f32_to_bf16(acc[p][u][1]) << 16),
                    (uint32_t)dk_f32_to_bf16(acc[p][u][2]) | ((uint32_t)dk_f32_to_bf16(acc[p][u][3]) << 16)};
                *reinterpret_cast<u32x2*>(reinterpret_cast<uint16_t*>(A.y) + e + 4 * u) = h;
            }
        }
    }
}

bool dw_nhwc_supported(const DirectArgs& a) {
    return a.Cg == 1 && a.Kg == 1 && a.C == a.K && a.C % 4 == 0 && a.N > 0 && a.Ho > 0 && a.Wo > 0;
}

template <bool S1, int CH>
static void launch_dw_nhwc_cfg(const DirectArgs& a, const void* wt, int xdt, int ydt, hipStream_t stream) {
    constexpr int PX = dwn_px<S1, CH>();
    const int64_t total = (int64_t)a.N * a.Ho * ((a.Wo + PX - 1) / PX) * (a.C / CH);
    dim3 grid((unsigned)((total + 255) / 256));
    if constexpr (CH == 4) {
        if (xdt == CONV2D_F32) {
            hipLaunchKernelGGL((dw_nhwc_kernel<float, float, S1, 4>), grid, dim3(256), 0, stream, a,
                               (const float*)wt, total);
            return;
        }
    }
    if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((dw_nhwc_kernel<uint16_t, uint16_t, S1, CH>), grid, dim3(256), 0, stream, a,
                           (const uint16_t*)wt, total);
    else
        hipLaunchKernelGGL((dw_nhwc_kernel<uint16_t, float, S1, CH>), grid, dim3(256), 0, stream, a,
                           (const uint16_t*)wt, total);
}

hipError_t launch_dw_nhwc(const DirectArgs& a, const void* wt, int xdt, int ydt, hipStream_t stream) {
    if (!dw_nhwc_supported(a)) return hipErrorInvalidValue;
    // upper bound of the work items of every configuration (4 channels, 4 pixels per thread)
    if ((int64_t)a.N * a.Ho * ((a.Wo + DWN_PX - 1) / DWN_PX) * (a.C / 4) > 0x7fffff00LL * 256)
        return hipErrorInvalidConfiguration;
    const bool s1 = a.sw == 1 && a.dw == 1 && a.S <= DWN_SMAX;
    // bf16 with C a multiple of 8: 8 channels per thread, 16-byte loads
    const bool ch8 = xdt == CONV2D_BF16 && a.C % 8 == 0;
    if (s1 && ch8) launch_dw_nhwc_cfg<true, 8>(a, wt, xdt, ydt, stream);
    else if (s1) launch_dw_nhwc_cfg<true, 4>(a, wt, xdt, ydt, stream);
    else if (ch8) launch_dw_nhwc_cfg<false, 8>(a, wt, xdt, ydt, stream);
    else launch_dw_nhwc_cfg<false, 4>(a, wt, xdt, ydt, stream);
    return hipGetLastError();
}

hipError_t launch_direct(const DirectArgs& a, int xdt, int ydt, hipStream_t stream) {
    // CONV2D_DW_GENERIC (tests): the generic per-plane kernel for every shape
    if (!std::getenv("CONV2D_DW_GENERIC")) {
        bool launched = false;
        hipError_t e = try_launch_dw_rows(a, xdt, ydt, stream, &launched);
        if (launched || e != hipSuccess) return e;
        e = try_launch_dw(a, xdt, ydt, stream, &launched);
        if (launched || e != hipSuccess) return e;
        e = try_launch_grouped_strip(a, xdt, ydt, stream, &launched);
        if (launched || e != hipSuccess) return e;
        e = try_launch_grouped(a, xdt, ydt, stream, &launched);
        if (launched || e != hipSuccess) return e;
    }
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
