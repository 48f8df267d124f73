// gemm_mfma.hip -- MFMA GEMM of the conv2d library for gfx950.
//
// One kernel body serves both algorithm families the paper compares:
//  * implicit ("sliced") convolution: the B operand is gathered straight from
//    the NCHW input into LDS, one im2col slice (BK reduction rows x BN output
//    pixels) at a time, with stride, zero padding and dilation resolved in the
//    loader; the epilogue adds the bias and writes y in NCHW.  Packing and
//    unpacking are fused into the microkernel (Sec. I: direct methods dilute
//    the packing into the convolution time).
//  * explicit im2col + GEMM: the B operand is the packed column matrix and the
//    result goes to a dense fp32 matrix that a separate unpack kernel turns
//    into y (the Im2col-GEMM baseline of Sec. III-C).
//
// C[m][p] = sum_kr A[m][kr] * B[kr][p], A = weights of one group (row-major,
// kr = (c, r, s) in the natural K x C/g x R x S order), per group gi = blockIdx.z.
//
// Every global access goes through a raw buffer resource: loads outside the
// buffer return zero and stores outside it are dropped, and masked elements
// use an offset beyond any valid record.
#include "conv2d_internal.h"

namespace cv {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define OOB_OFF 0x80000000u
#define RSRC_WORD3 0x00020000

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, RSRC_WORD3);
}

__device__ __forceinline__ float ld_f32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ uint16_t ld_u16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ void st_f32(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, 0);
}
__device__ __forceinline__ void st_u16(__amdgpu_buffer_rsrc_t r, uint32_t off, uint16_t v) {
    __builtin_amdgcn_raw_buffer_store_b16(v, r, off, 0, 0);
}

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename TOut>
__device__ __forceinline__ void store_out(__amdgpu_buffer_rsrc_t r, uint32_t elem_off_valid, bool ok,
                                          float v);
template <>
__device__ __forceinline__ void store_out<float>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok, float v) {
    st_f32(r, ok ? e * 4u : OOB_OFF, v);
}
template <>
__device__ __forceinline__ void store_out<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t e, bool ok,
                                                    float v) {
    st_u16(r, ok ? e * 2u : OOB_OFF, f32_to_bf16_rne(v));
}

// Linear block id -> tile id such that consecutive tile ids land on the same
// XCD (workgroups are handed to the 8 XCDs round-robin), so the M tiles of one
// pixel tile and neighbouring pixel tiles share an L2.
__device__ __forceinline__ int xcd_remap(int bid, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = bid & 7, slot = bid >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Per-column state of the implicit gather: window origin and base offset.
struct ColState {
    int64_t base;  // element offset of x[n, gi*Cg, hi0, wi0] (may be "negative" in padding)
    int32_t hi0, wi0;
};

__device__ __forceinline__ ColState col_state(const GemmArgs& A, int p, int gi) {
    ColState s;
    if (p < A.P) {
        const int n = p / A.HoWo;
        const int hw = p - n * A.HoWo;
        const int ho = hw / A.Wo;
        const int wo = hw - ho * A.Wo;
        s.hi0 = ho * A.sh - A.ph;
        s.wi0 = wo * A.sw - A.pw;
        s.base = (int64_t)n * A.x_nstride + (int64_t)gi * A.b_gstride + (int64_t)s.hi0 * A.W + s.wi0;
    } else {
        s.hi0 = KTAB_DEAD;
        s.wi0 = 0;
        s.base = 0;
    }
    return s;
}

// Byte offset of B[kr][col] for the implicit gather (or OOB_OFF for a zero tap).
template <int ESIZE>
__device__ __forceinline__ uint32_t implicit_off(const GemmArgs& A, const ColState& cs, const KTabEntry& e) {
    const int hi = cs.hi0 + e.roff;
    const int wi = cs.wi0 + e.soff;
    const bool ok = ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
    return ok ? (uint32_t)((cs.base + e.coff) * ESIZE) : OOB_OFF;
}

// Scalar (wave-uniform) read of one table entry.
__device__ __forceinline__ KTabEntry ktab_at(const KTabEntry* t, int kr) {
    kr = __builtin_amdgcn_readfirstlane(kr);
    return t[kr];
}

// ============================================================================ fp32
// Block: 256 threads = 4 waves arranged WM x WN over a BM x BN tile; each wave
// owns (BM/WM) x (BN/WN) = TM x TN MFMA 32x32x2 tiles.  BK = 16 reduction rows
// per stage, double-buffered in LDS (k-major, so one MFMA operand read is 32
// consecutive floats per half-wave).
template <int BM, int BN, int WM, int WN, int BSRC, int EPI, typename TOut>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs A) {
    constexpr int BK = 16;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "bad wave layout");
    constexpr int BNT = BN < 256 ? BN : 256;  // threads along pixels in the B loader
    constexpr int BKT = 256 / BNT;            // threads along k
    constexpr int BCOLS = BN / BNT;           // pixel columns per thread
    constexpr int BROWS = BK / BKT;           // k rows per thread
    constexpr int AROWS = BM * BK / 256;      // A elements per thread
    static_assert(BNT >= 64, "B loader needs wave-uniform k rows");

    __shared__ float As[2][BK][BM + 1];
    __shared__ float Bs[2][BK][BN];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int gi = blockIdx.z;

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int tile_p = tile / A.grid_m;
    const int tile_m = tile - tile_p * A.grid_m;
    const int p0 = tile_p * BN;
    const int m0 = tile_m * BM;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A.a, A.a_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(A.b, A.b_bytes);

    // ---- B loader state
    const int tn = t % BNT;
    const int tk = __builtin_amdgcn_readfirstlane(t / BNT);
    ColState cs[BCOLS];
    int pcol[BCOLS];
#pragma unroll
    for (int j = 0; j < BCOLS; ++j) {
        pcol[j] = p0 + tn + j * BNT;
        if (BSRC == BSRC_IMPLICIT_NCHW) cs[j] = col_state(A, pcol[j], gi);
    }
    // ---- A loader state: element (m = am + i*(256/BK), k = ak)
    const int ak = t % BK;
    const int am = t / BK;
    const int64_t a_base = (int64_t)gi * A.a_gstride;

    float breg[BROWS][BCOLS];
    float areg[AROWS];

    auto load_stage = [&](int stage) {
        const int k0 = stage * BK;
#pragma unroll
        for (int i = 0; i < BROWS; ++i) {
            const int kr = k0 + tk + i * BKT;
            if (BSRC == BSRC_IMPLICIT_NCHW) {
                const KTabEntry e = ktab_at(A.ktab, kr);
#pragma unroll
                for (int j = 0; j < BCOLS; ++j) breg[i][j] = ld_f32(rb, implicit_off<4>(A, cs[j], e));
            } else {
#pragma unroll
                for (int j = 0; j < BCOLS; ++j) {
                    const bool ok = (kr < A.Kred) & (pcol[j] < A.P);
                    const int64_t e = (int64_t)gi * A.b_gstride + (int64_t)kr * A.ldb + pcol[j];
                    breg[i][j] = ld_f32(rb, ok ? (uint32_t)(e * 4) : OOB_OFF);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < AROWS; ++i) {
            const int m = m0 + am + i * (256 / BK);
            const int kr = k0 + ak;
            const bool ok = (m < A.M) & (kr < A.Kred);
            const int64_t e = a_base + (int64_t)m * A.lda + kr;
            areg[i] = ld_f32(ra, ok ? (uint32_t)(e * 4) : OOB_OFF);
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int i = 0; i < BROWS; ++i)
#pragma unroll
            for (int j = 0; j < BCOLS; ++j) Bs[buf][tk + i * BKT][tn + j * BNT] = breg[i][j];
#pragma unroll
        for (int i = 0; i < AROWS; ++i) As[buf][ak][am + i * (256 / BK)] = areg[i];
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int wm0 = (wave % WM) * WTM;
    const int wn0 = (wave / WM) * WTN;
    const int lrow = lane >> 5;  // which of the two k rows this half-wave feeds
    const int lcol = lane & 31;

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int st = 0; st < A.nstages; ++st) {
        const int buf = st & 1;
        const bool more = st + 1 < A.nstages;
        if (more) load_stage(st + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 2; ++ks) {
            float a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[buf][2 * ks + lrow][wm0 + i * 32 + lcol];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[buf][2 * ks + lrow][wn0 + j * 32 + lcol];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (more) store_stage(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue.  Accumulator v of lane l holds row 8*(v/4) + 4*(l/32) + v%4, column l%32.
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int p = p0 + wn0 + j * 32 + lcol;
        const bool pok = p < A.P;
        int64_t ybase;
        if (EPI == EPI_NCHW) {
            const int n = p / A.HoWo;
            const int hw = p - n * A.HoWo;
            ybase = (int64_t)n * A.y_nstride + (int64_t)gi * A.M * A.HoWo + hw;
        } else {
            ybase = (int64_t)gi * A.c_gstride + p;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm0 + i * 32 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                const bool ok = pok & (m < A.M);
                float val = acc[i][j][v];
                if (EPI == EPI_NCHW) {
                    if (A.bias != nullptr && ok) val += A.bias[gi * A.M + m];
                    store_out<TOut>(ry, (uint32_t)(ybase + (int64_t)m * A.HoWo), ok, val);
                } else {
                    store_out<float>(ry, (uint32_t)(ybase + (int64_t)m * A.ldc), ok, val);
                }
            }
        }
    }
}

// ============================================================================ bf16
// Same structure with MFMA 32x32x16 bf16 (fp32 accumulation).  LDS tiles are
// m-major / n-major with 8 consecutive k per 16-byte chunk, which is exactly
// one lane's MFMA operand; rows are padded by 8 elements.
template <int BM, int BN, int WM, int WN, int BSRC, int EPI, typename TOut>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs A) {
    constexpr int BK = 32;
    constexpr int LDK = BK + 8;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "bad wave layout");
    static_assert(BN <= 256 && 256 % BN == 0 && BN >= 64, "B loader assumes one column per thread");
    constexpr int BUNITS = BN * (BK / 8) / 256;  // 8-element B chunks per thread
    constexpr int AUNITS = BM * (BK / 8) / 256;  // 8-element A chunks per thread

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][LDK];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int gi = blockIdx.z;

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int tile_p = tile / A.grid_m;
    const int tile_m = tile - tile_p * A.grid_m;
    const int p0 = tile_p * BN;
    const int m0 = tile_m * BM;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A.a, A.a_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(A.b, A.b_bytes);

    // B: unit u = t + i*256 -> column n = u % BN (same for all i), k chunk kc = u / BN
    const int bn = t % BN;
    const int bkc0 = __builtin_amdgcn_readfirstlane(t / BN);
    const int pcol = p0 + bn;
    ColState cs;
    if (BSRC == BSRC_IMPLICIT_NCHW) cs = col_state(A, pcol, gi);
    // A: unit u = t + i*256 -> row m = u / 4, k chunk kc = u % 4
    const int64_t a_base = (int64_t)gi * A.a_gstride;

    u32x4 breg[BUNITS];
    u32x4 areg[AUNITS];

    auto load_stage = [&](int stage) {
        const int k0 = stage * BK;
#pragma unroll
        for (int i = 0; i < BUNITS; ++i) {
            const int kc = bkc0 + i * (256 / BN);
            uint16_t h[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int kr = k0 + kc * 8 + q;
                uint32_t off;
                if (BSRC == BSRC_IMPLICIT_NCHW) {
                    off = implicit_off<2>(A, cs, ktab_at(A.ktab, kr));
                } else {
                    const bool ok = (kr < A.Kred) & (pcol < A.P);
                    const int64_t e = (int64_t)gi * A.b_gstride + (int64_t)kr * A.ldb + pcol;
                    off = ok ? (uint32_t)(e * 2) : OOB_OFF;
                }
                h[q] = ld_u16(rb, off);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) breg[i][q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
        }
#pragma unroll
        for (int i = 0; i < AUNITS; ++i) {
            const int u = t + i * 256;
            const int m = m0 + u / (BK / 8);
            const int kc = u % (BK / 8);
            uint16_t h[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int kr = k0 + kc * 8 + q;
                const bool ok = (m < A.M) & (kr < A.Kred);
                const int64_t e = a_base + (int64_t)m * A.lda + kr;
                h[q] = ld_u16(ra, ok ? (uint32_t)(e * 2) : OOB_OFF);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) areg[i][q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int i = 0; i < BUNITS; ++i) {
            const int kc = bkc0 + i * (256 / BN);
            *reinterpret_cast<u32x4*>(&Bs[buf][bn][kc * 8]) = breg[i];
        }
#pragma unroll
        for (int i = 0; i < AUNITS; ++i) {
            const int u = t + i * 256;
            *reinterpret_cast<u32x4*>(&As[buf][u / (BK / 8)][(u % (BK / 8)) * 8]) = areg[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int wm0 = (wave % WM) * WTM;
    const int wn0 = (wave / WM) * WTN;
    const int lrow = lane >> 5;
    const int lcol = lane & 31;

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int st = 0; st < A.nstages; ++st) {
        const int buf = st & 1;
        const bool more = st + 1 < A.nstages;
        if (more) load_stage(st + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[i] = *reinterpret_cast<const bf16x8*>(&As[buf][wm0 + i * 32 + lcol][ks * 16 + 8 * lrow]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][wn0 + j * 32 + lcol][ks * 16 + 8 * lrow]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (more) store_stage(buf ^ 1);
        __syncthreads();
    }

    const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int p = p0 + wn0 + j * 32 + lcol;
        const bool pok = p < A.P;
        int64_t ybase;
        if (EPI == EPI_NCHW) {
            const int n = p / A.HoWo;
            const int hw = p - n * A.HoWo;
            ybase = (int64_t)n * A.y_nstride + (int64_t)gi * A.M * A.HoWo + hw;
        } else {
            ybase = (int64_t)gi * A.c_gstride + p;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm0 + i * 32 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                const bool ok = pok & (m < A.M);
                float val = acc[i][j][v];
                if (EPI == EPI_NCHW) {
                    if (A.bias != nullptr && ok) val += A.bias[gi * A.M + m];
                    store_out<TOut>(ry, (uint32_t)(ybase + (int64_t)m * A.HoWo), ok, val);
                } else {
                    store_out<float>(ry, (uint32_t)(ybase + (int64_t)m * A.ldc), ok, val);
                }
            }
        }
    }
}

// ============================================================================ dispatch
template <int BM, int BN, int WM, int WN>
static hipError_t launch_tile(const GemmArgs& a, int bsrc, int epi, int xdt, int ydt, int groups,
                              hipStream_t stream) {
    dim3 grid((unsigned)(a.grid_p * a.grid_m), 1, (unsigned)groups);
    dim3 block(256);
#define CV_LAUNCH(KER, BS, EP, TO) hipLaunchKernelGGL((KER<BM, BN, WM, WN, BS, EP, TO>), grid, block, 0, stream, a)
    if (xdt == CONV2D_F32) {
        if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_NCHW) CV_LAUNCH(gemm_f32_kernel, BSRC_IMPLICIT_NCHW, EPI_NCHW, float);
        else if (bsrc == BSRC_DENSE && epi == EPI_DENSE) CV_LAUNCH(gemm_f32_kernel, BSRC_DENSE, EPI_DENSE, float);
        else return hipErrorInvalidValue;
    } else {
        if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_NCHW) {
            if (ydt == CONV2D_BF16) CV_LAUNCH(gemm_bf16_kernel, BSRC_IMPLICIT_NCHW, EPI_NCHW, uint16_t);
            else CV_LAUNCH(gemm_bf16_kernel, BSRC_IMPLICIT_NCHW, EPI_NCHW, float);
        } else if (bsrc == BSRC_DENSE && epi == EPI_DENSE) {
            CV_LAUNCH(gemm_bf16_kernel, BSRC_DENSE, EPI_DENSE, float);
        } else {
            return hipErrorInvalidValue;
        }
    }
#undef CV_LAUNCH
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, int tile, int bsrc, int epi, int xdt, int ydt, int groups,
                       hipStream_t stream) {
    switch (tile) {
        case TILE_64x64: return launch_tile<64, 64, 2, 2>(a, bsrc, epi, xdt, ydt, groups, stream);
        case TILE_64x128: return launch_tile<64, 128, 1, 4>(a, bsrc, epi, xdt, ydt, groups, stream);
        case TILE_64x256: return launch_tile<64, 256, 1, 4>(a, bsrc, epi, xdt, ydt, groups, stream);
        case TILE_128x128: return launch_tile<128, 128, 2, 2>(a, bsrc, epi, xdt, ydt, groups, stream);
        case TILE_128x64: return launch_tile<128, 64, 2, 2>(a, bsrc, epi, xdt, ydt, groups, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace cv
