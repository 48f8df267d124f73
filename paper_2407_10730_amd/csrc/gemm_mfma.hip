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
#include "device_common.h"

namespace cv {

// Epilogue of both kernels.  Accumulator v of lane l holds row 8*(v/4) + 4*(l/32) + v%4,
// column l%32 of its 32x32 tile.  All bias values of the rows a lane writes are loaded
// before its first store, so the stores leave back to back behind one wait (a load
// between two stores would make each store wait for the previous one).  NHWC y: element
// (p, channel gi*M + m) sits at p*ldc + gi*M + m (ldc = K), so the four consecutive rows a
// lane holds per v/4 are adjacent and go out as one 16-byte (fp32) or 8-byte (bf16) store
// when M is a multiple of 4.
template <int TM, int TN, int EPI, typename TOut>
__device__ __forceinline__ void store_tile(const GemmArgs& A, f32x16 (&acc)[TM][TN], int gi, int sp, int mb, int pb,
                                           int lrow, int lcol) {
    if (EPI != EPI_DENSE && A.bias != nullptr) {
        const __amdgpu_buffer_rsrc_t rbias = make_rsrc(A.bias, (uint32_t)(gridDim.z * A.M * 4));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = mb + i * 32 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                const float bv = ld_f32(rbias, m < A.M ? (uint32_t)((gi * A.M + m) * 4) : OOB_OFF);
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j][v] += bv;
            }
    }
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
    if (EPI == EPI_NHWC && A.M % 4 == 0) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int p = pb + j * 32 + lcol;
            const int64_t ybase = (int64_t)p * A.ldc + (int64_t)gi * A.M;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const int m = mb + i * 32 + 8 * v4 + 4 * lrow;
                    const bool ok = (p < A.P) & (m < A.M);
                    const float q[4] = {acc[i][j][4 * v4], acc[i][j][4 * v4 + 1], acc[i][j][4 * v4 + 2],
                                        acc[i][j][4 * v4 + 3]};
                    if constexpr (sizeof(TOut) == 4) {
                        const uint32_t off = ok ? (uint32_t)(ybase + m) * 4u : OOB_OFF;
                        __builtin_amdgcn_raw_buffer_store_b128(
                            u32x4{__builtin_bit_cast(uint32_t, q[0]), __builtin_bit_cast(uint32_t, q[1]),
                                  __builtin_bit_cast(uint32_t, q[2]), __builtin_bit_cast(uint32_t, q[3])},
                            ry, off, 0, 0);
                    } else {
                        const uint32_t off = ok ? (uint32_t)(ybase + m) * 2u : OOB_OFF;
                        __builtin_amdgcn_raw_buffer_store_b64(
                            u32x2{(uint32_t)f32_to_bf16_rne(q[0]) | ((uint32_t)f32_to_bf16_rne(q[1]) << 16),
                                  (uint32_t)f32_to_bf16_rne(q[2]) | ((uint32_t)f32_to_bf16_rne(q[3]) << 16)},
                            ry, off, 0, 0);
                    }
                }
        }
        return;
    }
    if constexpr (EPI == EPI_NCHW && sizeof(TOut) == 2) {
        if (mb + TM * 32 <= A.M) {
            // bf16 NCHW, the wave's rows all inside M: one byte base per lane and column tile,
            // the row offsets wave-uniform (the store's scalar offset), and one packed
            // conversion for each two rows of a lane (the rows of v and v + 1, v even)
            const int rs = A.HoWo * 2;  // bytes between output rows
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int p = pb + j * 32 + lcol;
                uint32_t lb = OOB_OFF;
                if (p < A.P) {
                    const int n_img = p / A.HoWo;
                    const int hw = p - n_img * A.HoWo;
                    lb = (uint32_t)((int64_t)n_img * A.y_nstride + ((int64_t)gi * A.M + mb + 4 * lrow) * A.HoWo + hw) * 2u;
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int v = 0; v < 16; v += 2) {
                        const uint32_t w = __builtin_bit_cast(
                            uint32_t, __builtin_convertvector(f32x2{acc[i][j][v], acc[i][j][v + 1]}, bf16x2));
                        const int r0 = i * 32 + 8 * (v >> 2) + (v & 3);
                        __builtin_amdgcn_raw_buffer_store_b16((uint16_t)w, ry, lb, r0 * rs, 0);
                        __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(w >> 16), ry, lb, (r0 + 1) * rs, 0);
                    }
            }
            return;
        }
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int p = pb + j * 32 + lcol;
        const bool pok = p < A.P;
        int64_t ybase;
        if (EPI == EPI_NCHW) {
            const int n_img = p / A.HoWo;
            const int hw = p - n_img * A.HoWo;
            ybase = (int64_t)n_img * A.y_nstride + (int64_t)gi * A.M * A.HoWo + hw;
        } else if (EPI == EPI_NHWC) {
            ybase = (int64_t)p * A.ldc + (int64_t)gi * A.M;
        } else {
            ybase = (int64_t)sp * A.c_sstride + (int64_t)gi * A.c_gstride + p;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = mb + i * 32 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                const bool ok = pok & (m < A.M);
                if (EPI == EPI_NCHW)
                    store_out<TOut>(ry, (uint32_t)(ybase + (int64_t)m * A.HoWo), ok, acc[i][j][v]);
                else if (EPI == EPI_NHWC)
                    store_out<TOut>(ry, (uint32_t)(ybase + m), ok, acc[i][j][v]);
                else
                    store_out<float>(ry, (uint32_t)(ybase + (int64_t)m * A.ldc), ok, acc[i][j][v]);
            }
    }
}

// Work of one block: its output tile and its stages [s_begin, s_end).  The blocks past
// the whole tiles of the grid are the pieces of the tail split (tail_tile >= 0).
struct BlockWork {
    int tile, s_begin, s_end, tail_tile, piece;
};

__device__ __forceinline__ BlockWork block_work(const GemmArgs& A, int ksplit, int sp) {
    BlockWork w;
    const int ndp = (int)gridDim.x - A.tail_tiles * A.tail_pieces;
    const int q = (int)blockIdx.x - ndp;
    if (q < 0) {
        w.tile = xcd_remap(blockIdx.x, ndp);
        w.s_begin = ksplit > 1 ? sp * A.split_stages : 0;
        w.s_end = ksplit > 1 ? min(w.s_begin + A.split_stages, A.nstages) : A.nstages;
        w.tail_tile = -1;
        w.piece = 0;
    } else {
        w.tail_tile = q / A.tail_pieces;
        w.piece = q - w.tail_tile * A.tail_pieces;
        w.tile = ndp + w.tail_tile;
        w.s_begin = w.piece * A.tail_stages;
        w.s_end = min(w.s_begin + A.tail_stages, A.nstages);
    }
    return w;
}

// Tail split: store this piece's partial tile, count its arrival, and in the piece that
// arrives last replace acc by the sum of all pieces of the tile in piece order (the same
// result whatever the arrival order).  Returns false in the other pieces, which are done.
// The pieces of a tile may run on different XCDs, whose L2 caches are not coherent with
// each other.  The partials are therefore stored and loaded with the device-scope cache
// policy (sc1: written through to, and read from, the point where all XCDs agree), and each
// piece waits for its stores to complete before it counts itself; no fence is used, since
// a device-scope fence writes back and invalidates the whole L2 of the XCD and costs every
// other block on it its cached input.  The counter is an atomic, coherent device-wide.
// Partial layout: 16-byte unit ((i*TN + j)*4 + q)*256 + t of the piece's BM x BN tile, through
// buffer operations with a wave-uniform base (no per-lane address kept alive).
template <int TM, int TN>
__device__ __forceinline__ bool tail_reduce(const GemmArgs& A, f32x16 (&acc)[TM][TN], const BlockWork& w,
                                            int t) {
    constexpr uint32_t PIECE = TM * TN * 4 * 256 * 16;  // bytes of one partial tile
    constexpr int SC1 = 1 << 4;                         // buffer cache policy bit: device scope
    __shared__ int s_last;
    const __amdgpu_buffer_rsrc_t rp =
        make_rsrc(A.tail_part, (uint32_t)A.tail_tiles * (uint32_t)A.tail_pieces * PIECE);
    const uint32_t tile_base = (uint32_t)w.tail_tile * (uint32_t)A.tail_pieces * PIECE;
    const uint32_t lane_off = (uint32_t)t * 16u;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f32x4 v{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                __builtin_amdgcn_raw_buffer_store_b128(
                    __builtin_bit_cast(u32x4, v), rp, lane_off,
                    (int)(tile_base + (uint32_t)w.piece * PIECE + (uint32_t)((i * TN + j) * 4 + q) * 4096u), SC1);
            }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the partial is complete device-wide
    __syncthreads();
    if (t == 0)
        s_last = __hip_atomic_fetch_add(A.tail_count + w.tail_tile, 1u, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(A.tail_pieces - 1);
    __syncthreads();
    if (!s_last) return false;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
#pragma unroll 1
    for (int pc = 0; pc < A.tail_pieces; ++pc) {
        const uint32_t base = tile_base + (uint32_t)pc * PIECE;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x4 v = __builtin_bit_cast(
                        f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                   rp, lane_off, (int)(base + (uint32_t)((i * TN + j) * 4 + q) * 4096u), SC1));
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
                }
    }
    // ready for the next launch
    if (t == 0) __hip_atomic_store(A.tail_count + w.tail_tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

// ============================================================================ fp32
// Block: 256 threads = 4 waves arranged WM x WN over a BM x BN tile; each wave
// owns (BM/WM) x (BN/WN) = TM x TN MFMA 32x32x2 tiles.  BK reduction rows per
// stage, double-buffered in LDS.  Both operands sit in LDS row-per-output
// ([m][k] and [p][k]) with the BK values of a row contiguous: the MFMA of step
// ks takes reduction index ks from lanes 0-31 and ks + BK/2 from lanes 32-63,
// so a lane reads its BK/2 operand values of a stage with 16-byte LDS loads,
// and a loader thread that holds 4 consecutive reduction rows of one output
// writes them with one 16-byte store.  The row pitch is BK + 4 floats.
// PF = 1: the global loads of stage s+1 are issued before the MFMAs of stage s;
// PF = 2: two register sets, the loads of stage s+2 are issued before the
// MFMAs of stage s, so a load has two stages of MFMA work to land.
// 64x64 tiles with 16-row stages fit seven blocks per CU (LDS 20 KiB each); the bound keeps
// the register budget at seven blocks with the tail-split epilogue compiled in.
// Window origin of output pixel p in an NHWC input: element offset of
// x[n, hi0, wi0, gi*Cg] (negative or past the row inside the padding).
__device__ __forceinline__ ColState col_state_nhwc(const GemmArgs& A, int p, int gi) {
    ColState s;
    if (p < A.P) {
        const int n = p / A.HoWo;
        const int hw = p - n * A.HoWo;
        const int ho = hw / A.Wo;
        const int wo = hw - ho * A.Wo;
        s.hi0 = ho * A.sh - A.ph;
        s.wi0 = wo * A.sw - A.pw;
        s.base = (((int64_t)n * A.H + s.hi0) * A.W + s.wi0) * A.Cx + (int64_t)gi * A.Cg;
    } else {
        s.hi0 = KTAB_DEAD;
        s.wi0 = 0;
        s.base = 0;
    }
    return s;
}

template <int BM, int BN, int WM, int WN, int BK, int PF, int BSRC, int EPI, typename TOut>
__global__ __launch_bounds__(256, (BM * BN <= 4096 && BK == 16 ? 7 : 1)) void gemm_f32_kernel(GemmArgs A) {
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "bad wave layout");
    static_assert(PF == 1 || PF == 2, "prefetch distance");
    static_assert(BK == 16 || BK == 32, "stage depth");
    constexpr int LDK = BK + 4;               // LDS row pitch in floats (16-byte aligned rows)
    constexpr int KH = BK / 2;                // reduction values per lane per stage
    constexpr int BNT = BN < 256 ? BN : 256;  // threads along pixels in the B loader
    constexpr int BKT = 256 / BNT;            // threads along k (each owns runs of 4 rows)
    constexpr int BCOLS = BN / BNT;           // pixel columns per thread
    constexpr int BRUNS = BK / (4 * BKT);     // runs of 4 consecutive k rows per thread
    constexpr int AQ = BM * BK / 4;           // runs of 4 consecutive k of one A row per stage
    constexpr int ARUNS = (AQ + 255) / 256;   // ... per thread (the last partly idle when BM = 32)
    static_assert(BNT >= 64, "B loader needs wave-uniform k rows");
    static_assert(BRUNS >= 1 && ARUNS >= 1, "loader layout");

    __shared__ __attribute__((aligned(16))) float As[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) float Bs[2][BN][LDK];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int ksplit = A.ksplit > 1 ? A.ksplit : 1;
    const int gi = blockIdx.z / ksplit;
    const int sp = blockIdx.z - gi * ksplit;
    // this block's tile and stages [s_begin, s_end)
    const BlockWork wk = block_work(A, ksplit, sp);
    const int s_begin = wk.s_begin, s_end = wk.s_end;
    const int tile = wk.tile;
    const int tile_p = tile / A.grid_m;
    const int tile_m = tile - tile_p * A.grid_m;
    const int p0 = tile_p * BN;
    const int m0 = tile_m * BM;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A.a, A.a_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(A.b, A.b_bytes);

    // ---- B loader: thread (tn, tk) loads pixels tn + j*BNT, k rows 4*(g*BKT + tk) + i
    const int tn = t % BNT;
    const int tk = __builtin_amdgcn_readfirstlane(t / BNT);
    ColState cs[BCOLS];
    uint32_t dvb[BCOLS];  // dense: byte offset of column j in row 0 of this group, or OOB
#pragma unroll
    for (int j = 0; j < BCOLS; ++j) {
        const int p = p0 + tn + j * BNT;
        if constexpr (BSRC == BSRC_NHWC_TAP) cs[j] = col_state_nhwc(A, p, gi);
        else if constexpr (BSRC != BSRC_DENSE) cs[j] = col_state(A, p, gi);
        dvb[j] = p < A.P ? (uint32_t)(((int64_t)gi * A.b_gstride + p) * 4) : OOB_OFF;
    }
    // ---- A loader: run g of thread t is row (t + g*256) / (BK/4), k 4*((t + g*256) % (BK/4)) + i
    const int64_t a_base = (int64_t)gi * A.a_gstride;

    f32x4 breg0[BRUNS][BCOLS], breg1[BRUNS][BCOLS];
    f32x4 areg0[ARUNS], areg1[ARUNS];
    // tap-major weights: byte offset of each A run's row and channel quad, computed once (a
    // stage then adds one uniform offset per load instead of 64-bit index arithmetic)
    uint32_t na_off[ARUNS];
#pragma unroll
    for (int g = 0; g < ARUNS; ++g) {
        const int q = t + g * 256;
        const bool qa = AQ % 256 == 0 || q < AQ;
        const int m = m0 + q / (BK / 4);
        na_off[g] = ((m < A.M) & qa) ? (uint32_t)(a_base + (int64_t)m * A.lda + 4 * (q % (BK / 4))) * 4u : OOB_OFF;
    }
    // tap-major cursor of the next stage to load.  Channel blocks outermost, filter
    // taps innermost: the taps of one channel block re-read the same input lines,
    // which then hit in L1.
    int cur_c0 = 0, cur_r = 0, cur_s = 0;
    if constexpr (BSRC == BSRC_IMPLICIT_TAP || BSRC == BSRC_NHWC_TAP) {
        const int tap = s_begin % A.RS;
        cur_c0 = (s_begin / A.RS) * BK;
        cur_r = tap / A.S;
        cur_s = tap - cur_r * A.S;
    }

    auto load_stage = [&](int stage, f32x4 (&breg)[BRUNS][BCOLS], f32x4 (&areg)[ARUNS]) {
        const int k0 = stage * BK;
        if constexpr (BSRC == BSRC_IMPLICIT_TAP || BSRC == BSRC_NHWC_TAP) {
            const int roff = cur_r * A.dh, soff = cur_s * A.dw;
            // NCHW: channels HW apart, 4 single loads per run; NHWC: the run's 4 channels are
            // contiguous, one 16-byte load
            const int tapoff = BSRC == BSRC_NHWC_TAP ? (roff * A.W + soff) * A.Cx + cur_c0 : roff * A.W + soff;
            uint32_t vb[BCOLS];
#pragma unroll
            for (int j = 0; j < BCOLS; ++j) {
                const int hi = cs[j].hi0 + roff, wi = cs[j].wi0 + soff;
                const bool ok = ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
                vb[j] = ok ? (uint32_t)(((int32_t)cs[j].base + tapoff) * 4) : OOB_OFF;
            }
            if constexpr (BSRC == BSRC_NHWC_TAP) {
#pragma unroll
                for (int g = 0; g < BRUNS; ++g)
#pragma unroll
                    for (int j = 0; j < BCOLS; ++j)
                        breg[g][j] = __builtin_bit_cast(
                            f32x4, PF == 1 ? __builtin_amdgcn_raw_buffer_load_b128(rb, vb[j], 4 * (g * BKT + tk) * 4, 0)
                                           : __builtin_amdgcn_raw_buffer_load_b128(
                                                 rb, vb[j] == OOB_OFF ? OOB_OFF : vb[j] + (uint32_t)(4 * (g * BKT + tk)) * 4u,
                                                 0, 0));
            } else {
#pragma unroll
                for (int g = 0; g < BRUNS; ++g)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        // the channel's offset is wave-uniform (tk is).  One set of staging
                        // registers: it goes in the load's scalar offset (a lane out of range
                        // stays out of range, the others address inside x), so the loads share
                        // the lanes' address registers (N32 256->64 56x56 1x1: 3 % faster).  Two
                        // sets: added per lane (the scalar form measured 7 % slower on N32
                        // 64->64 56x56 3x3).
                        const int cofs = (cur_c0 + 4 * (g * BKT + tk) + i) * A.HW * 4;
#pragma unroll
                        for (int j = 0; j < BCOLS; ++j)
                            breg[g][j][i] = PF == 1 ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, vb[j], cofs, 0))
                                                    : ld_f32(rb, vb[j] + (uint32_t)cofs);
                    }
            }
            // weights in tap-major order [K][R*S][C/g]: 4 consecutive channels per 16-byte load
            const int ab = ((cur_r * A.S + cur_s) * A.Cg + cur_c0) * 4;
#pragma unroll
            for (int g = 0; g < ARUNS; ++g) {
                // bit-cast the whole vector: casting its elements one by one made this
                // compiler emit a single-dword load
                areg[g] = __builtin_bit_cast(f32x4, PF == 1 ? __builtin_amdgcn_raw_buffer_load_b128(ra, na_off[g], ab, 0)
                                                            : __builtin_amdgcn_raw_buffer_load_b128(ra, na_off[g] + (uint32_t)ab, 0, 0));
            }
            if (++cur_s == A.S) {
                cur_s = 0;
                if (++cur_r == A.R) {
                    cur_r = 0;
                    cur_c0 += BK;
                }
            }
        } else {
#pragma unroll
            for (int g = 0; g < BRUNS; ++g) {
                const int kb = k0 + 4 * (g * BKT + tk);
                if constexpr (BSRC == BSRC_IMPLICIT_NCHW) {
                    KTabEntry e[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) e[i] = ktab_at(A.ktab, kb + i);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < BCOLS; ++j) breg[g][j][i] = ld_f32(rb, implicit_off<4>(A, cs[j], e[i]));
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int kr = kb + i;
                        const bool kok = kr < A.Kred;
#pragma unroll
                        for (int j = 0; j < BCOLS; ++j)
                            breg[g][j][i] = ld_f32(rb, kok ? dvb[j] + (uint32_t)kr * (uint32_t)A.ldb * 4u : OOB_OFF);
                    }
                }
            }
#pragma unroll
            for (int g = 0; g < ARUNS; ++g) {
                const int q = t + g * 256;
                const bool qa = AQ % 256 == 0 || q < AQ;
                const int m = m0 + q / (BK / 4);
                const int kb = k0 + 4 * (q % (BK / 4));
                const int64_t e = a_base + (int64_t)m * A.lda + kb;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool ok = (m < A.M) & (kb + i < A.Kred) & qa;
                    areg[g][i] = ld_f32(ra, ok ? (uint32_t)((e + i) * 4) : OOB_OFF);
                }
            }
        }
    };
    auto store_stage = [&](int buf, const f32x4 (&breg)[BRUNS][BCOLS], const f32x4 (&areg)[ARUNS]) {
#pragma unroll
        for (int g = 0; g < BRUNS; ++g)
#pragma unroll
            for (int j = 0; j < BCOLS; ++j)
                *reinterpret_cast<f32x4*>(&Bs[buf][tn + j * BNT][4 * (g * BKT + tk)]) = breg[g][j];
#pragma unroll
        for (int g = 0; g < ARUNS; ++g) {
            const int q = t + g * 256;
            if (AQ % 256 == 0 || q < AQ) *reinterpret_cast<f32x4*>(&As[buf][q / (BK / 4)][4 * (q % (BK / 4))]) = areg[g];
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
    const int lrow = lane >> 5;  // 0: first half of the stage's reduction rows, 1: second half
    const int lcol = lane & 31;

    auto compute = [&](int buf) {
        f32x4 a[TM][KH / 4], b[TN][KH / 4];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < KH / 4; ++v)
                a[i][v] = *reinterpret_cast<const f32x4*>(&As[buf][wm0 + i * 32 + lcol][KH * lrow + 4 * v]);
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < KH / 4; ++v)
                b[j][v] = *reinterpret_cast<const f32x4*>(&Bs[buf][wn0 + j * 32 + lcol][KH * lrow + 4 * v]);
#pragma unroll
        for (int ks = 0; ks < KH; ++ks)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][ks / 4][ks % 4], b[j][ks / 4][ks % 4],
                                                                     acc[i][j], 0, 0, 0);
    };

    // stages s_begin + j, j < n; LDS buffer j & 1
    const int n = s_end - s_begin;
    if constexpr (PF == 1) {
        load_stage(s_begin, breg0, areg0);
        store_stage(0, breg0, areg0);
        __syncthreads();
        for (int j = 0; j < n; ++j) {
            const int buf = j & 1;
            const bool more = j + 1 < n;
            if (more) load_stage(s_begin + j + 1, breg0, areg0);
            if (!A.loader_only) compute(buf);
            if (more) store_stage(buf ^ 1, breg0, areg0);
            __syncthreads();
        }
    } else {
        // The loads past the block's last stage are issued too (except through the tap table,
        // which they would read past): they read inside or past the tensors, where the buffer
        // range check returns zero, and are never stored.  With a condition on them, the wait
        // before the LDS stores would have to cover the path without them and so would wait
        // for the loads just issued as well.  (Storing those sets as well, which removes the
        // conditions on the stores, measured 2 % slower on N32 64->64 56x56 3x3.)
        constexpr bool kAlways = BSRC != BSRC_IMPLICIT_NCHW;
        load_stage(s_begin, breg0, areg0);
        if (n > 1) load_stage(s_begin + 1, breg1, areg1);
        store_stage(0, breg0, areg0);
        __syncthreads();
        for (int j = 0; j < n; j += 2) {
            // even stage: set 0 is free, set 1 holds stage j+1
            if (kAlways || j + 2 < n) load_stage(s_begin + j + 2, breg0, areg0);
            if (!A.loader_only) compute(0);
            if (j + 1 < n) store_stage(1, breg1, areg1);
            __syncthreads();
            if (j + 1 >= n) break;
            // odd stage: set 1 is free, set 0 holds stage j+2
            if (kAlways || j + 3 < n) load_stage(s_begin + j + 3, breg1, areg1);
            if (!A.loader_only) compute(1);
            if (j + 2 < n) store_stage(0, breg0, areg0);
            __syncthreads();
        }
    }

    if (A.loader_only) return;
    if constexpr (EPI != EPI_DENSE) {
        if (wk.tail_tile >= 0 && !tail_reduce<TM, TN>(A, acc, wk, t)) return;
    }
    store_tile<TM, TN, EPI, TOut>(A, acc, gi, sp, m0 + wm0, p0 + wn0, lrow, lcol);
}

// ============================================================================ bf16
// Same structure with MFMA 32x32x16 bf16 (fp32 accumulation).  LDS tiles are
// m-major / n-major with 8 consecutive k per 16-byte chunk, which is exactly
// one lane's MFMA operand; rows are padded by 8 elements.  BK = 32 or 64
// reduction rows per stage.
//
// B sources: the NCHW gathers (tap table or tap-major) read one 2-byte element
// per load, 8 loads per 16-byte chunk.  NHWC_TAP reads a channel-contiguous
// copy of x (NHWC): in tap-major order one chunk is 8 consecutive channels of
// one pixel at one tap, a single 16-byte load, and the 4 or 8 chunks of a
// pixel's stage row come from consecutive threads (one 64- or 128-byte run).


template <int BM, int BN, int WM, int WN, int BK, int PF, int BSRC, int EPI, typename TOut>
__global__ __launch_bounds__(256, (BM * BN <= 4096 && BK == 32 ? 7 : 1)) void gemm_bf16_kernel(GemmArgs A) {
    constexpr int LDK = BK + 8;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(BK == 32 || BK == 64, "stage depth");
    static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "bad wave layout");
    static_assert(BN <= 256 && 256 % BN == 0 && BN >= 64, "B loader assumes one column per thread");
    constexpr int CPR = BK / 8;                  // 16-byte chunks per tile row
    constexpr int BUNITS = BN * CPR / 256;       // 8-element B chunks per thread
    constexpr int AQ = BM * CPR;                 // 8-element A chunks per stage
    constexpr int AUNITS = (AQ + 255) / 256;     // ... per thread (the last partly idle when BM = 32)
    constexpr bool NHWC = BSRC == BSRC_NHWC_TAP;
    // B columns whose reduction values are contiguous in memory (NHWC gather, or a dense B^T
    // [P][ldb]): one 16-byte load moves 8 reduction values of one column
    constexpr bool KCONT = NHWC || BSRC == BSRC_DENSE_T;

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][LDK];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int ksplit = A.ksplit > 1 ? A.ksplit : 1;
    const int gi = blockIdx.z / ksplit;
    const int sp = blockIdx.z - gi * ksplit;
    // this block's tile and stages [s_begin, s_end)
    const BlockWork wk = block_work(A, ksplit, sp);
    const int s_begin = wk.s_begin, s_end = wk.s_end;
    const int tile = wk.tile;
    const int tile_p = tile / A.grid_m;
    const int tile_m = tile - tile_p * A.grid_m;
    const int p0 = tile_p * BN;
    const int m0 = tile_m * BM;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A.a, A.a_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(A.b, A.b_bytes);

    // B, NCHW sources: unit u = t + i*256 -> column n = u % BN (same for all i), chunk u / BN.
    // B, NHWC: unit u = t + i*256 -> column u / CPR, chunk u % CPR.
    const int bn = t % BN;
    const int bkc0 = __builtin_amdgcn_readfirstlane(t / BN);
    const int pcol = p0 + bn;
    ColState cs;
    ColState csn[NHWC ? BUNITS : 1];
    if constexpr (NHWC) {
#pragma unroll
        for (int i = 0; i < BUNITS; ++i) csn[i] = col_state_nhwc(A, p0 + (t + i * 256) / CPR, gi);
    } else if (BSRC != BSRC_DENSE && BSRC != BSRC_DENSE_T) {
        cs = col_state(A, pcol, gi);
    }
    const uint32_t dvb = pcol < A.P ? (uint32_t)(((int64_t)gi * A.b_gstride + pcol) * 2) : OOB_OFF;
    // A: unit u = t + i*256 -> row m = u / CPR, k chunk kc = u % CPR
    const int64_t a_base = (int64_t)gi * A.a_gstride;

    // staging registers: PF sets, the loads of a stage issued PF stages before its compute
    static_assert(PF == 1 || PF == 2, "prefetch distance");
    u32x4 bset[PF][BUNITS];
    u32x4 aset[PF][AUNITS];
    int cur_c0 = 0, cur_r = 0, cur_s = 0;  // tap-major cursor of the next stage
    if constexpr (BSRC == BSRC_IMPLICIT_TAP || BSRC == BSRC_NHWC_TAP) {
        if (A.Cg >= BK) {  // (C/g < BK, 32-deep stages only: the small-group NHWC gather indexes by stage)
            const int cblocks = A.Cg / BK;
            const int tap = s_begin / cblocks;
            cur_c0 = (s_begin - tap * cblocks) * BK;
            cur_r = tap / A.S;
            cur_s = tap - cur_r * A.S;
        }
        // the divisions above run on the vector unit; the cursor is block-uniform, and taking
        // it into scalar registers keeps its per-stage update off the vector ALU
        cur_c0 = __builtin_amdgcn_readfirstlane(cur_c0);
        cur_r = __builtin_amdgcn_readfirstlane(cur_r);
        cur_s = __builtin_amdgcn_readfirstlane(cur_s);
    }

    auto load_weights_tap = [&](u32x4 (&areg)[AUNITS]) {
        // weights in tap-major order [K][R*S][C/g]: 8 consecutive channels per 16-byte load
        const int tap = cur_r * A.S + cur_s;
#pragma unroll
        for (int i = 0; i < AUNITS; ++i) {
            const int u = t + i * 256;
            const bool qa = AQ % 256 == 0 || u < AQ;
            const int m = m0 + u / CPR;
            const int kc = u % CPR;
            const int64_t e0 = a_base + (int64_t)m * A.lda + (int64_t)tap * A.Cg + cur_c0 + kc * 8;
            areg[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, ((m < A.M) & qa) ? (uint32_t)(e0 * 2) : OOB_OFF, 0, 0);
        }
    };
    // NHWC gather with C/g >= BK: 32-bit byte offsets per load unit computed once, so a stage
    // adds one wave-uniform offset per load (the 64-bit address arithmetic and the bounds tests
    // per load had cost about 9 vector instructions per MFMA, and the vector ALU does not run
    // beside the MFMAs).  nb_off: window origin + chunk of unit i (a window starting in the
    // padding wraps; the offset of every tap inside the image comes out right modulo 2^32);
    // vb_off: the same plus the current tap's offset, or out of range where that tap falls
    // outside the image (recomputed when the tap changes); na_off: weight row + chunk.
    uint32_t nb_off[NHWC ? BUNITS : 1], vb_off[NHWC ? BUNITS : 1], na_off[NHWC ? AUNITS : 1];
    auto tap_offsets = [&]() {
        if constexpr (NHWC) {
            const int roff = cur_r * A.dh, soff = cur_s * A.dw;
            const uint32_t tb = (uint32_t)((roff * A.W + soff) * A.Cx) * 2u;
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const bool ok = ((unsigned)(csn[i].hi0 + roff) < (unsigned)A.H) &
                                ((unsigned)(csn[i].wi0 + soff) < (unsigned)A.W);
                vb_off[i] = ok ? nb_off[i] + tb : OOB_OFF;
            }
        }
    };
    const bool nhwc_fast = NHWC && (BK == 64 || A.Cg >= BK);
    if constexpr (NHWC) {
        if (nhwc_fast) {
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const int kc = (t + i * 256) % CPR;
                nb_off[i] = (uint32_t)(csn[i].base + kc * 8) * 2u;
            }
#pragma unroll
            for (int i = 0; i < AUNITS; ++i) {
                const int u = t + i * 256;
                const bool qa = AQ % 256 == 0 || u < AQ;
                const int m = m0 + u / CPR;
                const int kc = u % CPR;
                na_off[i] = ((m < A.M) & qa) ? (uint32_t)(a_base + (int64_t)m * A.lda + kc * 8) * 2u : OOB_OFF;
            }
            tap_offsets();
        }
    }
    auto advance_tap = [&]() {
        cur_c0 += BK;
        if (cur_c0 >= A.Cg) {
            cur_c0 = 0;
            if (++cur_s == A.S) {
                cur_s = 0;
                ++cur_r;
            }
        }
    };

    auto load_stage = [&](int stage, u32x4 (&breg)[BUNITS], u32x4 (&areg)[AUNITS]) {
        const int k0 = stage * BK;
        uint16_t h[8];
        if constexpr (BSRC == BSRC_DENSE_T) {
            // B^T[gi][p][k] (row pitch ldb) and A[gi][m][k] (row pitch lda), 8 values per load
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const int u = t + i * 256;
                const int col = p0 + u / CPR;
                const int kr = k0 + (u % CPR) * 8;
                const int64_t e = (int64_t)gi * A.b_gstride + (int64_t)col * A.ldb + kr;
                breg[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    rb, (col < A.P) & (kr < A.Kred) ? (uint32_t)(e * 2) : OOB_OFF, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < AUNITS; ++i) {
                const int u = t + i * 256;
                const bool qa = AQ % 256 == 0 || u < AQ;
                const int m = m0 + u / CPR;
                const int kr = k0 + (u % CPR) * 8;
                const int64_t e0 = a_base + (int64_t)m * A.lda + kr;
                areg[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    ra, (m < A.M) & (kr < A.Kred) & qa ? (uint32_t)(e0 * 2) : OOB_OFF, 0, 0);
            }
        } else if (NHWC && BK == 32 && A.Cg < BK) {
            // C/g = 8 or 16: a stage holds BK / (C/g) whole taps; chunk kc of a pixel is the
            // 8 channels (kc*8) % (C/g) .. +7 of tap k0/(C/g) + kc*8/(C/g) (zero past the last tap)
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const int kc = (t + i * 256) % CPR;
                const int kr = k0 + kc * 8;
                const int tap = kr / A.Cg;
                const int c = kr - tap * A.Cg;
                const int r = tap / A.S, sx = tap - (tap / A.S) * A.S;
                const int hi = csn[i].hi0 + r * A.dh, wi = csn[i].wi0 + sx * A.dw;
                const bool ok = (tap < A.RS) & ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
                const int64_t e = csn[i].base + ((int64_t)(r * A.dh) * A.W + sx * A.dw) * A.Cx + c;
                breg[i] = __builtin_amdgcn_raw_buffer_load_b128(rb, ok ? (uint32_t)(e * 2) : OOB_OFF, 0, 0);
            }
            // weights in tap-major order [K][R*S][C/g]: row m, reduction k0 + kc*8 .. +7
#pragma unroll
            for (int i = 0; i < AUNITS; ++i) {
                const int u = t + i * 256;
                const bool qa = AQ % 256 == 0 || u < AQ;
                const int m = m0 + u / CPR;
                const int kr = k0 + (u % CPR) * 8;
                const int64_t e0 = a_base + (int64_t)m * A.lda + kr;
                areg[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    ra, (m < A.M) & (kr < A.Kred) & qa ? (uint32_t)(e0 * 2) : OOB_OFF, 0, 0);
            }
        } else if constexpr (NHWC) {
            // the stage's uniform part goes in the scalar offset: lanes whose vector offset is
            // out of range stay out of range, the others address inside the tensor
            const int cb = cur_c0 * 2;
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) breg[i] = __builtin_amdgcn_raw_buffer_load_b128(rb, vb_off[i], cb, 0);
            const int ab = ((cur_r * A.S + cur_s) * A.Cg + cur_c0) * 2;
#pragma unroll
            for (int i = 0; i < AUNITS; ++i) areg[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, na_off[i], ab, 0);
            advance_tap();
            if (cur_c0 == 0) tap_offsets();
        } else if constexpr (BSRC == BSRC_IMPLICIT_TAP) {
            const int roff = cur_r * A.dh, soff = cur_s * A.dw;
            const int hi = cs.hi0 + roff, wi = cs.wi0 + soff;
            const bool ok = ((unsigned)hi < (unsigned)A.H) & ((unsigned)wi < (unsigned)A.W);
            const uint32_t vb = ok ? (uint32_t)(((int32_t)cs.base + roff * A.W + soff) * 2) : OOB_OFF;
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const int kc = bkc0 + i * (256 / BN);
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    h[q] = ld_u16(rb, vb + (uint32_t)((cur_c0 + kc * 8 + q) * A.HW) * 2u);
#pragma unroll
                for (int q = 0; q < 4; ++q) breg[i][q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
            }
            load_weights_tap(areg);
            advance_tap();
        } else {
#pragma unroll
            for (int i = 0; i < BUNITS; ++i) {
                const int kc = bkc0 + i * (256 / BN);
                if constexpr (BSRC == BSRC_IMPLICIT_NCHW) {
                    KTabEntry e[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) e[q] = ktab_at(A.ktab, k0 + kc * 8 + q);
#pragma unroll
                    for (int q = 0; q < 8; ++q) h[q] = ld_u16(rb, implicit_off<2>(A, cs, e[q]));
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const int kr = k0 + kc * 8 + q;
                        h[q] = ld_u16(rb, kr < A.Kred ? dvb + (uint32_t)kr * (uint32_t)A.ldb * 2u : OOB_OFF);
                    }
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) breg[i][q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
            }
#pragma unroll
            for (int i = 0; i < AUNITS; ++i) {
                const int u = t + i * 256;
                const bool qa = AQ % 256 == 0 || u < AQ;
                const int m = m0 + u / CPR;
                const int kc = u % CPR;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int kr = k0 + kc * 8 + q;
                    const bool ok = (m < A.M) & (kr < A.Kred) & qa;
                    const int64_t e = a_base + (int64_t)m * A.lda + kr;
                    h[q] = ld_u16(ra, ok ? (uint32_t)(e * 2) : OOB_OFF);
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) areg[i][q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
            }
        }
    };
    // LDS byte offsets of this thread's B chunks (K-contiguous sources), computed once and kept
    // in registers (recomputing them per stage cost vector instructions)
    uint32_t bs_off[KCONT ? BUNITS : 1];
    if constexpr (KCONT) {
#pragma unroll
        for (int i = 0; i < BUNITS; ++i) {
            const int u = t + i * 256;
            bs_off[i] = (uint32_t)(((u / CPR) * LDK + (u % CPR) * 8) * 2);
            asm volatile("" : "+v"(bs_off[i]));
        }
    }
    uint32_t as_off[AUNITS];
#pragma unroll
    for (int i = 0; i < AUNITS; ++i) {
        const int u = t + i * 256;
        as_off[i] = (uint32_t)(((u / CPR) * LDK + (u % CPR) * 8) * 2);
        asm volatile("" : "+v"(as_off[i]));
    }
    auto store_stage = [&](int buf, const u32x4 (&breg)[BUNITS], const u32x4 (&areg)[AUNITS]) {
#pragma unroll
        for (int i = 0; i < BUNITS; ++i) {
            if constexpr (KCONT) {
                *reinterpret_cast<u32x4*>(reinterpret_cast<char*>(&Bs[buf][0][0]) + bs_off[i]) = breg[i];
            } else {
                const int kc = bkc0 + i * (256 / BN);
                *reinterpret_cast<u32x4*>(&Bs[buf][bn][kc * 8]) = breg[i];
            }
        }
#pragma unroll
        for (int i = 0; i < AUNITS; ++i) {
            const int u = t + i * 256;
            if (AQ % 256 == 0 || u < AQ)
                *reinterpret_cast<u32x4*>(reinterpret_cast<char*>(&As[buf][0][0]) + as_off[i]) = areg[i];
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

    auto compute = [&](int buf) {
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
    };

    // The 128 x 128 tile's stage with 64-deep reduction in one scheduling region: the operand
    // reads of k-step ks + 1 and the LDS stores of the next stage (set sb/sa into buffer wb)
    // are issued between the MFMAs of k-step ks, in the order the group barriers below give,
    // so that the matrix unit is not left waiting on LDS latency between k-steps.
    auto compute_store = [&](int rb, int wb, const u32x4 (&sb)[BUNITS], const u32x4 (&sa)[AUNITS]) {
        bf16x8 a[2][TM], b[2][TN];
        auto rd = [&](int ks, int o) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[o][i] = *reinterpret_cast<const bf16x8*>(&As[rb][wm0 + i * 32 + lcol][ks * 16 + 8 * lrow]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[o][j] = *reinterpret_cast<const bf16x8*>(&Bs[rb][wn0 + j * 32 + lcol][ks * 16 + 8 * lrow]);
        };
        rd(0, 0);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            if (ks + 1 < BK / 16) rd(ks + 1, (ks + 1) & 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks & 1][i], b[ks & 1][j], acc[i][j], 0, 0, 0);
        }
        store_stage(wb, sb, sa);
        if constexpr (TM == 2 && TN == 2 && BK == 64 && BUNITS + AUNITS == 8) {
#define CV_SG(mask, cnt) __builtin_amdgcn_sched_group_barrier(mask, cnt, 0)
            CV_SG(0x100, 4);  // operands of k-step 0
#pragma unroll
            for (int r = 0; r < 3; ++r) {  // k-steps 0..2: 4 MFMAs, 4 reads, 2 LDS stores each
                CV_SG(0x008, 1); CV_SG(0x100, 1); CV_SG(0x008, 1); CV_SG(0x100, 1); CV_SG(0x200, 1);
                CV_SG(0x008, 1); CV_SG(0x100, 1); CV_SG(0x008, 1); CV_SG(0x100, 1); CV_SG(0x200, 1);
            }
            CV_SG(0x008, 1); CV_SG(0x200, 1); CV_SG(0x008, 1); CV_SG(0x008, 1); CV_SG(0x200, 1); CV_SG(0x008, 1);
#undef CV_SG
        }
    };

    // Stage jj is computed from LDS buffer jj & 1 while register set jj % PF (free since its
    // stage went to LDS) takes the loads of stage jj + PF, and set (jj + 1) % PF, stage jj + 1,
    // goes to the other buffer.  The loop body is unrolled over two stages so that every
    // buffer and register set index is a constant.
    constexpr int U = 2;
    const int n = s_end - s_begin;
#pragma unroll
    for (int q = 0; q < PF; ++q)
        if (q < n) load_stage(s_begin + q, bset[q], aset[q]);
    store_stage(0, bset[0], aset[0]);
    __syncthreads();
    for (int j = 0; j < n; j += U) {
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int jj = j + q;
            if (jj >= n) break;
            // Issued on every stage, also past the block's last one (those loads read inside or
            // past the tensors, where the buffer range check returns zero, and are never
            // stored): with a condition here, the wait before the LDS stores would have to cover
            // the path without these loads and so wait for them too.  Not through the tap
            // table, which the loads past the end would read past.
            if (BSRC != BSRC_IMPLICIT_NCHW || jj + PF < n) load_stage(s_begin + jj + PF, bset[q % PF], aset[q % PF]);
            if (TM == 2 && TN == 2 && BK == 64 && PF == 2 && !A.loader_only) {
                // (the last stage also stores a stale set into the buffer no stage reads)
                compute_store(q & 1, (q + 1) & 1, bset[(q + 1) % PF], aset[(q + 1) % PF]);
            } else {
                if (!A.loader_only) compute(q & 1);
                if (jj + 1 < n) store_stage((q + 1) & 1, bset[(q + 1) % PF], aset[(q + 1) % PF]);
            }
            __syncthreads();
        }
    }

    if (A.loader_only) return;
    if constexpr (EPI != EPI_DENSE) {
        if (wk.tail_tile >= 0 && !tail_reduce<TM, TN>(A, acc, wk, t)) return;
    }
    store_tile<TM, TN, EPI, TOut>(A, acc, gi, sp, m0 + wm0, p0 + wn0, lrow, lcol);
}

// ============================================================================ dispatch
template <int BM, int BN, int WM, int WN, int BK, int PF>
static hipError_t launch_f32(const GemmArgs& a, int bsrc, int epi, int groups, hipStream_t stream) {
    dim3 grid((unsigned)(a.grid_p * a.grid_m + a.tail_tiles * (a.tail_pieces - 1)), 1,
              (unsigned)(groups * (a.ksplit > 1 ? a.ksplit : 1)));
#define CV_F32(BS, EP) \
    hipLaunchKernelGGL((gemm_f32_kernel<BM, BN, WM, WN, BK, PF, BS, EP, float>), grid, dim3(256), 0, stream, a)
    if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_NCHW) CV_F32(BSRC_IMPLICIT_NCHW, EPI_NCHW);
    else if (bsrc == BSRC_IMPLICIT_TAP && epi == EPI_NCHW) CV_F32(BSRC_IMPLICIT_TAP, EPI_NCHW);
    else if (bsrc == BSRC_DENSE && epi == EPI_DENSE) CV_F32(BSRC_DENSE, EPI_DENSE);
    // partial sums of a split reduction
    else if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_DENSE) CV_F32(BSRC_IMPLICIT_NCHW, EPI_DENSE);
    else if (bsrc == BSRC_IMPLICIT_TAP && epi == EPI_DENSE) CV_F32(BSRC_IMPLICIT_TAP, EPI_DENSE);
    // NHWC x with channel runs of 4 (C and C/g multiples of 4, C/g of the stage depth)
    else if (bsrc == BSRC_NHWC_TAP && (a.Cx % 4 != 0 || a.Cg % BK != 0)) return hipErrorInvalidValue;
    else if (bsrc == BSRC_NHWC_TAP && epi == EPI_NCHW) CV_F32(BSRC_NHWC_TAP, EPI_NCHW);
    else if (bsrc == BSRC_NHWC_TAP && epi == EPI_DENSE) CV_F32(BSRC_NHWC_TAP, EPI_DENSE);
    else if (bsrc == BSRC_NHWC_TAP && epi == EPI_NHWC) CV_F32(BSRC_NHWC_TAP, EPI_NHWC);
    else return hipErrorInvalidValue;
#undef CV_F32
    return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int BK, int PF>
static hipError_t launch_bf16(const GemmArgs& a, int bsrc, int epi, int ydt, int groups, hipStream_t stream) {
    dim3 grid((unsigned)(a.grid_p * a.grid_m + a.tail_tiles * (a.tail_pieces - 1)), 1,
              (unsigned)(groups * (a.ksplit > 1 ? a.ksplit : 1)));
    // NHWC gather: 16-byte channel runs, so C and C/g multiples of 8, and C/g a multiple of the
    // stage depth or (32-deep stages) a divisor of it
    if (bsrc == BSRC_NHWC_TAP && (a.Cg % 8 != 0 || a.Cx % 8 != 0 || (a.Cg >= BK ? a.Cg % BK : BK % a.Cg) != 0 ||
                                  (BK == 64 && a.Cg < BK)))
        return hipErrorInvalidValue;
    // dense B^T: 16-byte rows of 8 reduction values
    if (bsrc == BSRC_DENSE_T && (a.Kred % 8 != 0 || a.ldb % 8 != 0 || a.lda % 8 != 0 || epi != EPI_DENSE))
        return hipErrorInvalidValue;
#define CV_BF(BS, EP, TO) \
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, BK, PF, BS, EP, TO>), grid, dim3(256), 0, stream, a)
    if (bsrc == BSRC_NHWC_TAP && epi == EPI_NCHW) {
        if (ydt == CONV2D_BF16) CV_BF(BSRC_NHWC_TAP, EPI_NCHW, uint16_t);
        else CV_BF(BSRC_NHWC_TAP, EPI_NCHW, float);
    } else if (bsrc == BSRC_NHWC_TAP && epi == EPI_NHWC) {
        if (ydt == CONV2D_BF16) CV_BF(BSRC_NHWC_TAP, EPI_NHWC, uint16_t);
        else CV_BF(BSRC_NHWC_TAP, EPI_NHWC, float);
    } else if (bsrc == BSRC_NHWC_TAP && epi == EPI_DENSE) {
        CV_BF(BSRC_NHWC_TAP, EPI_DENSE, float);  // partial sums of a split reduction
    } else if constexpr (PF != 1) {
        return hipErrorInvalidValue;  // two register sets only with the NHWC gather
    } else if (bsrc == BSRC_DENSE_T) {
        CV_BF(BSRC_DENSE_T, EPI_DENSE, float);
    } else if (BK != 32) {
        return hipErrorInvalidValue;  // the NCHW gathers and the dense source use 32-row stages
    } else if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_NCHW) {
        if (ydt == CONV2D_BF16) CV_BF(BSRC_IMPLICIT_NCHW, EPI_NCHW, uint16_t);
        else CV_BF(BSRC_IMPLICIT_NCHW, EPI_NCHW, float);
    } else if (bsrc == BSRC_IMPLICIT_TAP && epi == EPI_NCHW) {
        if (ydt == CONV2D_BF16) CV_BF(BSRC_IMPLICIT_TAP, EPI_NCHW, uint16_t);
        else CV_BF(BSRC_IMPLICIT_TAP, EPI_NCHW, float);
    } else if (bsrc == BSRC_DENSE && epi == EPI_DENSE) {
        CV_BF(BSRC_DENSE, EPI_DENSE, float);
    } else if (bsrc == BSRC_IMPLICIT_NCHW && epi == EPI_DENSE) {
        CV_BF(BSRC_IMPLICIT_NCHW, EPI_DENSE, float);  // partial sums of a split reduction
    } else if (bsrc == BSRC_IMPLICIT_TAP && epi == EPI_DENSE) {
        CV_BF(BSRC_IMPLICIT_TAP, EPI_DENSE, float);
    } else {
        return hipErrorInvalidValue;
    }
#undef CV_BF
    return hipGetLastError();
}

bool gemm32_f32_supported(int tile, int bk, int pf) {
    if (tile < 0 || tile >= TILE_COUNT || (pf != 1 && pf != 2)) return false;
    if (bk == 16) return true;
    return bk == 32 && (tile == TILE_64x64 || tile == TILE_64x128);
}

hipError_t launch_gemm(const GemmArgs& a, int tile, int bk, int pf, int bsrc, int epi, int xdt, int ydt,
                       int groups, hipStream_t stream) {
    if (a.tail_tiles != 0) {
        // the tail split covers whole tiles of one group, every piece non-empty
        const int64_t tiles = (int64_t)a.grid_p * a.grid_m;
        if (a.tail_tiles < 0 || a.tail_tiles > tiles || a.tail_pieces < 2 || a.tail_stages < 1 ||
            groups != 1 || a.ksplit > 1 || !a.tail_part || !a.tail_count ||
            (int64_t)a.tail_pieces * a.tail_stages < a.nstages ||
            (int64_t)(a.tail_pieces - 1) * a.tail_stages >= a.nstages ||
            tiles + (int64_t)a.tail_tiles * (a.tail_pieces - 1) > 0x7fffffffLL)
            return hipErrorInvalidValue;
    }
    if (xdt == CONV2D_BF16) {
        // two register sets (pf 2): 64-deep stages with the NHWC gather only
        if ((bk != 32 && bk != 64) || (pf != 1 && (pf != 2 || bk != 64 || bsrc != BSRC_NHWC_TAP)))
            return hipErrorInvalidValue;
#define CV_TB(BMV, BNV, WMV, WNV) \
    return bk == 64 ? (pf == 2 ? launch_bf16<BMV, BNV, WMV, WNV, 64, 2>(a, bsrc, epi, ydt, groups, stream) \
                               : launch_bf16<BMV, BNV, WMV, WNV, 64, 1>(a, bsrc, epi, ydt, groups, stream)) \
                    : launch_bf16<BMV, BNV, WMV, WNV, 32, 1>(a, bsrc, epi, ydt, groups, stream)
        switch (tile) {
            case TILE_64x64: CV_TB(64, 64, 2, 2);
            case TILE_64x128: CV_TB(64, 128, 1, 4);
            case TILE_64x256: CV_TB(64, 256, 1, 4);
            case TILE_128x128: CV_TB(128, 128, 2, 2);
            case TILE_128x64: CV_TB(128, 64, 2, 2);
            case TILE_32x128: CV_TB(32, 128, 1, 4);
            case TILE_32x256: CV_TB(32, 256, 1, 4);
            default: return hipErrorInvalidValue;
        }
#undef CV_TB
    }
    if (!gemm32_f32_supported(tile, bk, pf)) return hipErrorInvalidValue;
#define CV_T(TL, BMV, BNV, WMV, WNV)                                                          \
    if (tile == TL) {                                                                        \
        if (bk == 16 && pf == 1) return launch_f32<BMV, BNV, WMV, WNV, 16, 1>(a, bsrc, epi, groups, stream); \
        if (bk == 16 && pf == 2) return launch_f32<BMV, BNV, WMV, WNV, 16, 2>(a, bsrc, epi, groups, stream); \
    }
    CV_T(TILE_64x64, 64, 64, 2, 2)
    CV_T(TILE_64x128, 64, 128, 1, 4)
    CV_T(TILE_64x256, 64, 256, 1, 4)
    CV_T(TILE_128x128, 128, 128, 2, 2)
    CV_T(TILE_128x64, 128, 64, 2, 2)
    CV_T(TILE_32x128, 32, 128, 1, 4)
    CV_T(TILE_32x256, 32, 256, 1, 4)
#undef CV_T
    if (tile == TILE_64x64 && bk == 32 && pf == 1) return launch_f32<64, 64, 2, 2, 32, 1>(a, bsrc, epi, groups, stream);
    if (tile == TILE_64x64 && bk == 32 && pf == 2) return launch_f32<64, 64, 2, 2, 32, 2>(a, bsrc, epi, groups, stream);
    if (tile == TILE_64x128 && bk == 32 && pf == 1) return launch_f32<64, 128, 1, 4, 32, 1>(a, bsrc, epi, groups, stream);
    if (tile == TILE_64x128 && bk == 32 && pf == 2) return launch_f32<64, 128, 1, 4, 32, 2>(a, bsrc, epi, groups, stream);
    return hipErrorInvalidValue;
}

}  // namespace cv
