// conv2d_internal.h -- shared declarations of the gfx950 conv2d library (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "conv2d.h"

namespace cv {

// Operation classes (bit positions of conv2d_plan_info::op_class).
enum { OPC_POINTWISE = 1, OPC_GROUPED = 2, OPC_DEPTHWISE = 4, OPC_DILATED = 8,
       OPC_RECTANGULAR = 16, OPC_STRIDED = 32 };

// Everything the kernels need to know about one convolution, in logical NCHW terms.
struct Geometry {
    int64_t N, C, H, W, K, R, S, Ho, Wo;
    int32_t sh, sw, ph, pw, dh, dw, G;
    int64_t Cg, Kg, Kred, P;   // P = N*Ho*Wo output pixels
    int32_t layout, xdt, ydt, has_bias;
    int64_t x_elems, w_elems, y_elems;
};

// Tile configurations of the MFMA GEMM kernels.
enum TileCfg { TILE_64x64 = 0, TILE_64x128 = 1, TILE_64x256 = 2, TILE_128x128 = 3,
               TILE_128x64 = 4, TILE_32x128 = 5, TILE_32x256 = 6, TILE_COUNT = 7 };
struct TileShape { int bm, bn; };
static const TileShape kTileShapes[TILE_COUNT] = {{64, 64}, {64, 128}, {64, 256}, {128, 128}, {128, 64},
                                                  {32, 128}, {32, 256}};

// Source of the GEMM's B operand (the im2col matrix, Kred x P).
//  IMPLICIT_NCHW : gathered from NCHW x, reduction index kr = (c, r, s) looked up in the tap table
//  DENSE         : read from a packed column matrix [G][Kred][ldb]
//  IMPLICIT_TAP  : gathered from NCHW x in tap-major order kr' = (r, s, c); one filter tap per
//                  stage, so needs C/g to be a multiple of the stage depth (no table)
//  NHWC_TAP      : (bf16) the same order gathered from an NHWC copy of x, 16 bytes per load
enum BSrc { BSRC_IMPLICIT_NCHW = 0, BSRC_DENSE = 1, BSRC_IMPLICIT_TAP = 2, BSRC_NHWC_TAP = 3, BSRC_DENSE_T = 4 };
// Destination of the GEMM result: NCHW y, a dense fp32 matrix, or NHWC y (ldc = K channels per
// pixel; NHWC gather source only).
enum Epi { EPI_NCHW = 0, EPI_DENSE = 1, EPI_NHWC = 2 };

// Per reduction index kr (one im2col row) of an NCHW input: the element offset
// of tap (c, r, s) relative to the window origin, and the row / column shifts
// used for the zero-padding test.  Rows beyond Kred carry roff = KTAB_DEAD so
// every bounds test fails and they read zero.
struct KTabEntry { int32_t coff, roff, soff, pad; };
constexpr int32_t KTAB_DEAD = -(1 << 29);
constexpr int KTAB_ALIGN = 64;   // table length is Kred rounded up to this

// Arguments of one MFMA GEMM launch (both algorithm families).
struct GemmArgs {
    const void* a;        // weights, [G][Kg][lda] in x dtype
    uint32_t a_bytes;
    int32_t lda;
    int64_t a_gstride;    // elements between groups
    const void* b;        // implicit: x (NCHW); dense: col [G][Kred][ldb]
    uint32_t b_bytes;
    int64_t b_gstride;    // elements between groups
    int32_t ldb;
    const KTabEntry* ktab;
    int32_t H, W, Ho, Wo, sh, sw, ph, pw;
    int32_t dh, dw, R, S, RS, Cg, HW;  // tap-major gather: filter dims, R*S, channels per group, H*W
    int32_t Cx;           // NHWC source: channels per pixel (all groups)
    int64_t x_nstride;    // C*H*W
    int32_t M, Kred, P, nstages;
    int32_t grid_p, grid_m;   // pixel tiles x channel tiles
    void* y;              // NCHW y, NHWC y, or dense C [G][M][ldc] (fp32)
    uint32_t y_bytes;
    const float* bias;    // may be NULL
    int64_t y_nstride;    // K*Ho*Wo
    int32_t HoWo;
    int32_t ldc;
    int64_t c_gstride;
    int32_t p_offset;     // global index of column 0 (explicit chunks)
    // split reduction: blockIdx.z = group * ksplit + split; split s runs stages
    // [s*split_stages, min((s+1)*split_stages, nstages)) and writes its partial result (dense
    // epilogue) at offset s*c_sstride.  ksplit 0 or 1: no split.
    int32_t ksplit, split_stages;
    int64_t c_sstride;
    // tail split (ksplit 1, one group): the last tail_tiles output tiles are each computed by
    // tail_pieces blocks of tail_stages consecutive stages, placed after the other blocks of the
    // grid.  Each piece writes its fp32 partial tile to tail_part; the last piece of a tile to
    // arrive (counted in tail_count, zero before a launch and reset to zero by that piece) adds
    // the partials in piece order and stores the tile.  tail_tiles 0: no tail split.
    int32_t tail_tiles, tail_pieces, tail_stages;
    float* tail_part;      // [tail_tiles][tail_pieces][BM*BN]
    uint32_t* tail_count;  // [tail_tiles]
    // pack probe: 1 runs the loader only (gathers into LDS, barriers), no MFMA, no output
    int32_t loader_only;
};

// 32x32-MFMA kernels.  fp32: stage depth bk in {16, 32}, register prefetch distance pf in {1, 2};
// bf16: bk in {32, 64} (64 only with the NHWC source), pf ignored.
bool gemm32_f32_supported(int tile, int bk, int pf);
hipError_t launch_gemm(const GemmArgs& a, int tile, int bk, int pf, int bsrc, int epi, int xdt, int ydt,
                       int groups, hipStream_t stream);


// im2col of a chunk of output pixels [p_begin, p_begin + pc): col[g][kr][pl].
struct Im2colArgs {
    const void* x;
    uint32_t x_bytes;     // x below 2 GiB: the gathers use 32-bit offsets into a range-checked
                          // buffer; 0: 64-bit addresses
    void* col;
    uint32_t col_bytes;
    const KTabEntry* ktab;
    int32_t H, W, Ho, Wo, sh, sw, ph, pw;
    int64_t x_nstride, x_gstride;
    int32_t Kred, pc;
    int64_t p_begin;
};
hipError_t launch_im2col(const Im2colArgs& a, int xdt, int groups, hipStream_t stream);

// unpack C[g][m][pl] (fp32) to NCHW y, or NHWC y with nhwc = 1 (+bias, cast).  With splits > 1
// the value is the sum, in split order, of C + s*split_stride over s < splits (a split
// reduction's partials).
struct UnpackArgs {
    const float* c;
    void* y;
    uint32_t y_bytes;
    const float* bias;
    int32_t Kg, pc, HoWo;
    int64_t p_begin;
    int64_t y_nstride;
    int32_t splits;
    int64_t split_stride;
    int32_t nhwc;
};
hipError_t launch_unpack(const UnpackArgs& a, int ydt, int groups, hipStream_t stream);

// direct convolution (NCHW) for depthwise / small-group layers.
struct DirectArgs {
    const void* x;
    const void* w;
    const float* bias;
    void* y;
    uint32_t x_bytes, y_bytes;
    uint32_t w_bytes;  // filters (range of the grouped kernels' buffer loads)
    int32_t C, H, W, K, Ho, Wo, R, S, sh, sw, ph, pw, dh, dw, Cg, Kg;
    int32_t N;
};
// Winograd F(mt x mt, 3x3), mt = 2 or 4: tiles t0 .. t0+tc-1 of th x tw tiles per image.
struct WinoArgs {
    const void* x;
    uint32_t x_bytes;
    void* y;
    uint32_t y_bytes;
    const float* bias;  // may be NULL
    int32_t C, H, W, K, Ho, Wo, ph, pw;
    int32_t mt;         // output tile edge (2 or 4); (mt+2)^2 transformed positions
    int32_t th, tw;     // tiles per image: ceil(Ho/mt) x ceil(Wo/mt)
    int64_t t0;
    int32_t tc;
};
// dt = CONV2D_F32 (F(2x2) or F(4x4)) or CONV2D_BF16 (F(2x2), w and U in bf16)
hipError_t launch_wino_filter(const void* w, void* u, int K, int C, int mt, int dt, hipStream_t stream);
hipError_t launch_wino_input(const WinoArgs& a, float* v, hipStream_t stream);
// bf16: V [16][tc][C] from the NHWC copy of x
hipError_t launch_wino_input_nhwc(const WinoArgs& a, uint16_t* v, hipStream_t stream);
hipError_t launch_wino_output(const WinoArgs& a, const float* m, int ydt, hipStream_t stream);

// Grouped direct kernel plan: bands of TR output rows, GB groups per block, CC input
// channels staged at a time (window in_rows x in_cols each, xfloats LDS floats for all of
// them; CC = GB * C/g when GB > 1), kchunks chunks of output channels per group, lds_bytes
// of dynamic LDS.
struct GrpPlan {
    int32_t TR, nbands, GB, CC, in_rows, in_cols, xfloats, kchunks, lds_bytes;
};
hipError_t launch_direct(const DirectArgs& a, int xdt, int ydt, hipStream_t stream);
// Ungrouped layers with K <= 4 and square 1/3/5/7 filters on the vector ALUs; the input
// channels split into `ranges` ranges (fp32 partials [range][K][P] in part, added by
// launch_unpack) or one range (y written directly, part = NULL).
struct SmallKArgs {
    int32_t cper;  // input channels per range
    float* part;
};
bool smallk_supported(const DirectArgs& a);
int smallk_ranges(const DirectArgs& a);
hipError_t launch_smallk(const DirectArgs& a, float* part, int ranges, int xdt, int ydt, hipStream_t stream);
// Depthwise layers (C/g = K/g = 1, C a multiple of 4) with NHWC x and y; wt = the filters
// as [R*S][C] (x dtype).
bool dw_nhwc_supported(const DirectArgs& a);
hipError_t launch_dw_nhwc(const DirectArgs& a, const void* wt, int xdt, int ydt, hipStream_t stream);
// Blocks the grouped direct kernel launches for this shape (0: it does not take the shape).
int64_t grouped_blocks(const DirectArgs& a);

// Division by a runtime divisor d >= 1 through a multiplier and a shift (round-up method of
// Granlund and Montgomery): n / d = (umulhi(n, m) + n) >> s for 0 <= n < 2^31, with
// s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1.
struct FastDiv {
    uint32_t m, s;
};
inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    const uint64_t m = ((1ull << 32) * ((1ull << s) - d)) / d + 1;
    return FastDiv{(uint32_t)m, s};
}

// Sliced direct convolution on MFMA (small C/g * R * S): per block the filters of 64 output
// channels, the input rows of 256 consecutive output pixels of one image and a table of the
// slice offset of every reduction index sit in LDS (weights at byte 0, then the table at
// lds_k_off, then the slice at lds_x_off).  Persistent blocks walk the tiles
// (group x channel tile, image, pixel tile).  NCHW x; NCHW or NHWC y.
constexpr int64_t SLICE_MAX_KRED = 1024;
constexpr int64_t SLICE_MAX_LDS = 80 * 1024;     // two blocks per CU
constexpr int64_t SLICE_MAX_LDS_1 = 160 * 1024;  // one block per CU
struct SliceArgs {
    const void* x;
    uint32_t x_bytes;
    const void* w;        // [K][C/g][R][S]
    uint32_t w_bytes;
    const float* bias;    // may be NULL
    void* y;
    uint32_t y_bytes;
    int32_t C, H, W, K, Ho, Wo, R, S, sh, sw, ph, pw, dh, dw, Cg, Kg;
    int32_t kred, kh;     // reduction length; per lane-half length (2*kh >= kred)
    int32_t ph_max, pwp;  // slice rows per channel (capacity), slice row length
    int32_t N, tiles_px, grid_m;
    int32_t tiles_total;  // G * grid_m * N * tiles_px
    int32_t nblocks;      // persistent grid size
    int32_t lds_k_off, lds_x_off, lds_bytes;
    int32_t loader_only;  // pack probe: slice copies and filter loads only, no MFMA, no output
    int32_t y_nhwc;       // 1: y is NHWC (x stays NCHW)
    // Last-round split: tiles [tail_start, tiles_total) (fewer than nblocks) are each computed
    // by tail_q blocks (a power of two dividing the waves per block), piece j of a tile by
    // the waves [j*nw/tail_q, (j+1)*nw/tail_q); block b takes piece b % tail_q of tile
    // tail_start + b / tail_q.  The tiles before tail_start are whole rounds of nblocks.
    // tail_q 0: no split (tail_start = tiles_total).
    int32_t tail_start, tail_q;
    // packed rows (bf16, column dilation 1, S <= 8, W even, x 4-byte aligned): the slice holds
    // bf16 pairs (input columns wi, wi + 1 with wi even) at column j = wi + pw + pk_shift,
    // pk_shift = pw % 2; the reduction runs over filter rows (c, r) padded to 8 taps, two rows
    // per MFMA step (kh = 8 * steps per lane half).
    int32_t pk, pk_shift;
    // slice buffers (1 or 2; with 2 the next tile's copy overlaps this tile's MFMAs), words each
    int32_t nbuf, xwords;
    // fp32 lines copied 16 bytes per lane (x4 = 1; W % 4 == 0, x 16-byte aligned): input column
    // wi sits at word wi + pw + xshift, xshift = (-pw) mod 4, so every 4-word group of a line is
    // wholly inside or wholly outside the image; the pixel bases move by xshift
    int32_t x4, xshift;
    // divisions of the tile and pixel decode and the filter load: by N*tiles_px, tiles_px,
    // grid_m, Wo and the filter row length 2*kh
    FastDiv fd_pergz, fd_tpx, fd_gm, fd_wo, fd_kw;
};
struct SlicePlan {
    bool ok;
    bool pk;              // packed-row bf16 layout (SliceArgs::pk)
    int32_t nw;           // waves per block (tile = 32*nw pixels)
    int32_t kh, ph_max, pwp, lds_k_off, lds_x_off, lds_bytes;
    int32_t pk_shift;
    int32_t nbuf, xwords;  // slice buffers and their size in 4-byte words
};
// pk: try the packed-row bf16 layout (falls back to one word per element when it does not apply);
// db: fp32 may take two slice buffers and the whole LDS of a CU (enough tiles for that)
SlicePlan slice_plan(int64_t Cg, int64_t R, int64_t S, int64_t Ho, int64_t Wo, int sh, int sw, int dh, int dw,
                     int xdt, int nw, int64_t W = 0, int pw = 0, bool pk = false, bool db = false);
hipError_t launch_slice(const SliceArgs& a, int xdt, int ydt, int nw, hipStream_t stream);

// weight repack to tap-major order: w [K][C/g][R*S] -> wr [K][R*S][C/g].
hipError_t launch_repack_tap_major(const void* w, void* wr, int64_t k, int64_t cg, int64_t rs, int elem_bytes,
                                   hipStream_t stream);

// dst[0:n] = value (counters that a launch expects at zero).
hipError_t launch_fill_u32(uint32_t* dst, int64_t n, uint32_t value, hipStream_t stream);
// The tap table (len entries, Kred live ones) written by a kernel: the same entries the
// planner computes on the host, for the entry point that uploads nothing.
hipError_t launch_ktab_fill(KTabEntry* t, int64_t len, int64_t kred, int64_t cg, int64_t r, int64_t s, int64_t h,
                            int64_t w, int dh, int dw, hipStream_t stream);

// layout transforms between NHWC and NCHW (one image = a [HW x C] <-> [C x HW] transpose).
hipError_t launch_nhwc_to_nchw(const void* src, void* dst, int64_t n, int64_t c, int64_t hw,
                               int elem_bytes, hipStream_t stream);
hipError_t launch_nchw_to_nhwc(const void* src, void* dst, int64_t n, int64_t c, int64_t hw,
                               int elem_bytes, hipStream_t stream);

}  // namespace cv
