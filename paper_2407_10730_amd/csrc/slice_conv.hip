// slice_conv.hip -- sliced direct convolution on MFMA for small reductions.
//
// For layers whose reduction C/g * R * S is short (stems: few input channels,
// large filters), an im2col column of one output pixel is a handful of input
// values that neighbouring pixels share many times over.  Gathering them from
// global memory per GEMM stage (the implicit GEMM) spends most of its time in
// address arithmetic and small loads, and the explicit path writes them all
// out.  Here one block stages, in LDS,
//   * the filters of 64 output channels, [64][kred] in the natural (c, r, s)
//     order with the reduction split into two halves of kh values,
//   * the input slice those pixels read: every input row a run of 256
//     consecutive output pixels of one image touches, zero-filled where the
//     window leaves the image (padding),
//   * a table of the slice offset of every reduction index,
// and the MFMA loop then reads each im2col column straight out of the slice
// (the paper's sliced convolution keeps input slices in fast memory and
// skips the packing step, Sec. II; this is that idea on the LDS of one CU).
//
// A tile is 64 output channels x 256 consecutive output pixels of one image;
// wave w (of 8, two per SIMD) computes the 64 x 32 tile of pixels 32w..32w+31;
// lane l covers pixel l%32 and the reduction half l/32, so the weight operand
// of a lane is a contiguous run of its LDS row (16-byte reads) and the input
// operand is one LDS read per reduction index at (pixel base + table offset).
//
// Blocks are persistent: each walks the tiles blockIdx.x, +gridDim.x, ... in
// (group, channel tile, image, pixel tile) order, permuted within each round of gridDim.x
// tiles so that the blocks of one XCD take consecutive tiles, and keeps the filters while
// the channel tile stays the same.  When the tiles do not fill whole rounds of the
// grid, the tiles of the last round are split: each goes to 2, 4 or 8 blocks, every
// block computing the pixels of some of its waves, so that round costs a fraction of a
// tile instead of a whole one on a few blocks while the rest wait.
// The slice is copied global -> LDS by the
// buffer unit itself (buffer loads with the LDS bit: no registers, padding
// comes back as zero from out-of-range offsets), one 4-byte LDS word per
// element for both dtypes.
#include "device_common.h"

namespace cv {

constexpr int SLICE_BM = 64;    // output channels per tile
constexpr int SLICE_UNR = 8;    // loads in flight per thread in the filter copy
constexpr int SLICE_LP = 256;   // slice line pitch in words (one column per thread)

// Buffer load of one element per lane straight into LDS: lane l writes the 4-byte LDS word
// lds_addr + 4*l (2-byte elements are zero-extended to a word); out-of-range offsets write
// zero.  Issued as inline assembly so that the compiler does not add a wait for these writes
// before every later LDS read: the kernel orders them itself (vmcnt wait, then a barrier).
__device__ __forceinline__ void lds_dma_b32(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_addr) {
    asm volatile("buffer_load_dword %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(lds_addr) : "memory");
}
// 16 bytes per lane: lane l writes LDS bytes lds_addr + 16*l .. + 15.
__device__ __forceinline__ void lds_dma_b128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_addr) {
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(lds_addr) : "memory");
}
__device__ __forceinline__ void lds_dma_u16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds_addr) {
    asm volatile("buffer_load_ushort %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(lds_addr) : "memory");
}
// Workgroup barrier after this wave's LDS operations complete.  Unlike __syncthreads it does
// not also wait for outstanding global loads and stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <typename T> struct SliceTraits;
template <> struct SliceTraits<float> { static constexpr int wpad = 4; };
template <> struct SliceTraits<uint16_t> { static constexpr int wpad = 8; };

// NW waves per block (4 or 8), tiles of 32*NW pixels.  The element-wise slice has one buffer:
// it is copied between tiles, and a second resident block keeps the MFMAs busy meanwhile (a
// second buffer would halve the resident blocks, which measured slower).  The packed-row slice
// is half the size, so two buffers fit beside the filters at two blocks per CU (A.nbuf = 2):
// the next tile's copy then goes out before the current tile's MFMAs.
// PK (bf16 only): the packed-row layout.  The slice holds bf16 pairs, one 4-byte word per two
// input columns (copied with dword loads), and the reduction runs over filter rows (c, r),
// each padded to 8 taps with zero weights, two rows per MFMA step (lane half h takes row
// 2*step + h).  The 8 values a lane feeds one MFMA are then 8 consecutive input columns of
// one slice line starting at j0 = ow*sw + shift: 5 word reads and 4 funnel shifts (by 16 bits
// when j0 is odd) instead of 8 single reads, a table lookup and the packing.
// fp32 and packed-row kernels are held to 128 registers: the planner puts 16 waves on a CU
// (4 per SIMD) and 129 registers would leave room for 3 (the element-wise bf16 kernels would
// spill under that limit and keep their 136).
template <typename T, typename TOut, int NW, bool PK>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 4 || PK ? 4 : 1))) void
slice_conv_kernel(SliceArgs A) {
    constexpr int SLICE_THREADS = 64 * NW;
    constexpr int SLICE_NPX = 32 * NW;
    extern __shared__ __attribute__((aligned(16))) char lds[];
    constexpr int ES = sizeof(T);
    const int wpitch = 2 * A.kh + SliceTraits<T>::wpad;  // LDS filter row pitch, elements
    T* wl = reinterpret_cast<T*>(lds);
    int32_t* ko = reinterpret_cast<int32_t*>(lds + A.lds_k_off);
    uint32_t* xs = reinterpret_cast<uint32_t*>(lds + A.lds_x_off);  // slice, one word per element

    const int t = threadIdx.x;
    const int lane = t & 63;

    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // wave-uniform: keeps the control flow scalar
    const int lcol = lane & 31;
    const int lrow = lane >> 5;
    const int howo = A.Ho * A.Wo;
    const int per_gz = A.N * A.tiles_px;  // tiles of one (group, channel tile)
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(A.x, A.x_bytes);

    // ---- slice offset of every reduction index (0 for the zero-weight tail); packed rows: word
    // offset of the slice line of every filter row (c, r)
    if constexpr (PK) {
        const int nr = A.Cg * A.R;
        for (int k = t; k < 2 * A.kh / 8; k += SLICE_THREADS) {
            int off = 0;
            if (k < nr) {
                const int c = k / A.R;
                const int r = k - c * A.R;
                off = (c * A.ph_max + r * A.dh) * (SLICE_LP / 2);
            }
            ko[k] = off;
        }
    } else {
        const int rs = A.R * A.S;
        for (int k = t; k < 2 * A.kh; k += SLICE_THREADS) {
            int off = 0;
            if (k < A.kred) {
                const int c = k / rs;
                const int q = k - c * rs;
                const int r = q / A.S;
                const int s = q - r * A.S;
                off = (c * A.ph_max + r * A.dh) * SLICE_LP + s * A.dw;
            }
            ko[k] = off;
        }
    }

    // Work items of this block: whole tiles b, b + nb, ... below tail_start, then (with the
    // last-round split) one piece of a tile past it.  Item i -> tile index and the waves that
    // compute it.
    const int nb = (int)gridDim.x;
    const int bid = (int)blockIdx.x;
    const int nfull = bid < A.tail_start ? (A.tail_start - bid + nb - 1) / nb : 0;
    const bool piece = A.tail_q > 0 && bid < (A.tiles_total - A.tail_start) * A.tail_q;
    const int nitems = nfull + (piece ? 1 : 0);
    const int pw_n = A.tail_q > 0 ? NW / A.tail_q : NW;  // waves of a piece
    const int pw0 = A.tail_q > 0 ? (bid % A.tail_q) * pw_n : 0;

    // Geometry of tile w: image n, first pixel p0, first slice row hi0.
    struct Tile { int gz, n, p0, oh0, hi0; };
    // (wave-uniform arithmetic; divisions by the launch's runtime sizes use their FastDiv)
    auto decode = [&](int i) {
        int w;
        if (i < nfull) {
            // round i; XCD-contiguous order: the blocks of one XCD take consecutive tiles of
            // each round of nb tiles, so input rows that neighbouring tiles share stay in one L2
            w = i * nb + xcd_remap(bid, min(nb, A.tail_start - i * nb));
        } else {
            w = A.tail_start + bid / A.tail_q;
        }
        Tile tl;
        tl.gz = (int)fdiv((uint32_t)w, A.fd_pergz);
        const int rem = w - tl.gz * per_gz;
        tl.n = (int)fdiv((uint32_t)rem, A.fd_tpx);
        tl.p0 = (rem - tl.n * A.tiles_px) * SLICE_NPX;
        tl.oh0 = (int)fdiv((uint32_t)tl.p0, A.fd_wo);
        tl.hi0 = tl.oh0 * A.sh - A.ph;
        return tl;
    };

    // ---- slice of tile tl into buffer buf: line u = c*ph_max + row holds input row
    // hi0 + row of channel c in columns j = wi + pw; lane t of the block copies column t of
    // every line
    // nwc: the waves that copy (all NW, or the first NW/2 while the others load the filters);
    // the other waves return at once
    auto copy_slice = [&](const Tile& tl, uint32_t* buf, int nwc) {
        if (wave >= nwc) return;
        const int gi = (int)fdiv((uint32_t)tl.gz, A.fd_gm);
        if constexpr (PK) {
            // packed rows: a line is 128 words; wave w copies words 64*(w%2) .. +63 of lines
            // w/2, w/2 + NW/2, ...; word m holds input columns wi, wi + 1 with
            // wi = 2m - pw - shift (even, so both are in the row or both in the padding)
            const int m = (wave & 1) * 64 + lane;
            const int wi = 2 * m - A.pw - A.pk_shift;
            const bool wok = (unsigned)wi < (unsigned)A.W;
            const uint32_t hw = (uint32_t)(A.H * A.W);
            const uint32_t plane0 = (uint32_t)(tl.n * A.C + gi * A.Cg) * hw;
            const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
                (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)(buf + (wave & 1) * 64));
            const int lines = A.Cg * A.ph_max;
            // line u = c*ph_max + row, walked with (c, row) kept alongside (nwc/2 < ph_max or
            // the inner loop steps c more than once)
            const int lstep = nwc >> 1;
            int c = 0, row = wave >> 1;
            while (row >= A.ph_max) {
                row -= A.ph_max;
                ++c;
            }
            uint32_t plane = plane0 + (uint32_t)c * hw;
            for (int u = wave >> 1; u < lines; u += lstep) {
                const int hi = tl.hi0 + row;
                const bool ok = wok & ((unsigned)hi < (unsigned)A.H);
                const uint32_t e = plane + (uint32_t)(hi * A.W + wi);
                lds_dma_b32(rx, ok ? e * 2u : OOB_OFF, lds0 + (uint32_t)(u * (SLICE_LP / 2) * 4));
                row += lstep;
                while (row >= A.ph_max) {
                    row -= A.ph_max;
                    ++c;
                    plane += hw;
                }
            }
            return;
        }
        if constexpr (ES == 4) {
            if (A.x4) {
                // 16 bytes per lane: wave w copies whole lines w, w + nwc, ...; lane l words
                // 4l .. 4l + 3, input columns 4l - pw - xshift ..
                const int wi = 4 * lane - A.pw - A.xshift;
                const bool wok = (4 * lane < A.pwp + A.xshift) & ((unsigned)wi < (unsigned)A.W);
                const uint32_t hw = (uint32_t)(A.H * A.W);
                const uint32_t plane0 = (uint32_t)(tl.n * A.C + gi * A.Cg) * hw;
                const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
                    (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)buf);
                const int lines = A.Cg * A.ph_max;
                int c = 0, row = wave;
                while (row >= A.ph_max) {
                    row -= A.ph_max;
                    ++c;
                }
                uint32_t plane = plane0 + (uint32_t)c * hw;
                for (int u = wave; u < lines; u += nwc) {
                    const int hi = tl.hi0 + row;
                    const bool ok = wok & ((unsigned)hi < (unsigned)A.H);
                    const uint32_t e = plane + (uint32_t)(hi * A.W + wi);
                    lds_dma_b128(rx, ok ? e * 4u : OOB_OFF, lds0 + (uint32_t)(u * SLICE_LP * 4));
                    row += nwc;
                    while (row >= A.ph_max) {
                        row -= A.ph_max;
                        ++c;
                        plane += hw;
                    }
                }
                return;
            }
        }
        const int col = t & (SLICE_LP - 1);    // each group of 4 waves covers the 256 columns
        const int half = wave >> 2;            // ... of every (nwc/4)-th line
        const int rstep = nwc >> 2;
        const int wi = col - A.pw;
        const bool wok = (col < A.pwp) & ((unsigned)wi < (unsigned)A.W);
        const uint32_t plane0 = (uint32_t)(tl.n * A.C + gi * A.Cg) * (uint32_t)(A.H * A.W);
        // LDS byte address of this wave's 64 columns of line 0
        const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
            (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)(buf + (wave & 3) * 64));
        const uint32_t hw = (uint32_t)(A.H * A.W);
        for (int c = 0; c < A.Cg; ++c) {
            const uint32_t plane = plane0 + (uint32_t)c * hw;
            for (int row = half; row < A.ph_max; row += rstep) {
                const int hi = tl.hi0 + row;
                const bool ok = wok & ((unsigned)hi < (unsigned)A.H);
                const uint32_t e = plane + (uint32_t)(hi * A.W + wi);
                // lane l of the wave lands in word l of the destination
                const uint32_t la = lds0 + (uint32_t)((c * A.ph_max + row) * SLICE_LP * 4);
                if constexpr (ES == 4)
                    lds_dma_b32(rx, ok ? e * 4u : OOB_OFF, la);
                else
                    lds_dma_u16(rx, ok ? e * 2u : OOB_OFF, la);
            }
        }
    };

    // ---- filters of channel tile gz: wl[m][k], zero beyond kred or Kg, loaded by the threads
    // t0 .. t0 + nth - 1 (the others return)
    auto load_filters = [&](const Tile& tl, int t0, int nth) {
        if (t < t0) return;
        const int gi = (int)fdiv((uint32_t)tl.gz, A.fd_gm);
        const int m0 = (tl.gz - gi * A.grid_m) * SLICE_BM;
        const __amdgpu_buffer_rsrc_t rw = make_rsrc(A.w, A.w_bytes);
        const int kw = 2 * A.kh;
        const int total = SLICE_BM * kw;
        if constexpr (PK) {
            // packed rows: one (channel m, filter row rr) pair per thread at a time: its S
            // taps are consecutive in the natural order (loads at immediate offsets), the
            // 8-tap row goes to LDS with one 16-byte store (taps past S are zero)
            const int nrow = kw >> 3;
            for (int pr = t - t0; pr < SLICE_BM * nrow; pr += nth) {
                const int m = (int)fdiv((uint32_t)(pr * 8), A.fd_kw);
                const int rr = pr - m * nrow;
                const bool ok = (m0 + m < A.Kg) & (rr < A.Cg * A.R);
                const uint32_t off =
                    ok ? ((uint32_t)(gi * A.Kg + m0 + m) * (uint32_t)A.kred + (uint32_t)(rr * A.S)) * 2u : OOB_OFF;
                uint32_t h[8];
#pragma unroll
                for (int sx = 0; sx < 8; ++sx) {
                    const uint32_t v = __builtin_amdgcn_raw_buffer_load_b16(rw, off + 2u * sx, 0, 0);
                    h[sx] = sx < A.S ? v : 0u;
                }
                *reinterpret_cast<u32x4*>(wl + m * wpitch + rr * 8) =
                    u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
            }
        } else
        for (int base = t - t0; base < total; base += nth * SLICE_UNR) {
            T v[SLICE_UNR];
            int dst[SLICE_UNR];
#pragma unroll
            for (int u = 0; u < SLICE_UNR; ++u) {
                const int i0 = base + u * nth;
                const int idx = i0;
                const int m = (int)fdiv((uint32_t)idx, A.fd_kw);
                const int k = idx - m * kw;
                const bool ok = (i0 < total) & (m0 + m < A.Kg) & (k < A.kred);
                const uint32_t e = (uint32_t)(gi * A.Kg + m0 + m) * (uint32_t)A.kred + (uint32_t)k;
                if constexpr (ES == 4)
                    v[u] = ld_f32(rw, ok ? e * 4u : OOB_OFF);
                else
                    v[u] = ld_u16(rw, ok ? e * 2u : OOB_OFF);
                dst[u] = i0 < total ? m * wpitch + k : -1;
            }
#pragma unroll
            for (int u = 0; u < SLICE_UNR; ++u)
                if (dst[u] >= 0) wl[dst[u]] = v[u];
        }
    };

    f32x16 acc0, acc1;
    float bv0[16], bv1[16];
    int stores_out = 0;  // output stores of the previous tile still counted in vmcnt
    int cur_gz = -1;
    Tile nxt{};  // the tile whose slice was copied last (the next item's)
    // slice buffer of item i (two buffers: items alternate, and the copy of item i + 1 goes out
    // as soon as item i's slice has landed, before its MFMAs)
    const bool dbuf = A.nbuf == 2;
    auto xbuf = [&](int i) { return dbuf && (i & 1) ? xs + A.xwords : xs; };
    // the bias of the lane's 32 output channels of channel tile gz, in registers
    auto load_bias = [&](const Tile& tl) {
        const int gi = (int)fdiv((uint32_t)tl.gz, A.fd_gm);
        const int m0 = (tl.gz - gi * A.grid_m) * SLICE_BM;
        const __amdgpu_buffer_rsrc_t rbias = make_rsrc(A.bias, A.bias ? (uint32_t)A.K * 4u : 0u);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int m = m0 + 8 * (v >> 2) + 4 * lrow + (v & 3);
            bv0[v] = ld_f32(rbias, A.bias && m < A.Kg ? (uint32_t)(gi * A.Kg + m) * 4u : OOB_OFF);
            bv1[v] = ld_f32(rbias, A.bias && m + 32 < A.Kg ? (uint32_t)(gi * A.Kg + m + 32) * 4u : OOB_OFF);
        }
    };
    if (nitems > 0) {
        // start-up: the first half of the waves copies the first slice while the second half
        // loads the filters, so the two round trips to memory overlap (no wave has read any
        // filters yet, so no barrier first).  The element-wise slice of 4-wave blocks needs
        // all four waves for a line: there every wave copies first.
        nxt = decode(0);
        const bool split = PK || NW >= 8;
        copy_slice(nxt, xs, split ? NW / 2 : NW);
        load_filters(nxt, split ? 32 * NW : 0, split ? 32 * NW : SLICE_THREADS);
        load_bias(nxt);
        cur_gz = nxt.gz;
    }
    for (int item = 0; item < nitems; ++item) {
        const Tile tl = nxt;
        uint32_t* const xcur = xbuf(item);
        // waves outside this item's piece only copy and wait (wave-uniform)
        const bool active = item < nfull || (wave >= pw0 && wave < pw0 + pw_n);
        const int gi = (int)fdiv((uint32_t)tl.gz, A.fd_gm);
        const int m0 = (tl.gz - gi * A.grid_m) * SLICE_BM;
        if (tl.gz != cur_gz) {
            __syncthreads();  // no wave still reads the previous filters
            load_filters(tl, 0, SLICE_THREADS);
            load_bias(tl);
            cur_gz = tl.gz;
        }
        // This wave's slice copies (and filter loads) have landed, then every other wave's.
        // Vector memory operations complete in issue order and the previous tile's output
        // stores were issued after this tile's copy, so waiting until no more than those stores
        // are outstanding waits for the copy alone: the stores drain while this tile computes.
        if (stores_out == 32)
            asm volatile("s_waitcnt vmcnt(32)" ::: "memory");
        else if (stores_out == 16)
            asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        else if (stores_out == 8)
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        else
            __builtin_amdgcn_s_waitcnt(0);
        stores_out = 0;
        lds_barrier();  // (also: every wave is done with the previous item's buffer)
        if (dbuf && item + 1 < nitems) {
            nxt = decode(item + 1);
            copy_slice(nxt, xbuf(item + 1), NW);
        }

        if (A.loader_only || !active) {
            // pack probe (the next slice copy only), or a wave outside the piece
            if (!dbuf) {
                lds_barrier();
                if (item + 1 < nitems) {
                    nxt = decode(item + 1);
                    copy_slice(nxt, xs, NW);
                }
            }
            continue;
        }
        const int p = tl.p0 + wave * 32 + lcol;
        int pixbase = 0;  // pixels past the end read a valid (discarded) column
        if (p < howo) {
            const int oh = (int)fdiv((uint32_t)p, A.fd_wo);
            const int ow = p - oh * A.Wo;
            pixbase = (oh - tl.oh0) * A.sh * SLICE_LP + ow * A.sw + A.xshift;
        }
        const T* wa0 = wl + lcol * wpitch + lrow * A.kh;
        const T* wa1 = wa0 + 32 * wpitch;
        const int32_t* kp = ko + lrow * A.kh;
        const uint32_t* xp = xcur + pixbase;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            // the bias goes in first: the MFMAs add the products to it
            acc0[v] = bv0[v];
            acc1[v] = bv1[v];
        }

        if constexpr (PK) {
            // packed rows: step st feeds filter row rr = 2*st + lrow (weights wl[m][rr][8]) and
            // the 8 slice columns j0 .. j0 + 7 of that row's line
            int pw_ = 0, sha = 0;
            if (p < howo) {
                const int oh = (int)fdiv((uint32_t)p, A.fd_wo);
                const int ow = p - oh * A.Wo;
                const int j0 = ow * A.sw + A.pk_shift;
                pw_ = (oh - tl.oh0) * A.sh * (SLICE_LP / 2) + (j0 >> 1);
                sha = (j0 & 1) * 16;
            }
            const uint32_t* xb = xcur + pw_;
            const uint16_t* wr0 = reinterpret_cast<const uint16_t*>(wl) + lcol * wpitch + lrow * 8;
            const uint16_t* wr1 = wr0 + 32 * wpitch;
            const int nst = A.kh >> 3;
            auto operand_b = [&](int st) {
                const uint32_t* q = xb + ko[2 * st + lrow];
                const uint32_t w0 = q[0], w1 = q[1], w2 = q[2], w3 = q[3], w4 = q[4];
                const u32x4 v{__builtin_amdgcn_alignbit(w1, w0, sha), __builtin_amdgcn_alignbit(w2, w1, sha),
                              __builtin_amdgcn_alignbit(w3, w2, sha), __builtin_amdgcn_alignbit(w4, w3, sha)};
                return __builtin_bit_cast(bf16x8, v);
            };
            // (the other waves of the SIMD hide the LDS latency; unrolled so the reads of the
            // next step can go out before the MFMAs of this one)
#pragma unroll 2
            for (int st = 0; st < nst; ++st) {
                const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(wr0 + 16 * st);
                const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(wr1 + 16 * st);
                const bf16x8 b = operand_b(st);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b, acc1, 0, 0, 0);
            }
        } else if constexpr (ES == 4) {
            // MFMA 32x32x2: step k takes reduction index k of the lane's half.  Software
            // pipelined: the operands of group kk+4 (and the offsets of kk+8) are read while
            // the MFMAs of group kk run; reads past the end are clamped to the last group.
            const int last = A.kh - 4;
            int4 o = *reinterpret_cast<const int4*>(kp);
            f32x4 a0 = *reinterpret_cast<const f32x4*>(wa0);
            f32x4 a1 = *reinterpret_cast<const f32x4*>(wa1);
            float b0 = __builtin_bit_cast(float, xp[o.x]), b1 = __builtin_bit_cast(float, xp[o.y]),
                  b2 = __builtin_bit_cast(float, xp[o.z]), b3 = __builtin_bit_cast(float, xp[o.w]);
            o = *reinterpret_cast<const int4*>(kp + min(4, last));
            auto group = [&](const f32x4& x0, const f32x4& x1, float y0, float y1, float y2, float y3) {
                acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(x0[0], y0, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(x1[0], y0, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(x0[1], y1, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(x1[1], y1, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(x0[2], y2, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(x1[2], y2, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(x0[3], y3, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(x1[3], y3, acc1, 0, 0, 0);
            };
            // two groups per trip, the operands alternating between two register sets (a
            // rotation at the end of every group cost 8 moves per 8 MFMAs, and the vector ALU
            // does not run beside the MFMAs)
            for (int kk = 0; kk < A.kh; kk += 8) {
                const int kn = min(kk + 4, last);
                const f32x4 a0n = *reinterpret_cast<const f32x4*>(wa0 + kn);
                const f32x4 a1n = *reinterpret_cast<const f32x4*>(wa1 + kn);
                const float c0 = __builtin_bit_cast(float, xp[o.x]), c1 = __builtin_bit_cast(float, xp[o.y]),
                            c2 = __builtin_bit_cast(float, xp[o.z]), c3 = __builtin_bit_cast(float, xp[o.w]);
                o = *reinterpret_cast<const int4*>(kp + min(kk + 8, last));
                // keep the next group's reads ahead of this group's MFMAs
                __builtin_amdgcn_sched_barrier(0);
                group(a0, a1, b0, b1, b2, b3);
                __builtin_amdgcn_sched_barrier(0);
                if (kk + 4 >= A.kh) break;
                const int km = min(kk + 8, last);
                a0 = *reinterpret_cast<const f32x4*>(wa0 + km);
                a1 = *reinterpret_cast<const f32x4*>(wa1 + km);
                b0 = __builtin_bit_cast(float, xp[o.x]);
                b1 = __builtin_bit_cast(float, xp[o.y]);
                b2 = __builtin_bit_cast(float, xp[o.z]);
                b3 = __builtin_bit_cast(float, xp[o.w]);
                o = *reinterpret_cast<const int4*>(kp + min(kk + 12, last));
                __builtin_amdgcn_sched_barrier(0);
                group(a0n, a1n, c0, c1, c2, c3);
            }
        } else {
            // MFMA 32x32x16 bf16: a step takes 8 consecutive reduction indices of the lane's
            // half; the raw values of the next step are read before this step's MFMAs and
            // packed after them.
            // slice words hold one bf16 each, zero-extended
            const int last = A.kh - 8;
            uint32_t h[8];
            auto gather = [&](const int4& q0, const int4& q1) {
                h[0] = xp[q0.x]; h[1] = xp[q0.y]; h[2] = xp[q0.z]; h[3] = xp[q0.w];
                h[4] = xp[q1.x]; h[5] = xp[q1.y]; h[6] = xp[q1.z]; h[7] = xp[q1.w];
            };
            auto pack = [&]() {
                u32x4 bw;
#pragma unroll
                for (int q = 0; q < 4; ++q) bw[q] = h[2 * q] | (h[2 * q + 1] << 16);
                return __builtin_bit_cast(bf16x8, bw);
            };
            int4 o0 = *reinterpret_cast<const int4*>(kp);
            int4 o1 = *reinterpret_cast<const int4*>(kp + 4);
            bf16x8 a0 = *reinterpret_cast<const bf16x8*>(wa0);
            bf16x8 a1 = *reinterpret_cast<const bf16x8*>(wa1);
            gather(o0, o1);
            bf16x8 b = pack();
            o0 = *reinterpret_cast<const int4*>(kp + min(8, last));
            o1 = *reinterpret_cast<const int4*>(kp + min(8, last) + 4);
            for (int kk = 0; kk < A.kh; kk += 8) {
                const int kn = min(kk + 8, last);
                const bf16x8 a0n = *reinterpret_cast<const bf16x8*>(wa0 + kn);
                const bf16x8 a1n = *reinterpret_cast<const bf16x8*>(wa1 + kn);
                gather(o0, o1);
                const int kn2 = min(kk + 16, last);
                o0 = *reinterpret_cast<const int4*>(kp + kn2);
                o1 = *reinterpret_cast<const int4*>(kp + kn2 + 4);
                __builtin_amdgcn_sched_barrier(0);
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b, acc1, 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                a0 = a0n;
                a1 = a1n;
                b = pack();
            }
        }

        // every wave is done with the slice: the next tile's copy goes out before this tile's
        // stores (see the wait at the top)
        if (!dbuf) {
            lds_barrier();
            if (item + 1 < nitems) {
                nxt = decode(item + 1);
                copy_slice(nxt, xs, NW);
            }
        }

        // ---- epilogue: accumulator v of lane l holds channel 8*(v/4) + 4*(l/32) + v%4 (+32
        // for acc1) and pixel l%32, its bias included
        // NHWC y: channel gi*Kg + m of pixel p at (n*howo + p)*K + gi*Kg + m, the 4 channels
        // of each v/4 group adjacent (one 16- or 8-byte store when Kg % 4 == 0)
        const bool pok = p < howo;
        const __amdgpu_buffer_rsrc_t ry = make_rsrc(A.y, A.y_bytes);
        if (A.y_nhwc) {
            const uint32_t pbase = ((uint32_t)tl.n * (uint32_t)howo + (uint32_t)p) * (uint32_t)A.K +
                                   (uint32_t)(gi * A.Kg);
            if ((A.Kg & 3) == 0) {
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const int m = m0 + 8 * v4 + 4 * lrow;
                    const int v = 4 * v4;
                    store_out4<TOut>(ry, pbase + (uint32_t)m, pok & (m < A.Kg), acc0[v],
                                     acc0[v + 1], acc0[v + 2], acc0[v + 3]);
                    store_out4<TOut>(ry, pbase + (uint32_t)(m + 32), pok & (m + 32 < A.Kg), acc1[v],
                                     acc1[v + 1], acc1[v + 2], acc1[v + 3]);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = m0 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                    store_out<TOut>(ry, pbase + (uint32_t)m, pok & (m < A.Kg), acc0[v]);
                    store_out<TOut>(ry, pbase + (uint32_t)(m + 32), pok & (m + 32 < A.Kg), acc1[v]);
                }
            }
        } else if (sizeof(TOut) == 2 && (howo & 1) == 0) {
            // NCHW bf16, pixels in pairs: lanes 2i and 2i+1 hold pixels p, p+1 (p even) of the
            // same channels; for each pair of channels (v, v+1) they swap one value, after which
            // the even lane holds channel v and the odd lane channel v+1 for both pixels, and
            // each stores them with one 4-byte store (instead of two 2-byte ones).  An even
            // plane size keeps every pair inside one plane and aligned.  (For fp32 output the
            // same pairing measured slower than single 4-byte stores: cfg4 101 vs 87 us.)
            const bool odd = lane & 1;
            const int pe = p & ~1;
            const bool pok2 = pe < howo;
            const uint32_t ybase = (uint32_t)(tl.n * A.K + gi * A.Kg) * (uint32_t)howo + (uint32_t)pe;
            if (m0 + 64 <= A.Kg) {
                // all 64 channels exist: one byte offset per lane, plus a wave-uniform step per
                // store (a lane past the plane starts in the out-of-range half and stays there)
                const uint32_t lb =
                    pok2 ? (ybase + (uint32_t)(m0 + 4 * lrow + (odd ? 1 : 0)) * (uint32_t)howo) * 2u : OOB_OFF;
                const __amdgpu_buffer_rsrc_t ry2 = make_rsrc(A.y, A.y_bytes);
#pragma unroll
                for (int v = 0; v < 16; v += 2) {
                    const uint32_t c0 = (uint32_t)(8 * (v >> 2) + (v & 3)) * (uint32_t)howo * 2u;
                    const uint32_t c1 = c0 + 32u * (uint32_t)howo * 2u;
                    {
                        const float fa = acc0[v], fb = acc0[v + 1];
                        const float r = swap_adjacent_lanes(odd ? fa : fb);
                        __builtin_amdgcn_raw_buffer_store_b32(
                            __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{odd ? r : fa, odd ? fb : r}, bf16x2)),
                            ry2, lb + c0, 0, 0);
                    }
                    {
                        const float fa = acc1[v], fb = acc1[v + 1];
                        const float r = swap_adjacent_lanes(odd ? fa : fb);
                        __builtin_amdgcn_raw_buffer_store_b32(
                            __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{odd ? r : fa, odd ? fb : r}, bf16x2)),
                            ry2, lb + c1, 0, 0);
                    }
                }
            } else
#pragma unroll
            for (int v = 0; v < 16; v += 2) {
                const int mA = m0 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                const int m = odd ? mA + 1 : mA;
                {
                    const float fa = acc0[v], fb = acc0[v + 1];
                    const float r = swap_adjacent_lanes(odd ? fa : fb);
                    store_out2<TOut>(ry, ybase + (uint32_t)m * (uint32_t)howo, pok2 & (m < A.Kg), odd ? r : fa,
                                     odd ? fb : r);
                }
                {
                    const float fa = acc1[v], fb = acc1[v + 1];
                    const float r = swap_adjacent_lanes(odd ? fa : fb);
                    store_out2<TOut>(ry, ybase + (uint32_t)(m + 32) * (uint32_t)howo, pok2 & (m + 32 < A.Kg),
                                     odd ? r : fa, odd ? fb : r);
                }
            }
        } else if (sizeof(TOut) == 4 && m0 + 64 <= A.Kg) {
            // NCHW fp32 with all 64 channels: one byte offset per lane plus a wave-uniform step
            // per store (one add instead of a bounds test and an address per store; a lane past
            // the plane starts in the out-of-range half and stays there)
            const uint32_t lb = pok ? ((uint32_t)(tl.n * A.K + gi * A.Kg + m0 + 4 * lrow) * (uint32_t)howo +
                                       (uint32_t)p) * 4u
                                    : OOB_OFF;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const uint32_t c0 = (uint32_t)(8 * (v >> 2) + (v & 3)) * (uint32_t)howo * 4u;
                const uint32_t c1 = c0 + 32u * (uint32_t)howo * 4u;
                // (through float temporaries: this compiler turns a bit cast of an element of a
                // 16-wide vector into element 0)
                const float f0 = acc0[v], f1 = acc1[v];
                st_f32(ry, lb + c0, f0);
                st_f32(ry, lb + c1, f1);
            }
        } else {
            const uint32_t ybase = (uint32_t)(tl.n * A.K + gi * A.Kg) * (uint32_t)howo + (uint32_t)p;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + 8 * (v >> 2) + 4 * lrow + (v & 3);
                store_out<TOut>(ry, ybase + (uint32_t)m * (uint32_t)howo, pok & (m < A.Kg), acc0[v]);
                store_out<TOut>(ry, ybase + (uint32_t)(m + 32) * (uint32_t)howo, pok & (m + 32 < A.Kg),
                                acc1[v]);
            }
        }
        // buffer store instructions this wave just issued (one per call above)
        stores_out = A.y_nhwc ? ((A.Kg & 3) == 0 ? 8 : 32) : (sizeof(TOut) == 2 && (howo & 1) == 0 ? 16 : 32);
    }
}

SlicePlan slice_plan(int64_t Cg, int64_t R, int64_t S, int64_t Ho, int64_t Wo, int sh, int sw, int dh, int dw,
                     int xdt, int nw, int64_t W, int pw, bool pk, bool db) {
    SlicePlan sp{};
    const int64_t SLICE_NPX = 32 * nw;
    const int64_t es = xdt == CONV2D_BF16 ? 2 : 4;
    const int64_t step = xdt == CONV2D_BF16 ? 8 : 4;
    const int64_t kred = Cg * R * S;
    if (kred > SLICE_MAX_KRED) return sp;
    int64_t rows = (SLICE_NPX + Wo - 2) / Wo + 1;  // output rows a tile's consecutive pixels can touch
    if (rows > Ho) rows = Ho;
    const int64_t ph_max = (rows - 1) * sh + (R - 1) * dh + 1;
    // packed rows: a lane reads 5 words from column j0 = ow*sw + shift, so the line must hold
    // (Wo - 1)*sw + shift + 10 columns
    const int64_t shift = pw & 1;
    if (pk && xdt == CONV2D_BF16 && dw == 1 && S <= 8 && W > 0 && W % 2 == 0 &&
        (Wo - 1) * sw + shift + 10 <= SLICE_LP) {
        const int64_t steps = (Cg * R + 1) / 2;
        const int64_t kh = steps * 8;
        const int64_t wbytes = SLICE_BM * (2 * kh + 8) * 2;
        const int64_t kbytes = 2 * kh * 4;
        const int64_t xbytes = Cg * ph_max * (SLICE_LP / 2) * 4;
        // two slice buffers when they fit beside the filters (two blocks per CU either way)
        const int nbuf = wbytes + kbytes + 2 * xbytes <= SLICE_MAX_LDS ? 2 : 1;
        const int64_t total = wbytes + kbytes + nbuf * xbytes;
        if (total <= SLICE_MAX_LDS) {
            sp.ok = true;
            sp.pk = true;
            sp.nbuf = nbuf;
            sp.xwords = (int32_t)(xbytes / 4);
            sp.nw = nw;
            sp.kh = (int32_t)kh;
            sp.ph_max = (int32_t)ph_max;
            sp.pwp = (int32_t)((Wo - 1) * sw + shift + 10);
            sp.pk_shift = (int32_t)shift;
            sp.lds_k_off = (int32_t)wbytes;
            sp.lds_x_off = (int32_t)(wbytes + kbytes);
            sp.lds_bytes = (int32_t)total;
            return sp;
        }
    }
    const int64_t kh = (kred + 2 * step - 1) / (2 * step) * step;
    const int64_t wbytes = SLICE_BM * (2 * kh + step) * es;
    const int64_t kbytes = 2 * kh * 4;
    const int64_t pwp = (Wo - 1) * sw + (S - 1) * dw + 1;
    if (pwp > SLICE_LP) return sp;  // one column per thread
    const int64_t xbytes = Cg * ph_max * SLICE_LP * 4;
    // fp32 with many tiles: two slice buffers, one block per CU, when both fit beside the
    // filters (the next tile's copy then overlaps this tile's MFMAs: cfg4 9 % faster than
    // one buffer and two blocks per CU, whose copies and MFMAs did not overlap)
    const bool two = db && es == 4 && wbytes + kbytes + 2 * xbytes <= SLICE_MAX_LDS_1;
    const int64_t total = wbytes + kbytes + (two ? 2 : 1) * xbytes;
    if (total > (two ? SLICE_MAX_LDS_1 : SLICE_MAX_LDS)) return sp;
    sp.ok = true;
    sp.nw = nw;
    sp.nbuf = two ? 2 : 1;
    sp.xwords = (int32_t)(xbytes / 4);
    sp.kh = (int32_t)kh;
    sp.ph_max = (int32_t)ph_max;
    sp.pwp = (int32_t)pwp;
    sp.lds_k_off = (int32_t)wbytes;
    sp.lds_x_off = (int32_t)(wbytes + kbytes);
    sp.lds_bytes = (int32_t)total;
    return sp;
}

template <int NW>
static void launch_slice_cfg(const SliceArgs& a, int xdt, int ydt, hipStream_t stream) {
    dim3 grid((unsigned)a.nblocks), block(64 * NW);
    if (xdt == CONV2D_F32)
        hipLaunchKernelGGL((slice_conv_kernel<float, float, NW, false>), grid, block, a.lds_bytes, stream, a);
    else if (a.pk && ydt == CONV2D_BF16)
        hipLaunchKernelGGL((slice_conv_kernel<uint16_t, uint16_t, NW, true>), grid, block, a.lds_bytes, stream, a);
    else if (a.pk)
        hipLaunchKernelGGL((slice_conv_kernel<uint16_t, float, NW, true>), grid, block, a.lds_bytes, stream, a);
    else if (ydt == CONV2D_BF16)
        hipLaunchKernelGGL((slice_conv_kernel<uint16_t, uint16_t, NW, false>), grid, block, a.lds_bytes, stream, a);
    else
        hipLaunchKernelGGL((slice_conv_kernel<uint16_t, float, NW, false>), grid, block, a.lds_bytes, stream, a);
}

hipError_t launch_slice(const SliceArgs& a, int xdt, int ydt, int nw, hipStream_t stream) {
    if (a.nblocks < 1 || a.tiles_total < 1) return hipErrorInvalidValue;
    if (nw == 4) launch_slice_cfg<4>(a, xdt, ydt, stream);
    else if (nw == 8) launch_slice_cfg<8>(a, xdt, ydt, stream);
    else if (nw == 16 && xdt == CONV2D_F32)
        hipLaunchKernelGGL((slice_conv_kernel<float, float, 16, false>), dim3((unsigned)a.nblocks), dim3(1024),
                           a.lds_bytes, stream, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace cv
