// conv2d_api.hip -- C ABI, planner, dispatcher and phase timer of the conv2d library.
//
// The planner is the library's "operation analysis" step (Sec. III-A, a
// pre-convolution routine): it validates the operation, derives the output
// size, classifies it the way the paper's operation set is described
// (pointwise, grouped, dilated, rectangular, regular; Sec. III-B), chooses the
// algorithm and GEMM tile, builds the per-reduction-index tap table used by
// both GEMM paths, and sizes the explicit path's workspace.  Its host time is
// booked once per descriptor as PRE_ANALYSIS.
//
// The timer mirrors the paper's timing tool (Sec. III-A): every phase launch
// is enclosed by a pair of HIP events on the caller's stream; elapsed time and
// call counts accumulate per phase and per algorithm; Operation Time is the
// sum of all phases and Convolution Time the sum of the in-convolution ones.
#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "conv2d_internal.h"

using namespace cv;

namespace {

constexpr int64_t kBufferLimit = 0x7fffffffLL;  // raw buffer offsets are 32-bit; keep tensors below 2 GiB

struct PhaseAcc {
    double ms[CONV2D_PH_COUNT];
    int64_t calls[CONV2D_PH_COUNT];
    int64_t fwd_calls;
    double total_ms;
    int64_t total_calls;
    bool used;
};

struct EvRec {
    int algo;
    int phase;  // -1: whole-call pair of TIMING_TOTAL
    hipEvent_t a, b;
};

struct GemmPlan {
    int kind = 0;  // 0: 32x32-MFMA tile kernels (tile config)
    int tile = TILE_64x128;
    int bm = 64, bn = 128;
    int bk = 16;   // reduction rows per stage
    int pf = 1;    // register prefetch distance (fp32 32x32 kernels)
    int nstages = 0;
    int ksplit = 1;        // split reduction (implicit path): partial sums reduced by the unpack kernel
    int split_stages = 0;  // stages per split
    int tail_tiles = 0;    // tail split (implicit path): tiles computed in pieces, see plan_tail
    int tail_pieces = 0;
    int tail_stages = 0;
};

struct ExplicitPlan {
    GemmPlan gemm;
    int64_t rows_per_chunk = 0;  // rows of the (n, ho) output grid per chunk
    int64_t chunks = 0;
    int64_t col_bytes = 0;       // per chunk
    int64_t c_bytes = 0;         // per chunk
    int status = CONV2D_OK;
};

// Winograd F(2x2, 3x3): transformed filters U [16][K][C] once per call, then chunks of tc
// tiles: transformed inputs V [16][C][tc] and GEMM results M [16][K][tc] in the workspace.
struct WinoPlan {
    bool ok = false;
    int status = CONV2D_E_UNSUPPORTED;
    int mt = 2;     // output tile edge: F(2x2, 3x3) or F(4x4, 3x3)
    int npos = 16;  // transformed positions (mt + 2)^2 = GEMMs per chunk
    int64_t tiles = 0, tc = 0, chunks = 0;
    int64_t u_bytes = 0, v_bytes = 0, m_bytes = 0;  // V and M per chunk
    GemmPlan gemm;
};

int64_t elem_size(int dt) { return dt == CONV2D_BF16 ? 2 : 4; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int64_t env_int64(const char* name, int64_t dflt) {
    const char* s = std::getenv(name);
    if (!s || !*s) return dflt;
    char* end = nullptr;
    long long v = std::strtoll(s, &end, 10);
    if (end == s) return dflt;
    return (int64_t)v;
}

// Initial timing mode: OFF unless CONV2D_TIMING = total | phases (events cost every caller
// time between kernels; the benchmark harness and the breakdown reports switch them on).
int env_timing() {
    const char* s = std::getenv("CONV2D_TIMING");
    if (!s) return CONV2D_TIMING_OFF;
    if (!std::strcmp(s, "total")) return CONV2D_TIMING_TOTAL;
    if (!std::strcmp(s, "phases")) return CONV2D_TIMING_PHASES;
    return CONV2D_TIMING_OFF;
}

// Choose the GEMM kernel and block tile.  Cost = (most tiles any CU runs) x
// (work of one tile) / (MFMA efficiency of its wave tile): with many more tiles
// than CUs the tiles are dealt out evenly, so the busiest CU sets the time.
// CONV2D_GEMM = "k32:TILE[:BK[:PF]]" overrides the choice for tuning.
// nhwc: bf16 with the channel-contiguous gather (BK 64 when C/g allows).
// dense: the B operand is a packed matrix (explicit path), where 64 x 128 tiles measured
// 10-25 % faster than 64 x 64 on every fixed workload (fp32 and bf16).
GemmPlan choose_tile(int64_t M, int64_t P, int64_t G, int64_t kred, int xdt, int64_t cg, bool nhwc = false,
                     bool dense = false) {
    const int cus = 256;
    GemmPlan best;
    double best_cost = 1e300;
    // Candidate block tiles of the 32x32-MFMA kernels, with the measured MFMA efficiency of
    // their wave tiles relative to 64x64 (fp32, MI355X); with the bf16 16-byte gather the
    // larger tiles reuse each LDS operand more and win.
    struct Cand { int tile; double eff; };
    // The 32-row tiles (four 32x32 or 32x64 wave tiles side by side) are for layers with few
    // output channels per group, where a 64-row tile would leave half or more of every MFMA
    // idle; rated below their 64-row peers so that they win only when they save tiles.
    const Cand cands_f32[] = {{TILE_64x64, 1.0}, {TILE_64x128, 1.0}, {TILE_64x256, 0.8},
                              {TILE_128x64, 0.9}, {TILE_128x128, 0.85}, {TILE_32x128, 0.9},
                              {TILE_32x256, 0.75}};
    const Cand cands_bf16[] = {{TILE_64x64, 0.7}, {TILE_64x128, 0.8}, {TILE_64x256, 0.6},
                               {TILE_128x64, 0.85}, {TILE_128x128, 1.0}, {TILE_32x128, 0.6},
                               {TILE_32x256, 0.7}};
    // bf16 tiles need two resident blocks per CU to hide their load latency: count rounds
    // of two blocks per CU (a single block per CU measured well below its share)
    const bool bfc = xdt == CONV2D_BF16;
    const int per_round = bfc && nhwc ? 2 * cus : cus;
    for (const Cand& c : bfc && nhwc ? cands_bf16 : cands_f32) {
        const TileShape ts = kTileShapes[c.tile];
        const int64_t tiles = ceil_div(M, ts.bm) * ceil_div(P, ts.bn) * G;
        const double eff = c.eff * (dense && c.tile == TILE_64x128 ? 1.25 : 1.0);
        // at most 32 output channels per group, fewer tiles than one round and a long reduction:
        // the split reduction fills the chip, so the time follows the total tile work (a 64-row
        // tile then does twice the work of a 32-row one) rather than whole rounds.  (Applied to
        // larger layers this rating picked 128 x 128 tiles with split reductions, measured up to
        // 1.8x slower than 64 x 64 without.)
        const double rounds = M <= 32 && tiles < per_round && kred >= 512 ? (double)tiles / per_round
                                                                          : (double)ceil_div(tiles, per_round);
        const double cost = rounds * ts.bm * ts.bn / eff;
        if (cost < best_cost) {
            best_cost = cost;
            best.kind = 0;
            best.tile = c.tile;
            best.bm = ts.bm;
            best.bn = ts.bn;
        }
    }
    // (64-deep bf16 stages only on 64-row tiles: a 32 x 256 tile with them holds 83 KiB of LDS)
    if (best.kind == 0) best.bk = xdt == CONV2D_BF16 ? (nhwc && cg % 64 == 0 && best.bm > 32 ? 64 : 32) : 16;
    // bf16 NHWC gather with 64-deep stages: two register sets, the loads two stages ahead
    // (1-4 % on large layers; CONV2D_BF16_PF=1 takes one set)
    if (xdt == CONV2D_BF16 && nhwc && best.bk == 64) {
        const char* e = std::getenv("CONV2D_BF16_PF");
        best.pf = e && e[0] == '1' ? 1 : 2;
    }
    // fp32 64x64 tiles over a long tap-major reduction: 32-deep stages with the loads two
    // stages ahead (half the barriers per MFMA; cfg2 76 -> 72-74 us, N31 71.5 -> 69.4 us on
    // MI355X; no gain at reductions of 256)
    if (xdt == CONV2D_F32 && !dense && best.tile == TILE_64x64 && kred >= 512 && cg % 32 == 0) {
        best.bk = 32;
        best.pf = 2;
    }
    const char* ov = std::getenv("CONV2D_GEMM");
    if (ov) {
        int a = 0, b = 0, c = 16;
        if (std::sscanf(ov, "k32:%d:%d:%d", &a, &b, &c) >= 1 && a >= 0 && a < TILE_COUNT) {
            const bool has_bk = std::strchr(ov + 4, ':') != nullptr;
            int bk = xdt == CONV2D_BF16 ? (nhwc && has_bk && b == 64 && cg % 64 == 0 ? 64 : 32)
                                        : (has_bk ? b : 16);
            int pf = has_bk && std::strchr(std::strchr(ov + 4, ':') + 1, ':') ? c : 1;
            if (xdt == CONV2D_BF16 || gemm32_f32_supported(a, bk, pf)) {
                best.kind = 0; best.tile = a; best.bm = kTileShapes[a].bm; best.bn = kTileShapes[a].bn;
                best.bk = bk;
                best.pf = xdt == CONV2D_BF16 ? (nhwc && bk == 64 && pf == 2 ? 2 : 1) : pf;
            }
        }
    }
    best.nstages = (int)ceil_div(kred, best.bk);
    return best;
}

hipError_t dispatch_gemm(const GemmPlan& gp, const GemmArgs& a_in, int bsrc, int epi, int xdt, int ydt,
                         int groups, hipStream_t s) {
    const GemmArgs& a = a_in;
    // (bf16: the two-stage register prefetch exists for the NHWC gather only)
    const int pf = xdt == CONV2D_BF16 && bsrc != BSRC_NHWC_TAP ? 1 : gp.pf;
    return launch_gemm(a, gp.tile, gp.bk, pf, bsrc, epi, xdt, ydt, groups, s);
}

// Workspace slots of a descriptor (one use each).
enum BufSlot {
    BUF_WS,    // explicit path: col [g][Kred][P_chunk] then the GEMM result [g][Kg][P_chunk]
    BUF_XR,    // NCHW copy of an NHWC input, or NHWC copy of an NCHW one (channel-contiguous gathers)
    BUF_YR,    // NCHW result before the NHWC reorder
    BUF_WR,    // weights in tap-major order for the implicit GEMM
    BUF_SK,    // partial sums of the split reduction
    BUF_DK,    // partial sums of the few-output-channel direct kernel's channel ranges
    BUF_WD,    // depthwise filters as [R*S][C] for the NHWC depthwise kernel
    BUF_WU,    // Winograd transformed filters
    BUF_WVM,   // Winograd V and M of one chunk
    BUF_TP,    // partial tiles of the tail split
    BUF_KTAB,  // the tap table, written on the device (no-allocation entry point only)
    BUF_COUNT
};

}  // namespace

struct conv2d_desc {
    conv2d_params prm;
    Geometry g;
    uint32_t opclass = 0;
    int auto_algo = CONV2D_ALGO_IMPLICIT_GEMM;
    bool implicit_ok = false, direct_ok = false;
    bool implicit_tap = false;  // tap-major gather (C/g a multiple of the stage depth)
    int smallk_ranges = 0;      // > 0: DIRECT runs the few-output-channel kernel with this many channel ranges
    bool direct_nhwc = false;   // DIRECT runs the NHWC depthwise kernel on NHWC x and y
    void* wd = nullptr;         // its filters as [R*S][C]
    int64_t wd_bytes = 0;
    bool implicit_slice = false;  // sliced direct MFMA kernel instead of the GEMM
    bool implicit_nhwc = false;   // bf16 GEMM gathering from an NHWC copy of x (16-byte loads)
    GemmPlan implicit;
    SlicePlan slice{};    // the sliced kernel's plan (packed rows where they apply)
    SlicePlan slice_u{};  // one word per element: the fallback when x is not 4-byte aligned
    ExplicitPlan expl;
    std::vector<KTabEntry> ktab_host;

    WinoPlan wino;

    int device = -1;
    int cus = 256;  // compute units of that device
    KTabEntry* ktab_dev = nullptr;
    // Workspaces (BufSlot), allocated on first use.  Each slot has one size per descriptor,
    // fixed by the plan, so a slot is allocated once and never resized.
    void* buf[BUF_COUNT] = {};
    int64_t buf_bytes[BUF_COUNT] = {};
    uint32_t* tc = nullptr;  // arrival counters of the tail split (zeroed once, reset by the kernel)
    // Ordering between calls: a call on another stream than the previous call's records `done`
    // on that previous stream (behind everything queued there, the previous call included) and
    // makes its own stream wait for it, so calls that share the workspaces above never overlap.
    // Calls on the same stream are ordered by the stream and record nothing.
    hipEvent_t done = nullptr;
    hipStream_t last_stream = nullptr;
    bool has_last = false;
    bool implicit_ran = false;  // an implicit conv2d_fwd made the internal copies the probes read

    int timing = CONV2D_TIMING_OFF;
    double analysis_ms = 0.0;
    PhaseAcc acc[CONV2D_ALGO_COUNT];
    int last_algo = -1;
    std::vector<hipEvent_t> free_events;
    std::vector<EvRec> pending;
};

namespace {

int validate(const conv2d_params* p, Geometry* g) {
    if (p->n < 1 || p->c < 1 || p->h < 1 || p->w < 1 || p->k < 1 || p->r < 1 || p->s < 1)
        return CONV2D_E_INVALID;
    if (p->stride_h < 1 || p->stride_w < 1 || p->dil_h < 1 || p->dil_w < 1) return CONV2D_E_INVALID;
    if (p->pad_h < 0 || p->pad_w < 0 || p->groups < 1) return CONV2D_E_INVALID;
    if (p->c % p->groups || p->k % p->groups) return CONV2D_E_INVALID;
    if (p->layout != CONV2D_NCHW && p->layout != CONV2D_NHWC) return CONV2D_E_INVALID;
    if (p->x_dtype != CONV2D_F32 && p->x_dtype != CONV2D_BF16) return CONV2D_E_INVALID;
    if (p->y_dtype != CONV2D_F32 && p->y_dtype != CONV2D_BF16) return CONV2D_E_INVALID;
    if (p->x_dtype == CONV2D_F32 && p->y_dtype == CONV2D_BF16) return CONV2D_E_UNSUPPORTED;
    // window extents: the last window start must lie inside the padded input
    const int64_t span_h = p->h + 2 * (int64_t)p->pad_h - (int64_t)p->dil_h * (p->r - 1) - 1;
    const int64_t span_w = p->w + 2 * (int64_t)p->pad_w - (int64_t)p->dil_w * (p->s - 1) - 1;
    if (span_h < 0 || span_w < 0) return CONV2D_E_SHAPE;
    Geometry& G = *g;
    G.N = p->n; G.C = p->c; G.H = p->h; G.W = p->w; G.K = p->k; G.R = p->r; G.S = p->s;
    G.sh = p->stride_h; G.sw = p->stride_w; G.ph = p->pad_h; G.pw = p->pad_w;
    G.dh = p->dil_h; G.dw = p->dil_w; G.G = p->groups;
    G.Ho = span_h / p->stride_h + 1;
    G.Wo = span_w / p->stride_w + 1;
    G.Cg = p->c / p->groups;
    G.Kg = p->k / p->groups;
    G.Kred = G.Cg * G.R * G.S;
    G.P = G.N * G.Ho * G.Wo;
    G.layout = p->layout; G.xdt = p->x_dtype; G.ydt = p->y_dtype; G.has_bias = p->has_bias ? 1 : 0;
    G.x_elems = G.N * G.C * G.H * G.W;
    G.w_elems = G.K * G.Kred;
    G.y_elems = G.N * G.K * G.Ho * G.Wo;
    return CONV2D_OK;
}

uint32_t classify(const Geometry& g) {
    uint32_t c = 0;
    if (g.R == 1 && g.S == 1) c |= OPC_POINTWISE;
    if (g.G > 1) c |= OPC_GROUPED;
    if (g.G > 1 && g.Cg == 1) c |= OPC_DEPTHWISE;
    if (g.dh > 1 || g.dw > 1) c |= OPC_DILATED;
    if (g.R != g.S) c |= OPC_RECTANGULAR;
    if (g.sh > 1 || g.sw > 1) c |= OPC_STRIDED;
    return c;
}

void build_ktab(conv2d_desc* d) {
    const Geometry& g = d->g;
    const int64_t len = ceil_div(g.Kred, KTAB_ALIGN) * KTAB_ALIGN;
    d->ktab_host.assign((size_t)len, KTabEntry{0, KTAB_DEAD, 0, 0});
    int64_t kr = 0;
    for (int64_t c = 0; c < g.Cg; ++c)
        for (int64_t r = 0; r < g.R; ++r)
            for (int64_t s = 0; s < g.S; ++s, ++kr) {
                KTabEntry& e = d->ktab_host[(size_t)kr];
                e.roff = (int32_t)(r * g.dh);
                e.soff = (int32_t)(s * g.dw);
                e.coff = (int32_t)(c * g.H * g.W + e.roff * g.W + e.soff);
                e.pad = 0;
            }
}

// Split reduction for layers with too few output tiles to fill the chip (batch 1, small
// planes, few channels) and a long reduction: split s of S runs a contiguous range of
// stages and writes fp32 partial sums, and the unpack kernel adds the S partials in split
// order (deterministic) with the bias.  Aim for two tiles per CU,
// keep at least 8 stages per split and the partials under 256 MiB.  CONV2D_KSPLIT forces S.
void plan_split(conv2d_desc* d) {
    const Geometry& g = d->g;
    GemmPlan& gp = d->implicit;
    gp.ksplit = 1;
    gp.split_stages = gp.nstages;
    const int64_t tiles = ceil_div(g.Kg, gp.bm) * ceil_div(g.P, gp.bn) * g.G;
    int64_t S = 1;
    if (tiles < 512) S = std::min<int64_t>(ceil_div(512, tiles), gp.nstages / 8);
    const int64_t force = env_int64("CONV2D_KSPLIT", 0);
    if (force > 0) S = std::min<int64_t>(force, gp.nstages);
    const int64_t part_bytes = g.G * g.Kg * g.P * 4;
    while (S > 1 && S * part_bytes > ((int64_t)256 << 20)) --S;
    if (S > 256) S = 256;
    if (S < 2 || g.G * S > 65535) return;
    const int64_t per = ceil_div(gp.nstages, S);
    gp.ksplit = (int)ceil_div(gp.nstages, per);  // every split non-empty
    gp.split_stages = (int)per;
}

// Tail split.  With one tile per block and every tile resident at once, the CUs that hold
// one tile more than the others set the time: 1568 tiles on 256 CUs run as 7 rounds of
// tile work although the average is 6.1.  When the tiles past the last multiple of the CU
// count are at most half the CUs, each of them is computed instead by q blocks of
// consecutive stages (about one extra block per CU, q <= 16, at least 2 stages each); the
// last piece of a tile to finish adds the q partials in piece order and stores the tile.
// One group and no split reduction.  CONV2D_TAIL=0 switches it off; CONV2D_TAIL=q forces q
// pieces (at least one stage each) on the tiles past the last multiple of the CU count, or on
// every tile when that count divides the tiles.
void plan_tail(conv2d_desc* d) {
    const Geometry& g = d->g;
    GemmPlan& gp = d->implicit;
    gp.tail_tiles = gp.tail_pieces = gp.tail_stages = 0;
    if (gp.ksplit > 1 || g.G != 1) return;
    const int64_t cus = 256;
    const int64_t tiles = ceil_div(g.Kg, gp.bm) * ceil_div(g.P, gp.bn);
    const int64_t full = tiles / cus;
    int64_t rem = tiles % cus;
    const int64_t force = env_int64("CONV2D_TAIL", -1);
    int64_t q = 0;
    if (force > 0) {
        if (rem == 0) rem = tiles;
        q = std::min<int64_t>(force, gp.nstages);
    } else if (force < 0 && full >= 1 && rem > 0 && rem <= cus / 2) {
        q = std::min<int64_t>(std::min<int64_t>(cus / rem, 16), gp.nstages / 2);
    }
    if (q < 2 || tiles + rem * (q - 1) > 0x7fffffffLL) return;
    const int64_t per = ceil_div(gp.nstages, q);
    const int64_t pieces = ceil_div(gp.nstages, per);  // every piece non-empty
    if (pieces < 2 || rem * pieces * gp.bm * gp.bn * 4 >= ((int64_t)1 << 31)) return;
    gp.tail_tiles = (int)rem;
    gp.tail_pieces = (int)pieces;
    gp.tail_stages = (int)per;
}

int64_t tail_part_bytes(const GemmPlan& gp) {
    return (int64_t)gp.tail_tiles * gp.tail_pieces * gp.bm * gp.bn * 4;
}

// Winograd F(2x2, 3x3) or F(4x4, 3x3) runs 3x3 filters at stride 1 and dilation 1 with one
// group in fp32.  Tiles go in chunks whose V and M fit CONV2D_WORKSPACE_LIMIT_BYTES (default
// 1 GiB) and the 2 GiB buffer limit.  F(4x4) does 2.25x fewer multiplications than F(2x2) and
// moves 1.8x fewer transformed values per output; measured 1.2-1.9x faster on MI355X for output
// planes of 14x14 and larger (C, K = 64 .. 1024), while on 7x7 planes the padding of the last
// tile row and column costs more than that (F(2x2) 53 us, F(4x4) 74 us for 8 x 512 -> 512).
// CONV2D_WINO_TILE = 2 / 4 forces the output tile.
int wino_auto_tile(const Geometry& g) { return std::min(g.Ho, g.Wo) >= 8 ? 4 : 2; }

void plan_winograd(conv2d_desc* d) {
    const Geometry& g = d->g;
    WinoPlan& p = d->wino;
    p = WinoPlan{};
    // bf16 (x and w; y bf16 or fp32): F(2x2) only, with U and V rounded to bf16 and fp32 GEMM
    // sums (F(4x4)'s larger transform constants put bf16 rounding past the 1e-2 gate in a CPU
    // study: 2e-2 at C = 16, against 1.8e-3 for F(2x2)); V is laid out [16][tiles][C] from the
    // NHWC copy of x so that the GEMM reads 8 channels per 16-byte load (C a multiple of 8)
    const bool bf = g.xdt == CONV2D_BF16;
    if (g.R != 3 || g.S != 3 || g.sh != 1 || g.sw != 1 || g.dh != 1 || g.dw != 1 || g.G != 1 ||
        (g.xdt == CONV2D_F32 && g.ydt != CONV2D_F32) || (bf && g.C % 8 != 0) ||
        g.x_elems * elem_size(g.xdt) > kBufferLimit || g.y_elems * elem_size(g.ydt) > kBufferLimit)
        return;
    const int64_t es = elem_size(g.xdt);  // bytes of U and V elements
    const int64_t force = env_int64("CONV2D_WINO_TILE", 0);
    p.mt = bf ? 2 : force == 2 || force == 4 ? (int)force : wino_auto_tile(g);
    p.npos = (p.mt + 2) * (p.mt + 2);
    const int64_t np = p.npos;
    p.u_bytes = np * g.K * g.C * es;
    if (p.u_bytes > kBufferLimit) return;
    p.tiles = g.N * ceil_div(g.Ho, p.mt) * ceil_div(g.Wo, p.mt);
    int64_t cap = env_int64("CONV2D_WORKSPACE_LIMIT_BYTES", (int64_t)1 << 30);
    if (cap < 0) cap = 0;
    int64_t tc = cap / (np * (g.C * es + g.K * 4));
    tc = std::min<int64_t>(tc, kBufferLimit / (np * g.C * es));
    tc = std::min<int64_t>(tc, kBufferLimit / (np * g.K * 4));
    tc = std::min<int64_t>(tc, p.tiles);
    if (tc < 1) {
        p.status = CONV2D_E_ALLOC;
        return;
    }
    p.tc = tc;
    p.chunks = ceil_div(p.tiles, tc);
    p.v_bytes = np * g.C * tc * es;
    p.m_bytes = np * g.K * tc * 4;
    // 64 x 128 tiles: measured fastest for these GEMMs (dense operands, reductions of a few
    // hundred channels) on MI355X, ahead of 64 x 64, 128 x 128 and 64 x 256; bf16 takes the
    // planner's bf16 choice for 16-byte operand loads
    p.gemm = choose_tile(g.K, tc, np, g.C, g.xdt, g.C, bf);
    if (!bf && !std::getenv("CONV2D_GEMM")) {
        p.gemm.tile = TILE_64x128;
        p.gemm.bm = kTileShapes[TILE_64x128].bm;
        p.gemm.bn = kTileShapes[TILE_64x128].bn;
        p.gemm.bk = 16;
        p.gemm.pf = 1;
        p.gemm.nstages = (int)ceil_div(g.C, 16);
    }
    p.ok = true;
    p.status = CONV2D_OK;
}

void plan_explicit(conv2d_desc* d) {
    const Geometry& g = d->g;
    ExplicitPlan& e = d->expl;
    const int64_t xs = elem_size(g.xdt);
    const int64_t row_col = g.Wo * g.G * g.Kred * xs;  // col bytes of one output row (all groups)
    const int64_t row_c = g.Wo * g.G * g.Kg * 4;        // GEMM result bytes of one output row
    int64_t cap = env_int64("CONV2D_WORKSPACE_LIMIT_BYTES", (int64_t)1 << 30);
    if (cap < 0) cap = 0;
    const int64_t total_rows = g.N * g.Ho;
    int64_t rows = cap / (row_col + row_c);
    rows = std::min<int64_t>(rows, kBufferLimit / row_col);
    rows = std::min<int64_t>(rows, kBufferLimit / row_c);
    rows = std::min<int64_t>(rows, total_rows);
    if (rows < 1) {
        e.status = CONV2D_E_ALLOC;
        e.rows_per_chunk = 0;
        e.chunks = 0;
        return;
    }
    e.status = CONV2D_OK;
    e.rows_per_chunk = rows;
    e.chunks = ceil_div(total_rows, rows);
    e.col_bytes = rows * row_col;
    e.c_bytes = rows * row_c;
    e.gemm = choose_tile(g.Kg, rows * g.Wo, g.G, g.Kred, g.xdt, g.Cg, false, true);
}

// ------------------------------------------------------------------ events
hipError_t get_event(conv2d_desc* d, hipEvent_t* ev) {
    if (!d->free_events.empty()) {
        *ev = d->free_events.back();
        d->free_events.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(ev);
}

// Fold the recorded event pairs into the per-algorithm totals.  block = false folds only the
// pairs whose end event has completed (hipEventQuery) and keeps the rest pending, so a call
// never waits for the GPU; block = true waits for every pair.
int harvest(conv2d_desc* d, bool block = true) {
    int st = CONV2D_OK;
    std::vector<EvRec> keep;
    for (const EvRec& r : d->pending) {
        if (!block) {
            const hipError_t q = hipEventQuery(r.b);
            if (q == hipErrorNotReady) {
                keep.push_back(r);
                continue;
            }
        }
        float ms = 0.0f;
        if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
            st = CONV2D_E_HIP;
        } else {
            PhaseAcc& a = d->acc[r.algo];
            if (r.phase < 0) {
                a.total_ms += ms;
                a.total_calls += 1;
            } else {
                a.ms[r.phase] += ms;
                a.calls[r.phase] += 1;
            }
        }
        d->free_events.push_back(r.a);
        d->free_events.push_back(r.b);
    }
    d->pending.swap(keep);
    return st;
}

// Encloses one phase launch (PHASES mode) or a whole call (TOTAL mode).
struct Scope {
    conv2d_desc* d;
    int algo, phase;
    hipStream_t s;
    hipEvent_t a = nullptr;
    bool active;
    Scope(conv2d_desc* d_, int algo_, int phase_, hipStream_t s_, bool active_)
        : d(d_), algo(algo_), phase(phase_), s(s_), active(active_) {}
    ~Scope() {
        if (a) d->free_events.push_back(a);  // an error path left the pair open
    }
    int begin() {
        if (!active) return CONV2D_OK;
        if (get_event(d, &a) != hipSuccess || hipEventRecord(a, s) != hipSuccess) return CONV2D_E_HIP;
        return CONV2D_OK;
    }
    int end() {
        if (!active || !a) return CONV2D_OK;
        hipEvent_t b = nullptr;
        if (get_event(d, &b) != hipSuccess || hipEventRecord(b, s) != hipSuccess) return CONV2D_E_HIP;
        d->pending.push_back(EvRec{algo, phase, a, b});
        a = nullptr;
        return CONV2D_OK;
    }
};

// A call on stream s waits for the previous call on this descriptor when that one went to
// another stream (see conv2d_desc::done).  last_stream must still exist.
int order_after_last(conv2d_desc* d, hipStream_t s) {
    if (d->has_last && s != d->last_stream) {
        if (hipEventRecord(d->done, d->last_stream) != hipSuccess || hipStreamWaitEvent(s, d->done, 0) != hipSuccess)
            return CONV2D_E_HIP;
    }
    d->last_stream = s;
    d->has_last = true;
    return CONV2D_OK;
}

// ------------------------------------------------------------------ device resources
int ensure_device(conv2d_desc* d, hipStream_t s) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CONV2D_E_HIP;
    if (d->device >= 0 && d->device != dev) return CONV2D_E_UNSUPPORTED;
    if (d->device < 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
            d->cus = cus;
        if (!d->done && hipEventCreateWithFlags(&d->done, hipEventDisableTiming) != hipSuccess) {
            d->done = nullptr;
            return CONV2D_E_HIP;
        }
        const size_t bytes = d->ktab_host.size() * sizeof(KTabEntry);
        if (hipMalloc(&d->ktab_dev, bytes) != hipSuccess) {
            d->ktab_dev = nullptr;
            return CONV2D_E_ALLOC;
        }
        if (hipMemcpyAsync(d->ktab_dev, d->ktab_host.data(), bytes, hipMemcpyHostToDevice, s) != hipSuccess)
            return CONV2D_E_HIP;
        d->device = dev;
    }
    return CONV2D_OK;
}

// Where one call's workspaces come from.  Normally the descriptor's own buffers, allocated
// on first use; a slot that ever needed more would first wait for the descriptor's previous
// call (its `done` event: the buffer may still be read by it), never for the whole device.
// For the no-allocation entry point, consecutive 256-byte aligned pieces of the static scratch
// array (the tail split's counters sit in its own fixed region, see there).
struct Ws {
    conv2d_desc* d;
    char* scratch = nullptr;  // non-null: carve from here
    int64_t cap = 0, used = 0;
    uint32_t* counters = nullptr;  // scratch mode: tail-split counters (kept at zero between launches)
    int64_t counter_cap = 0;
    int cus = 256;  // compute units of the device the call runs on

    int get(int slot, int64_t need, void** out) {
        if (need <= 0) need = 1;
        if (scratch) {
            const int64_t at = (used + 255) / 256 * 256;
            if (at + need > cap) return CONV2D_E_SCRATCH;
            *out = scratch + at;
            used = at + need;
            return CONV2D_OK;
        }
        if (d->buf[slot] && d->buf_bytes[slot] >= need) {
            *out = d->buf[slot];
            return CONV2D_OK;
        }
        if (d->buf[slot]) {
            // the buffer may still be read by queued work of this descriptor, all of which sits
            // on last_stream
            if (d->has_last && (hipEventRecord(d->done, d->last_stream) != hipSuccess ||
                                hipEventSynchronize(d->done) != hipSuccess))
                return CONV2D_E_HIP;
            hipFree(d->buf[slot]);
            d->buf[slot] = nullptr;
            d->buf_bytes[slot] = 0;
        }
        if (hipMalloc(&d->buf[slot], (size_t)need) != hipSuccess) {
            d->buf[slot] = nullptr;
            return CONV2D_E_ALLOC;
        }
        d->buf_bytes[slot] = need;
        *out = d->buf[slot];
        return CONV2D_OK;
    }
    // arrival counters of the tail split, zero at every launch start
    int tail_counters(int64_t n, hipStream_t s, uint32_t** out) {
        if (scratch) {
            if (n > counter_cap) return CONV2D_E_SCRATCH;
            *out = counters;
            return CONV2D_OK;
        }
        if (!d->tc) {
            if (hipMalloc(&d->tc, (size_t)n * sizeof(uint32_t)) != hipSuccess) {
                d->tc = nullptr;
                return CONV2D_E_ALLOC;
            }
            if (launch_fill_u32(d->tc, n, 0u, s) != hipSuccess) return CONV2D_E_HIP;
        }
        *out = d->tc;
        return CONV2D_OK;
    }
    // the tap table: uploaded once by ensure_device, or written into the scratch by a kernel
    int table(hipStream_t s, const KTabEntry** out) {
        if (!scratch) {
            *out = d->ktab_dev;
            return CONV2D_OK;
        }
        const int64_t len = (int64_t)d->ktab_host.size();
        void* p = nullptr;
        const int st = get(BUF_KTAB, len * (int64_t)sizeof(KTabEntry), &p);
        if (st != CONV2D_OK) return st;
        const Geometry& g = d->g;
        if (launch_ktab_fill(static_cast<KTabEntry*>(p), len, g.Kred, g.Cg, g.R, g.S, g.H, g.W, g.dh, g.dw, s) !=
            hipSuccess)
            return CONV2D_E_HIP;
        *out = static_cast<const KTabEntry*>(p);
        return CONV2D_OK;
    }
};

#define CV_TRY(expr)                 \
    do {                             \
        int _st = (expr);            \
        if (_st != CONV2D_OK) return _st; \
    } while (0)

#define CV_HIP(expr)                                   \
    do {                                               \
        if ((expr) != hipSuccess) return CONV2D_E_HIP; \
    } while (0)

// ------------------------------------------------------------------ algorithms (NCHW tensors)
// The sliced kernel's plan for this x: the packed rows copy input pairs with 4-byte loads, so
// an x that is not 4-byte aligned takes the element-wise layout, or (when that does not fit
// LDS) no sliced plan at all (nullptr: the tiled GEMM runs instead).
const SlicePlan* slice_for(const conv2d_desc* d, const void* x) {
    if (!d->slice.pk || ((uintptr_t)x & 3u) == 0) return &d->slice;
    return d->slice_u.ok ? &d->slice_u : nullptr;
}

int run_slice(conv2d_desc* d, const SlicePlan& sp, const Ws& ws, const void* x, const void* w, const float* bias,
              void* y, hipStream_t s, bool ph, bool probe) {
    const Geometry& g = d->g;
    SliceArgs a{};
    a.x = x;
    a.x_bytes = (uint32_t)(g.x_elems * elem_size(g.xdt));
    a.w = w;
    a.w_bytes = (uint32_t)(g.w_elems * elem_size(g.xdt));
    a.bias = g.has_bias ? bias : nullptr;
    a.y = y;
    a.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
    a.C = (int32_t)g.C; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.K = (int32_t)g.K;
    a.Ho = (int32_t)g.Ho; a.Wo = (int32_t)g.Wo; a.R = (int32_t)g.R; a.S = (int32_t)g.S;
    a.sh = g.sh; a.sw = g.sw; a.ph = g.ph; a.pw = g.pw; a.dh = g.dh; a.dw = g.dw;
    a.Cg = (int32_t)g.Cg; a.Kg = (int32_t)g.Kg;
    a.kred = (int32_t)g.Kred;
    a.kh = sp.kh;
    a.ph_max = sp.ph_max;
    a.pwp = sp.pwp;
    a.N = (int32_t)g.N;
    a.tiles_px = (int32_t)ceil_div(g.Ho * g.Wo, 32 * sp.nw);
    a.grid_m = (int32_t)ceil_div(g.Kg, 64);
    a.tiles_total = (int32_t)(g.G * a.grid_m * g.N * a.tiles_px);
    const int per_cu = std::max(1, std::min(16 / sp.nw, (int)((160 << 10) / sp.lds_bytes)));
    a.nblocks = std::min(a.tiles_total, ws.cus * per_cu);
    // Persistent blocks take whole rounds of tiles; a last, partial round would leave most
    // blocks idle while a few compute whole tiles (cfg4: 1568 tiles on 512 blocks, 3.06
    // rounds run as 4), so its tiles are split by wave groups over the idle blocks.
    a.tail_start = a.tiles_total;
    a.tail_q = 0;
    {
        const int nb = a.nblocks, full = a.tiles_total / nb, rem = a.tiles_total % nb;
        int q = 1;
        while (q * 2 <= sp.nw && rem * q * 2 <= nb) q *= 2;
        if (full >= 1 && rem > 0 && q >= 2) {
            a.tail_start = full * nb;
            a.tail_q = q;
        }
    }
    a.lds_k_off = sp.lds_k_off;
    a.lds_x_off = sp.lds_x_off;
    a.lds_bytes = sp.lds_bytes;
    a.loader_only = probe ? 1 : 0;
    a.y_nhwc = g.layout == CONV2D_NHWC ? 1 : 0;
    a.pk = sp.pk ? 1 : 0;
    a.pk_shift = sp.pk_shift;
    a.nbuf = sp.nbuf;
    a.xwords = sp.xwords;
    // fp32 lines by 16-byte copies when every 4-word group of a line is wholly inside or
    // outside the image and the shifted line still fits
    // (CONV2D_SLICE_X1=1 keeps the 4-byte copies: tests run both)
    const char* x1 = std::getenv("CONV2D_SLICE_X1");
    a.xshift = (4 - a.pw % 4) % 4;
    a.x4 = g.xdt == CONV2D_F32 && !sp.pk && a.W % 4 == 0 && ((uintptr_t)x & 15) == 0 &&
           sp.pwp + a.xshift <= 256 && !(x1 && x1[0] == '1');
    if (!a.x4) a.xshift = 0;
    a.fd_pergz = make_fastdiv((uint32_t)(a.N * a.tiles_px));
    a.fd_tpx = make_fastdiv((uint32_t)a.tiles_px);
    a.fd_gm = make_fastdiv((uint32_t)a.grid_m);
    a.fd_wo = make_fastdiv((uint32_t)a.Wo);
    a.fd_kw = make_fastdiv((uint32_t)(2 * a.kh));
    Scope sc(d, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_PH_IN_MICROKERNEL, s, ph);
    CV_TRY(sc.begin());
    CV_HIP(launch_slice(a, g.xdt, g.ydt, sp.nw, s));
    return sc.end();
}

// An NHWC y is written by the sliced kernel, or by the GEMM's own epilogue or the unpack of a
// split reduction's partials when the GEMM gathers from NHWC x: no NCHW result, no
// post-convolution reordering.
bool implicit_writes_nhwc(const conv2d_desc* d) {
    return d->g.layout == CONV2D_NHWC && (d->implicit_slice || d->implicit_nhwc);
}

// probe: PROBE_LOADER runs only the microkernel's loader (the pack probe) and writes nothing;
// PROBE_KERNEL runs only the microkernel launch (no filter repack, no split-reduction unpack).
// Both read the internal copies that the last call made (tap-major weights).
enum { PROBE_NONE = 0, PROBE_LOADER = 1, PROBE_KERNEL = 2 };
int run_implicit(conv2d_desc* d, Ws& ws, const void* x, const void* w, const float* bias, void* y, hipStream_t s,
                 bool ph, int probe = PROBE_NONE) {
    const Geometry& g = d->g;
    const GemmPlan& gp = d->implicit;
    if (d->implicit_slice) {
        const SlicePlan* sp = slice_for(d, x);
        if (sp) return run_slice(d, *sp, ws, x, w, bias, y, s, ph, probe == PROBE_LOADER);
        // misaligned x without an element-wise plan: the tiled GEMM below, with its NCHW gathers
        if (d->implicit_nhwc) return CONV2D_E_UNSUPPORTED;
    }
    if ((d->implicit_tap || d->implicit_nhwc) && g.R * g.S > 1 && probe) {
        if (!d->buf[BUF_WR]) return CONV2D_E_NO_DATA;
        w = d->buf[BUF_WR];
    } else if ((d->implicit_tap || d->implicit_nhwc) && g.R * g.S > 1) {
        // pre-convolution reordering of the filters into the tap-major reduction order
        const int64_t wb = g.w_elems * elem_size(g.xdt);
        void* wr = nullptr;
        CV_TRY(ws.get(BUF_WR, wb, &wr));
        Scope sc(d, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_PH_PRE_REORDER, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(launch_repack_tap_major(w, wr, g.K, g.Cg, g.R * g.S, (int)elem_size(g.xdt), s));
        CV_TRY(sc.end());
        w = wr;
    }
    GemmArgs a{};
    a.a = w;
    a.a_bytes = (uint32_t)(g.w_elems * elem_size(g.xdt));
    a.lda = (int32_t)g.Kred;
    a.a_gstride = g.Kg * g.Kred;
    a.b = x;
    a.b_bytes = (uint32_t)(g.x_elems * elem_size(g.xdt));
    a.b_gstride = g.Cg * g.H * g.W;
    a.ktab = nullptr;
    if (!(d->implicit_tap || d->implicit_nhwc)) CV_TRY(ws.table(s, &a.ktab));
    a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.Ho = (int32_t)g.Ho; a.Wo = (int32_t)g.Wo;
    a.sh = g.sh; a.sw = g.sw; a.ph = g.ph; a.pw = g.pw;
    a.dh = g.dh; a.dw = g.dw; a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.RS = (int32_t)(g.R * g.S);
    a.Cg = (int32_t)g.Cg;
    a.HW = (int32_t)(g.H * g.W);
    a.Cx = (int32_t)g.C;
    a.x_nstride = g.C * g.H * g.W;
    a.M = (int32_t)g.Kg;
    a.Kred = (int32_t)g.Kred;
    a.P = (int32_t)g.P;
    a.nstages = gp.nstages;
    a.grid_m = (int32_t)ceil_div(g.Kg, gp.bm);
    a.grid_p = (int32_t)ceil_div(g.P, gp.bn);
    a.y = y;
    a.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
    a.bias = g.has_bias ? bias : nullptr;
    a.y_nstride = g.K * g.Ho * g.Wo;
    a.HoWo = (int32_t)(g.Ho * g.Wo);
    const int bsrc = d->implicit_nhwc ? BSRC_NHWC_TAP : d->implicit_tap ? BSRC_IMPLICIT_TAP : BSRC_IMPLICIT_NCHW;
    a.loader_only = probe == PROBE_LOADER ? 1 : 0;
    if (gp.ksplit <= 1) {
        if (gp.tail_tiles > 0) {
            void* tp = nullptr;
            CV_TRY(ws.get(BUF_TP, tail_part_bytes(gp), &tp));
            CV_TRY(ws.tail_counters(gp.tail_tiles, s, &a.tail_count));
            a.tail_tiles = gp.tail_tiles;
            a.tail_pieces = gp.tail_pieces;
            a.tail_stages = gp.tail_stages;
            a.tail_part = static_cast<float*>(tp);
        }
        const bool y_nhwc = implicit_writes_nhwc(d);
        if (y_nhwc) a.ldc = (int32_t)g.K;
        Scope sc(d, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_PH_IN_MICROKERNEL, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(dispatch_gemm(gp, a, bsrc, y_nhwc ? EPI_NHWC : EPI_NCHW, g.xdt, g.ydt, (int)g.G, s));
        return sc.end();
    }
    // split reduction: partial sums [split][g][m][p] in fp32, then the unpack kernel adds them
    const int64_t slice = g.G * g.Kg * g.P;  // elements of one split's partials
    void* sk = nullptr;
    CV_TRY(ws.get(BUF_SK, gp.ksplit * slice * 4, &sk));
    a.y = sk;
    a.y_bytes = (uint32_t)(gp.ksplit * slice * 4);
    a.ldc = (int32_t)g.P;
    a.c_gstride = g.Kg * g.P;
    a.ksplit = gp.ksplit;
    a.split_stages = gp.split_stages;
    a.c_sstride = slice;
    {
        Scope sc(d, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_PH_IN_MICROKERNEL, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(dispatch_gemm(gp, a, bsrc, EPI_DENSE, g.xdt, CONV2D_F32, (int)g.G, s));
        CV_TRY(sc.end());
    }
    if (probe) return CONV2D_OK;
    UnpackArgs u{};
    u.c = static_cast<const float*>(sk);
    u.y = y;
    u.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
    u.bias = g.has_bias ? bias : nullptr;
    u.Kg = (int32_t)g.Kg;
    u.pc = (int32_t)g.P;
    u.HoWo = (int32_t)(g.Ho * g.Wo);
    u.p_begin = 0;
    u.y_nstride = g.K * g.Ho * g.Wo;
    u.splits = gp.ksplit;
    u.split_stride = slice;
    u.nhwc = implicit_writes_nhwc(d) ? 1 : 0;
    Scope sc(d, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_PH_IN_UNPACKING, s, ph);
    CV_TRY(sc.begin());
    CV_HIP(launch_unpack(u, g.ydt, (int)g.G, s));
    return sc.end();
}

int run_winograd(conv2d_desc* d, Ws& ws, const void* x, const void* w, const float* bias, void* y, hipStream_t s,
                 bool ph) {
    const Geometry& g = d->g;
    const WinoPlan& p = d->wino;
    if (!p.ok) return p.status;
    void* wu = nullptr;
    void* wvm = nullptr;
    CV_TRY(ws.get(BUF_WU, p.u_bytes, &wu));
    CV_TRY(ws.get(BUF_WVM, p.v_bytes + p.m_bytes, &wvm));
    const bool bf = g.xdt == CONV2D_BF16;  // U and V bf16, V [16][tc][C] from NHWC x
    const int64_t es = elem_size(g.xdt);
    void* v = wvm;
    float* m = reinterpret_cast<float*>(static_cast<char*>(wvm) + p.v_bytes);
    {
        // pre-convolution reordering: the filter transform
        Scope sc(d, CONV2D_ALGO_WINOGRAD, CONV2D_PH_PRE_REORDER, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(launch_wino_filter(w, wu, (int)g.K, (int)g.C, p.mt, g.xdt, s));
        CV_TRY(sc.end());
    }
    WinoArgs wa{};
    wa.x = x;
    wa.x_bytes = (uint32_t)(g.x_elems * es);
    wa.y = y;
    wa.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
    wa.bias = g.has_bias ? bias : nullptr;
    wa.C = (int32_t)g.C; wa.H = (int32_t)g.H; wa.W = (int32_t)g.W; wa.K = (int32_t)g.K;
    wa.Ho = (int32_t)g.Ho; wa.Wo = (int32_t)g.Wo; wa.ph = g.ph; wa.pw = g.pw;
    wa.mt = p.mt;
    wa.th = (int32_t)ceil_div(g.Ho, p.mt);
    wa.tw = (int32_t)ceil_div(g.Wo, p.mt);
    for (int64_t t0 = 0; t0 < p.tiles; t0 += p.tc) {
        wa.t0 = t0;
        wa.tc = (int32_t)std::min<int64_t>(p.tc, p.tiles - t0);
        {
            Scope sc(d, CONV2D_ALGO_WINOGRAD, CONV2D_PH_IN_PACKING, s, ph);
            CV_TRY(sc.begin());
            if (bf)
                CV_HIP(launch_wino_input_nhwc(wa, static_cast<uint16_t*>(v), s));
            else
                CV_HIP(launch_wino_input(wa, static_cast<float*>(v), s));
            CV_TRY(sc.end());
        }
        {
            // one GEMM per transformed position: M[xi] = U[xi] (K x C) * V[xi] (C x tc); in bf16
            // V[xi] is stored transposed (tc x C)
            const GemmPlan& gp = p.gemm;
            GemmArgs a{};
            a.a = wu;
            a.a_bytes = (uint32_t)p.u_bytes;
            a.lda = (int32_t)g.C;
            a.a_gstride = g.K * g.C;
            a.b = v;
            a.b_bytes = (uint32_t)(p.npos * g.C * wa.tc * es);
            a.b_gstride = g.C * wa.tc;
            a.ldb = bf ? (int32_t)g.C : wa.tc;
            a.M = (int32_t)g.K;
            a.Kred = (int32_t)g.C;
            a.P = wa.tc;
            a.nstages = gp.nstages;
            a.grid_m = (int32_t)ceil_div(g.K, gp.bm);
            a.grid_p = (int32_t)ceil_div(wa.tc, gp.bn);
            a.y = m;
            a.y_bytes = (uint32_t)(p.npos * g.K * wa.tc * 4);
            a.ldc = wa.tc;
            a.c_gstride = g.K * wa.tc;
            a.HoWo = (int32_t)(g.Ho * g.Wo);
            Scope sc(d, CONV2D_ALGO_WINOGRAD, CONV2D_PH_IN_MICROKERNEL, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(dispatch_gemm(gp, a, bf ? BSRC_DENSE_T : BSRC_DENSE, EPI_DENSE, g.xdt, CONV2D_F32, p.npos, s));
            CV_TRY(sc.end());
        }
        {
            Scope sc(d, CONV2D_ALGO_WINOGRAD, CONV2D_PH_IN_UNPACKING, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(launch_wino_output(wa, m, g.ydt, s));
            CV_TRY(sc.end());
        }
    }
    return CONV2D_OK;
}

int run_explicit(conv2d_desc* d, Ws& ws, const void* x, const void* w, const float* bias, void* y, hipStream_t s,
                 bool ph) {
    const Geometry& g = d->g;
    const ExplicitPlan& e = d->expl;
    if (e.status != CONV2D_OK) return e.status;
    void* wsb = nullptr;
    CV_TRY(ws.get(BUF_WS, e.col_bytes + e.c_bytes, &wsb));
    const KTabEntry* ktab = nullptr;
    CV_TRY(ws.table(s, &ktab));
    char* col = static_cast<char*>(wsb);
    float* cbuf = reinterpret_cast<float*>(col + e.col_bytes);
    const int64_t total_rows = g.N * g.Ho;
    for (int64_t r0 = 0; r0 < total_rows; r0 += e.rows_per_chunk) {
        const int64_t rows = std::min<int64_t>(e.rows_per_chunk, total_rows - r0);
        const int64_t pc = rows * g.Wo;
        const int64_t p_begin = r0 * g.Wo;
        {
            Im2colArgs a{};
            a.x = x;
            a.x_bytes = g.x_elems * elem_size(g.xdt) <= kBufferLimit ? (uint32_t)(g.x_elems * elem_size(g.xdt)) : 0u;
            a.col = col;
            a.col_bytes = (uint32_t)(g.G * g.Kred * pc * elem_size(g.xdt));
            a.ktab = ktab;
            a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.Ho = (int32_t)g.Ho; a.Wo = (int32_t)g.Wo;
            a.sh = g.sh; a.sw = g.sw; a.ph = g.ph; a.pw = g.pw;
            a.x_nstride = g.C * g.H * g.W;
            a.x_gstride = g.Cg * g.H * g.W;
            a.Kred = (int32_t)g.Kred;
            a.pc = (int32_t)pc;
            a.p_begin = p_begin;
            Scope sc(d, CONV2D_ALGO_IM2COL_GEMM, CONV2D_PH_IN_PACKING, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(launch_im2col(a, g.xdt, (int)g.G, s));
            CV_TRY(sc.end());
        }
        {
            const GemmPlan& gp = e.gemm;
            GemmArgs a{};
            a.a = w;
            a.a_bytes = (uint32_t)(g.w_elems * elem_size(g.xdt));
            a.lda = (int32_t)g.Kred;
            a.a_gstride = g.Kg * g.Kred;
            a.b = col;
            a.b_bytes = (uint32_t)(g.G * g.Kred * pc * elem_size(g.xdt));
            a.b_gstride = g.Kred * pc;
            a.ldb = (int32_t)pc;
            a.M = (int32_t)g.Kg;
            a.Kred = (int32_t)g.Kred;
            a.P = (int32_t)pc;
            a.nstages = gp.nstages;
            a.grid_m = (int32_t)ceil_div(g.Kg, gp.bm);
            a.grid_p = (int32_t)ceil_div(pc, gp.bn);
            a.y = cbuf;
            a.y_bytes = (uint32_t)(g.G * g.Kg * pc * 4);
            a.ldc = (int32_t)pc;
            a.c_gstride = g.Kg * pc;
            a.HoWo = (int32_t)(g.Ho * g.Wo);
            Scope sc(d, CONV2D_ALGO_IM2COL_GEMM, CONV2D_PH_IN_MICROKERNEL, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(dispatch_gemm(gp, a, BSRC_DENSE, EPI_DENSE, g.xdt, CONV2D_F32, (int)g.G, s));
            CV_TRY(sc.end());
        }
        {
            UnpackArgs a{};
            a.c = cbuf;
            a.y = y;
            a.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
            a.bias = g.has_bias ? bias : nullptr;
            a.Kg = (int32_t)g.Kg;
            a.pc = (int32_t)pc;
            a.HoWo = (int32_t)(g.Ho * g.Wo);
            a.p_begin = p_begin;
            a.y_nstride = g.K * g.Ho * g.Wo;
            Scope sc(d, CONV2D_ALGO_IM2COL_GEMM, CONV2D_PH_IN_UNPACKING, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(launch_unpack(a, g.ydt, (int)g.G, s));
            CV_TRY(sc.end());
        }
    }
    return CONV2D_OK;
}

int run_direct(conv2d_desc* d, Ws& ws, const void* x, const void* w, const float* bias, void* y, hipStream_t s,
               bool ph) {
    const Geometry& g = d->g;
    DirectArgs a{};
    a.x = x; a.w = w; a.bias = g.has_bias ? bias : nullptr; a.y = y;
    a.x_bytes = (uint32_t)(g.x_elems * elem_size(g.xdt));
    a.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
    a.w_bytes = (uint32_t)std::min<int64_t>(g.w_elems * elem_size(g.xdt), kBufferLimit);
    a.C = (int32_t)g.C; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.K = (int32_t)g.K;
    a.Ho = (int32_t)g.Ho; a.Wo = (int32_t)g.Wo; a.R = (int32_t)g.R; a.S = (int32_t)g.S;
    a.sh = g.sh; a.sw = g.sw; a.ph = g.ph; a.pw = g.pw; a.dh = g.dh; a.dw = g.dw;
    a.Cg = (int32_t)g.Cg; a.Kg = (int32_t)g.Kg; a.N = (int32_t)g.N;
    if (d->direct_nhwc) {
        // pre-convolution reordering of the filters [C][R*S] -> [R*S][C] (4 channels per load)
        void* wd = nullptr;
        CV_TRY(ws.get(BUF_WD, g.w_elems * elem_size(g.xdt), &wd));
        {
            Scope sc(d, CONV2D_ALGO_DIRECT, CONV2D_PH_PRE_REORDER, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(launch_nchw_to_nhwc(w, wd, 1, g.C, g.R * g.S, (int)elem_size(g.xdt), s));
            CV_TRY(sc.end());
        }
        Scope sc(d, CONV2D_ALGO_DIRECT, CONV2D_PH_IN_MICROKERNEL, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(launch_dw_nhwc(a, wd, g.xdt, g.ydt, s));
        return sc.end();
    }
    if (d->smallk_ranges > 0) {
        // few output channels: channel ranges summed in fp32 partials, then the unpack kernel
        const int ranges = d->smallk_ranges;
        float* part = nullptr;
        if (ranges > 1) {
            void* dk = nullptr;
            CV_TRY(ws.get(BUF_DK, (int64_t)ranges * g.K * g.P * 4, &dk));
            part = static_cast<float*>(dk);
        }
        {
            Scope sc(d, CONV2D_ALGO_DIRECT, CONV2D_PH_IN_MICROKERNEL, s, ph);
            CV_TRY(sc.begin());
            CV_HIP(launch_smallk(a, part, ranges, g.xdt, g.ydt, s));
            CV_TRY(sc.end());
        }
        if (ranges == 1) return CONV2D_OK;
        UnpackArgs u{};
        u.c = part;
        u.y = y;
        u.y_bytes = (uint32_t)(g.y_elems * elem_size(g.ydt));
        u.bias = g.has_bias ? bias : nullptr;
        u.Kg = (int32_t)g.K;
        u.pc = (int32_t)g.P;
        u.HoWo = (int32_t)(g.Ho * g.Wo);
        u.p_begin = 0;
        u.y_nstride = g.K * g.Ho * g.Wo;
        u.splits = ranges;
        u.split_stride = g.K * g.P;
        Scope sc(d, CONV2D_ALGO_DIRECT, CONV2D_PH_IN_UNPACKING, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(launch_unpack(u, g.ydt, 1, s));
        return sc.end();
    }
    Scope sc(d, CONV2D_ALGO_DIRECT, CONV2D_PH_IN_MICROKERNEL, s, ph);
    CV_TRY(sc.begin());
    CV_HIP(launch_direct(a, g.xdt, g.ydt, s));
    return sc.end();
}

bool direct_supported(const Geometry& g) {
    if (g.x_elems * elem_size(g.xdt) > kBufferLimit || g.y_elems * elem_size(g.ydt) > kBufferLimit)
        return false;
    if (g.Wo > 1024 || g.N * g.K > 0x7fffffffLL) return false;
    const int64_t in_cols = (g.Wo - 1) * g.sw + (g.S - 1) * g.dw + 1;
    const int64_t in_rows = (g.R - 1) * g.dh + 1;
    return in_rows * in_cols <= 12288;
}

bool implicit_supported(const Geometry& g) {
    return g.x_elems * elem_size(g.xdt) <= kBufferLimit && g.y_elems * elem_size(g.ydt) <= kBufferLimit &&
           g.w_elems * elem_size(g.xdt) <= kBufferLimit && g.P <= 0x7fffffffLL && g.Kred <= 0x7fffffffLL;
}

// Argument and algorithm checks shared by both forward entry points; resolves AUTO.
int check_call(const conv2d_desc* d, const void* x, const void* w, const float* bias, const void* y, int* algo) {
    if (!d || !x || !w || !y) return CONV2D_E_NULL;
    if (d->g.has_bias && !bias) return CONV2D_E_NULL;
    if (*algo < 0 || *algo >= CONV2D_ALGO_COUNT) return CONV2D_E_INVALID;
    if (*algo == CONV2D_ALGO_AUTO) *algo = d->auto_algo;
    const Geometry& g = d->g;
    if (*algo == CONV2D_ALGO_IMPLICIT_GEMM && !d->implicit_ok) return CONV2D_E_UNSUPPORTED;
    if (*algo == CONV2D_ALGO_DIRECT && !d->direct_ok) return CONV2D_E_UNSUPPORTED;
    if (*algo == CONV2D_ALGO_WINOGRAD && !d->wino.ok) return d->wino.status;
    if (*algo == CONV2D_ALGO_IM2COL_GEMM) {
        if (d->expl.status != CONV2D_OK) return d->expl.status;
        if (g.y_elems * elem_size(g.ydt) > kBufferLimit) return CONV2D_E_UNSUPPORTED;
    }
    return CONV2D_OK;
}

// One forward convolution: the layout reorders around the algorithm's kernels, with the
// workspaces from ws.  ph: an event pair around every phase launch.
int fwd_core(conv2d_desc* d, Ws& ws, const void* x, const void* w, const float* bias, void* y, int algo,
             hipStream_t s, bool ph) {
    const Geometry& g = d->g;
    const void* xin = x;
    void* yout = y;
    const bool nhwc = g.layout == CONV2D_NHWC;
    // The bf16 NHWC gather and the bf16 Winograd input transform read x channel-contiguous: an
    // NHWC x goes in as it is, an NCHW x is reordered.  Every other kernel reads NCHW x.
    const bool x_nhwc = (algo == CONV2D_ALGO_IMPLICIT_GEMM && d->implicit_nhwc && !d->implicit_slice) ||
                        (algo == CONV2D_ALGO_WINOGRAD && g.xdt == CONV2D_BF16) ||
                        (algo == CONV2D_ALGO_DIRECT && d->direct_nhwc);
    if (nhwc != x_nhwc) {
        const int64_t xb = g.x_elems * elem_size(g.xdt);
        void* xr = nullptr;
        CV_TRY(ws.get(BUF_XR, xb, &xr));
        Scope sc(d, algo, CONV2D_PH_PRE_REORDER, s, ph);
        CV_TRY(sc.begin());
        if (nhwc)
            CV_HIP(launch_nhwc_to_nchw(x, xr, g.N, g.C, g.H * g.W, (int)elem_size(g.xdt), s));
        else
            CV_HIP(launch_nchw_to_nhwc(x, xr, g.N, g.C, g.H * g.W, (int)elem_size(g.xdt), s));
        CV_TRY(sc.end());
        xin = xr;
    }
    // NCHW result reordered to NHWC afterwards, unless the kernel writes NHWC y itself
    const bool y_reorder = nhwc && !(algo == CONV2D_ALGO_IMPLICIT_GEMM && implicit_writes_nhwc(d)) &&
                           !(algo == CONV2D_ALGO_DIRECT && d->direct_nhwc);
    if (y_reorder) {
        const int64_t yb = g.y_elems * elem_size(g.ydt);
        CV_TRY(ws.get(BUF_YR, yb, &yout));
    }
    int st = CONV2D_OK;
    switch (algo) {
        case CONV2D_ALGO_IMPLICIT_GEMM: st = run_implicit(d, ws, xin, w, bias, yout, s, ph); break;
        case CONV2D_ALGO_IM2COL_GEMM: st = run_explicit(d, ws, xin, w, bias, yout, s, ph); break;
        case CONV2D_ALGO_DIRECT: st = run_direct(d, ws, xin, w, bias, yout, s, ph); break;
        case CONV2D_ALGO_WINOGRAD: st = run_winograd(d, ws, xin, w, bias, yout, s, ph); break;
        default: st = CONV2D_E_INVALID;
    }
    if (st != CONV2D_OK) return st;
    if (y_reorder) {
        Scope sc(d, algo, CONV2D_PH_POST_REORDER, s, ph);
        CV_TRY(sc.begin());
        CV_HIP(launch_nchw_to_nhwc(yout, y, g.N, g.K, g.Ho * g.Wo, (int)elem_size(g.ydt), s));
        CV_TRY(sc.end());
    }
    return CONV2D_OK;
}

// ------------------------------------------------------------------ no-allocation scratch
// The workspaces of conv2d_fwd_noalloc live in this array: one copy per device, at a
// different address on each, held until the process ends.  Host code never passes the
// array's name to a kernel or a copy (on the host it is a stand-in symbol, not a device
// address): it uses the address hipGetSymbolAddress returned on that device.
// Bytes [0, kScratchCounterBytes) hold the tail split's arrival counters and nothing else:
// they are cleared once per device here, and the tail-split kernel returns every counter it
// uses to zero before it exits, so they are zero at the start of every launch.  The rest is
// carved into the call's workspaces; each call overwrites what the previous one left there.
constexpr int64_t kScratchCounterBytes = 4096;
static __device__ __align__(256) char scratch[CONV2D_NOALLOC_SCRATCH_BYTES];

struct ScratchDev {
    char* base;
    int cus;
};
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
ScratchDev g_scratch[kMaxDevices] = {};

int scratch_for(int dev, hipStream_t s, ScratchDev* out) {
    if (dev < 0 || dev >= kMaxDevices) return CONV2D_E_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchDev& e = g_scratch[dev];
    if (!e.base) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CONV2D_E_HIP;
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            return CONV2D_E_HIP;
        if (launch_fill_u32(static_cast<uint32_t*>(p), kScratchCounterBytes / (int64_t)sizeof(uint32_t), 0u, s) !=
            hipSuccess)
            return CONV2D_E_HIP;
        e.base = static_cast<char*>(p);
        e.cus = cus;
    }
    *out = e;
    return CONV2D_OK;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

int conv2d_desc_create(const conv2d_params* params, conv2d_desc** out) {
    const auto t0 = std::chrono::steady_clock::now();
    if (!params || !out) return CONV2D_E_NULL;
    *out = nullptr;
    Geometry g{};
    const int st = validate(params, &g);
    if (st != CONV2D_OK) return st;
    conv2d_desc* d = new (std::nothrow) conv2d_desc();
    if (!d) return CONV2D_E_ALLOC;
    d->prm = *params;
    d->g = g;
    d->opclass = classify(g);
    std::memset(d->acc, 0, sizeof(d->acc));
    d->timing = env_timing();
    d->implicit_ok = implicit_supported(g);
    d->direct_ok = direct_supported(g);
    {
        // ungrouped fp32 layers with K <= 4, square 1/3/5/7 filters and reductions C*R*S of at
        // least 2048: the few-output-channel direct kernel (any plane size; x and y below 2 GiB,
        // P below 2^31).  Measured on MI355X against the implicit GEMM (32-row tiles) and the
        // grouped direct kernel: 1.8-2.9x faster than the GEMM on 3x3-7x7 layers with C = 512 ..
        // 2048, but behind the grouped kernel on shorter reductions (64 channels x 5x5: 771 vs
        // 674 us) and, in bf16, behind the NHWC-gather GEMM and the grouped kernel.
        // CONV2D_SMALLK=0 / 1 forces it off / on (any dtype), CONV2D_SMALLK_RANGES=n forces n
        // channel ranges.
        DirectArgs da{};
        da.C = (int32_t)g.C; da.K = (int32_t)g.K; da.R = (int32_t)g.R; da.S = (int32_t)g.S;
        da.Cg = (int32_t)g.Cg; da.Kg = (int32_t)g.Kg; da.N = (int32_t)g.N;
        da.Ho = (int32_t)g.Ho; da.Wo = (int32_t)g.Wo;
        const bool fits = g.x_elems * elem_size(g.xdt) <= kBufferLimit &&
                          g.y_elems * elem_size(g.ydt) <= kBufferLimit && g.P <= 0x7fffffffLL;
        const int64_t mode = env_int64("CONV2D_SMALLK", -1);
        const bool want = mode > 0 || (mode < 0 && g.xdt == CONV2D_F32 && g.C * g.R * g.S >= 2048);
        if (fits && want && smallk_supported(da) && !std::getenv("CONV2D_DW_GENERIC")) {
            const int64_t force = env_int64("CONV2D_SMALLK_RANGES", 0);
            d->smallk_ranges = force > 0 ? (int)std::min<int64_t>(force, std::min<int64_t>(g.C, 65535))
                                         : smallk_ranges(da);
            d->direct_ok = true;
        }
        // depthwise layers with NHWC x and y: the NHWC depthwise kernel reads x and writes y as
        // they are (no layout reorders; CONV2D_DW_GENERIC keeps the NCHW kernels)
        if (fits && g.layout == CONV2D_NHWC && d->smallk_ranges == 0 && dw_nhwc_supported(da) &&
            !std::getenv("CONV2D_DW_GENERIC")) {
            d->direct_nhwc = true;
            d->direct_ok = true;
        }
    }
    // bf16 with C/g a multiple of 32, or C/g = 8 or 16 (whole taps per 32-deep stage): gather
    // 16-byte channel runs from an NHWC copy of x.  The copy costs 2|x| of HBM traffic (nothing
    // when x is already NHWC), so it is taken when the convolution does at least 1000 flops per
    // input byte, or at least 36 when a stride skips input columns: the element-wise gather then
    // uses half of every line it fetches: 9 strided bf16 layers at 36 to 512 flops per byte ran
    // 0.42-0.82x as long with the copy, one at 32 twice as long, and stride-1 layers at 147 to
    // 800 flops per byte 1.1-1.4x as long.  CONV2D_NHWC_GATHER=0 / 1 forces it.
    if (g.xdt == CONV2D_BF16 && (g.Cg % 32 == 0 || g.Cg == 8 || g.Cg == 16)) {
        const double flops = 2.0 * (double)g.N * g.K * g.Cg * g.R * g.S * g.Ho * g.Wo;
        const double xbytes = (double)g.x_elems * 2;
        const bool strided = g.sh > 1 || g.sw > 1;
        const int64_t force = env_int64("CONV2D_NHWC_GATHER", -1);
        d->implicit_nhwc = force < 0 ? (g.layout == CONV2D_NHWC || flops >= 1000.0 * xbytes ||
                                        (strided && flops >= 36.0 * xbytes))
                                     : force != 0;
    }
    // fp32 NHWC x with C/g a multiple of 16: gather 4-channel runs with 16-byte loads straight
    // from x (no reorder of x); NCHW fp32 x keeps the NCHW gathers (a copy of x would cost more
    // than the wider loads save).  CONV2D_NHWC_GATHER=0 / 1 forces it for such shapes.
    if (g.xdt == CONV2D_F32 && g.Cg % 16 == 0 && g.C % 4 == 0) {
        const int64_t force = env_int64("CONV2D_NHWC_GATHER", -1);
        d->implicit_nhwc = force < 0 ? g.layout == CONV2D_NHWC : force != 0;
    }
    d->implicit = choose_tile(g.Kg, g.P, g.G, g.Kred, g.xdt, g.Cg, d->implicit_nhwc);
    d->implicit_tap = g.Cg % d->implicit.bk == 0;
    plan_split(d);
    plan_tail(d);
    {
        // 8 waves (256-pixel tiles) unless an image has at most 128 output pixels; fp32 layers
        // with at least two rounds of 512-pixel tiles on one block per CU (256 CUs) take 16 waves
        // and two slice buffers, so the next tile's copy overlaps this tile's MFMAs with 4 waves
        // per SIMD (cfg4: 15 % faster than 8 waves, one buffer and two blocks per CU).
        // CONV2D_SLICE_WAVES = 4, 8 or 16 (fp32) and CONV2D_SLICE_DB = 0 / 1 override.
        const auto tiles = [&](int w) { return g.G * ceil_div(g.Kg, 64) * g.N * ceil_div(g.Ho * g.Wo, 32 * w); };
        int nw = g.Ho * g.Wo <= 128 ? 4 : 8;
        if (g.xdt == CONV2D_F32 && g.Ho * g.Wo >= 512 && tiles(16) >= 512) nw = 16;
        const int64_t force_nw = env_int64("CONV2D_SLICE_WAVES", 0);
        if (force_nw == 4 || force_nw == 8 || (force_nw == 16 && g.xdt == CONV2D_F32)) nw = (int)force_nw;
        const int64_t force_db = env_int64("CONV2D_SLICE_DB", -1);
        const bool db = force_db < 0 ? g.xdt == CONV2D_F32 && tiles(nw) >= 512 : force_db != 0;
        d->slice = slice_plan(g.Cg, g.R, g.S, g.Ho, g.Wo, g.sh, g.sw, g.dh, g.dw, g.xdt, nw, g.W, g.pw,
                              !std::getenv("CONV2D_SLICE_UNPACKED"), db);
        if (!d->slice.ok && nw == 16 && force_nw != 16) {
            nw = 8;
            d->slice = slice_plan(g.Cg, g.R, g.S, g.Ho, g.Wo, g.sh, g.sw, g.dh, g.dw, g.xdt, nw, g.W, g.pw,
                                  !std::getenv("CONV2D_SLICE_UNPACKED"), tiles(nw) >= 512);
        }
        d->slice_u = slice_plan(g.Cg, g.R, g.S, g.Ho, g.Wo, g.sh, g.sw, g.dh, g.dw, g.xdt, nw);
    }
    // The sliced kernel replaces the table-driven gather (C/g not a multiple of the stage
    // depth) when its LDS footprint fits; CONV2D_SLICE=0 / 1 forces the choice for tests.
    {
        const int64_t force = env_int64("CONV2D_SLICE", -1);
        const bool grid_ok = g.G * ceil_div(g.Kg, 64) * g.N * ceil_div(g.Ho * g.Wo, 128) <= 0x7fffffffLL;
        d->implicit_slice =
            d->slice.ok && grid_ok && (force < 0 ? !(d->implicit_tap || d->implicit_nhwc) : force != 0);
    }
    build_ktab(d);
    plan_explicit(d);
    plan_winograd(d);
    // Grouped layers with few channels per group sum on the vector ALUs (depthwise and the
    // grouped direct kernel): a short reduction and few output channels per group waste most of
    // an MFMA tile.  Measured crossover on MI355X: C/g <= 16 with K/g <= 32 runs faster there in
    // fp32 and bf16; C/g = K/g = 32 ties in fp32 and favours the bf16 MFMA path.
    //
    // Ungrouped layers with very few output channels (K <= 16) waste 3/4 or more of every
    // 64-row MFMA tile; the grouped direct kernel (one "group" of all channels) computes them on
    // the vector ALUs instead when its grid fills the chip (its blocks walk the whole reduction,
    // so a small grid leaves CUs idle) and the filter is not 1x1 (a pointwise layer is a plain
    // GEMM with no gather, which the MFMA path runs well even with few rows).  With 5..16 output
    // channels only short reductions stay there: since the 32-row tiles, the implicit GEMM ran
    // N32 64..512 -> 16 layers (reductions of 1152 to 4608) in 0.77-0.94x the time, while
    // 3 -> 16 5x5 (75) took 1.8x as long.
    bool direct_small_k = false;
    if (d->direct_ok && g.G == 1 && g.K <= 16 && g.R * g.S > 1 && (g.K <= 4 || g.Cg * g.R * g.S <= 256)) {
        DirectArgs da{};
        da.C = (int32_t)g.C; da.H = (int32_t)g.H; da.W = (int32_t)g.W; da.K = (int32_t)g.K;
        da.Ho = (int32_t)g.Ho; da.Wo = (int32_t)g.Wo; da.R = (int32_t)g.R; da.S = (int32_t)g.S;
        da.sh = g.sh; da.sw = g.sw; da.ph = g.ph; da.pw = g.pw; da.dh = g.dh; da.dw = g.dw;
        da.Cg = (int32_t)g.Cg; da.Kg = (int32_t)g.Kg; da.N = (int32_t)g.N;
        direct_small_k = grouped_blocks(da) >= 384;
    }
    if (d->direct_ok && ((g.G > 1 && (g.Cg <= 8 || (g.Cg <= 16 && g.Kg <= 32))) || direct_small_k ||
                         (d->smallk_ranges > 0 && g.R * g.S > 1)))
        d->auto_algo = CONV2D_ALGO_DIRECT;
    // 3x3 stride-1 fp32 layers with at least 128 input and output channels and output planes of
    // at least 8x8: Winograd F(4x4,3x3) does 4x fewer multiplications, which outweighs its
    // transforms (measured 1.6-2.0x faster than the implicit GEMM for C, K = 128 .. 1024 on
    // 14x14 to 112x112 planes on MI355X; 64 -> 64 channels on 56x56 gain under 10 %).  On 7x7
    // planes F(2x2,3x3) (2.25x fewer) pays off from about 4 GFLOP: 0.60-0.72x the time for N32
    // 512 -> 512, 256 -> 1024, 1024 -> 1024 and N8 2048 -> 2048, but 1.1x for N8 512 -> 512 and
    // 1.24x for N32 128 -> 128 (1.9 and 0.5 GFLOP), whose small per-position GEMMs stay inefficient.
    else if (d->wino.ok && g.xdt == CONV2D_F32 && g.C >= 128 && g.K >= 128 &&
             (std::min(g.Ho, g.Wo) >= 8 ||
              (std::min(g.Ho, g.Wo) >= 7 && 2.0 * g.N * g.K * g.C * 9.0 * g.Ho * g.Wo >= 4e9)))
        d->auto_algo = CONV2D_ALGO_WINOGRAD;
    else if (d->implicit_ok)
        d->auto_algo = CONV2D_ALGO_IMPLICIT_GEMM;
    else if (d->expl.status == CONV2D_OK && g.y_elems * elem_size(g.ydt) <= kBufferLimit)
        d->auto_algo = CONV2D_ALGO_IM2COL_GEMM;
    else if (d->direct_ok)
        d->auto_algo = CONV2D_ALGO_DIRECT;
    else
        d->auto_algo = CONV2D_ALGO_IMPLICIT_GEMM;  // conv2d_fwd will report E_UNSUPPORTED
    const auto t1 = std::chrono::steady_clock::now();
    d->analysis_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
    *out = d;
    return CONV2D_OK;
}

int conv2d_desc_destroy(conv2d_desc* d) {
    if (!d) return CONV2D_OK;
    for (const EvRec& r : d->pending) {
        hipEventDestroy(r.a);
        hipEventDestroy(r.b);
    }
    for (hipEvent_t e : d->free_events) hipEventDestroy(e);
    if (d->ktab_dev) hipFree(d->ktab_dev);
    for (int i = 0; i < BUF_COUNT; ++i)
        if (d->buf[i]) hipFree(d->buf[i]);
    if (d->tc) hipFree(d->tc);
    if (d->done) hipEventDestroy(d->done);
    delete d;
    return CONV2D_OK;
}

int conv2d_output_shape(const conv2d_desc* d, int64_t out_nkhw[4]) {
    if (!d || !out_nkhw) return CONV2D_E_NULL;
    out_nkhw[0] = d->g.N;
    out_nkhw[1] = d->g.K;
    out_nkhw[2] = d->g.Ho;
    out_nkhw[3] = d->g.Wo;
    return CONV2D_OK;
}

int conv2d_fwd(conv2d_desc* d, const void* x, const void* w, const float* bias, void* y, int algo,
               void* stream) {
    CV_TRY(check_call(d, x, w, bias, y, &algo));
    hipStream_t s = static_cast<hipStream_t>(stream);
    CV_TRY(ensure_device(d, s));
    // a call on another stream than the previous one waits for that call first (the two share
    // this descriptor's workspaces and counters)
    CV_TRY(order_after_last(d, s));
    if (d->pending.size() > 8192) CV_TRY(harvest(d, false));
    if (d->pending.size() > 65536) CV_TRY(harvest(d, true));

    Scope total(d, algo, -1, s, d->timing == CONV2D_TIMING_TOTAL);
    CV_TRY(total.begin());
    Ws ws{d};
    ws.cus = d->cus;
    CV_TRY(fwd_core(d, ws, x, w, bias, y, algo, s, d->timing == CONV2D_TIMING_PHASES));
    CV_TRY(total.end());
    d->acc[algo].fwd_calls += 1;
    d->acc[algo].used = true;
    d->last_algo = algo;
    if (algo == CONV2D_ALGO_IMPLICIT_GEMM) d->implicit_ran = true;
    return CONV2D_OK;
}

int conv2d_fwd_noalloc(const conv2d_desc* dc, const void* x, const void* w, const float* bias, void* y, int algo,
                       void* stream) {
    // Nothing below writes the descriptor: no events (timing is off for this entry point), no
    // device buffers (every workspace is carved from the scratch array), no uploaded table.
    conv2d_desc* d = const_cast<conv2d_desc*>(dc);
    CV_TRY(check_call(d, x, w, bias, y, &algo));
    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CONV2D_E_HIP;
    ScratchDev sd{};
    CV_TRY(scratch_for(dev, s, &sd));
    Ws ws{d};
    ws.scratch = sd.base + kScratchCounterBytes;
    ws.cap = CONV2D_NOALLOC_SCRATCH_BYTES - kScratchCounterBytes;
    ws.counters = reinterpret_cast<uint32_t*>(sd.base);
    ws.counter_cap = kScratchCounterBytes / (int64_t)sizeof(uint32_t);
    ws.cus = sd.cus;
    return fwd_core(d, ws, x, w, bias, y, algo, s, false);
}

int conv2d_pack_probe(conv2d_desc* d, const void* x, const void* w, void* stream) {
    if (!d || !x || !w) return CONV2D_E_NULL;
    if (!d->implicit_ok) return CONV2D_E_UNSUPPORTED;
    if (d->device < 0 || !d->implicit_ran) return CONV2D_E_NO_DATA;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CONV2D_E_HIP;
    if (dev != d->device) return CONV2D_E_UNSUPPORTED;
    const Geometry& g = d->g;
    // the x the microkernel reads: the internal copy when the layouts differ (made by the last call)
    const bool x_nhwc = d->implicit_nhwc && !d->implicit_slice;
    const void* xin = (g.layout == CONV2D_NHWC) != x_nhwc ? d->buf[BUF_XR] : x;
    if (!xin) return CONV2D_E_NO_DATA;
    hipStream_t s = static_cast<hipStream_t>(stream);
    CV_TRY(order_after_last(d, s));
    Ws ws{d};
    ws.cus = d->cus;
    return run_implicit(d, ws, xin, w, nullptr, nullptr, s, false, PROBE_LOADER);
}

int conv2d_kernel_probe(conv2d_desc* d, const void* x, const void* w, const float* bias, void* y, void* stream) {
    if (!d || !x || !w || !y) return CONV2D_E_NULL;
    if (d->g.has_bias && !bias) return CONV2D_E_NULL;
    if (!d->implicit_ok) return CONV2D_E_UNSUPPORTED;
    if (d->device < 0 || !d->implicit_ran) return CONV2D_E_NO_DATA;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CONV2D_E_HIP;
    if (dev != d->device) return CONV2D_E_UNSUPPORTED;
    const Geometry& g = d->g;
    // the x and y the microkernel reads and writes: the internal copies when the layouts differ
    const bool x_nhwc = d->implicit_nhwc && !d->implicit_slice;
    const void* xin = (g.layout == CONV2D_NHWC) != x_nhwc ? d->buf[BUF_XR] : x;
    void* yout = g.layout == CONV2D_NHWC && !implicit_writes_nhwc(d) ? d->buf[BUF_YR] : y;
    if (!xin || !yout) return CONV2D_E_NO_DATA;
    hipStream_t s = static_cast<hipStream_t>(stream);
    CV_TRY(order_after_last(d, s));
    Ws ws{d};
    ws.cus = d->cus;
    return run_implicit(d, ws, xin, w, bias, yout, s, false, PROBE_KERNEL);
}

int conv2d_breakdown(conv2d_desc* d, int algo, conv2d_breakdown_t* out) {
    if (!d || !out) return CONV2D_E_NULL;
    if (algo < 0 || algo >= CONV2D_ALGO_COUNT) return CONV2D_E_INVALID;
    if (algo == CONV2D_ALGO_AUTO) algo = d->last_algo;
    if (algo < 0) return CONV2D_E_NO_DATA;
    const int hst = harvest(d);
    const PhaseAcc& a = d->acc[algo];
    if (!a.used) return CONV2D_E_NO_DATA;
    std::memset(out, 0, sizeof(*out));
    for (int p = 0; p < CONV2D_PH_COUNT; ++p) {
        out->ms[p] = a.ms[p];
        out->calls[p] = a.calls[p];
    }
    out->ms[CONV2D_PH_PRE_ANALYSIS] = d->analysis_ms;
    out->calls[CONV2D_PH_PRE_ANALYSIS] = 1;
    if (algo == CONV2D_ALGO_IMPLICIT_GEMM)
        out->fused_mask = (1u << CONV2D_PH_IN_TILING) | (1u << CONV2D_PH_IN_PACKING) |
                          (d->implicit.ksplit > 1 && !d->implicit_slice ? 0u : (1u << CONV2D_PH_IN_UNPACKING));
    else if (algo == CONV2D_ALGO_IM2COL_GEMM || algo == CONV2D_ALGO_WINOGRAD)
        out->fused_mask = (1u << CONV2D_PH_IN_TILING);
    else
        out->fused_mask = (1u << CONV2D_PH_IN_TILING) | (1u << CONV2D_PH_IN_PACKING) |
                          (d->smallk_ranges > 1 ? 0u : (1u << CONV2D_PH_IN_UNPACKING));
    out->algo = algo;
    out->pack_is_preconv = algo == CONV2D_ALGO_IM2COL_GEMM ? 1 : 0;
    out->fwd_calls = a.fwd_calls;
    double op = 0.0, conv = 0.0;
    for (int p = 0; p < CONV2D_PH_COUNT; ++p) {
        op += out->ms[p];
        if (p >= CONV2D_PH_IN_TILING && p <= CONV2D_PH_IN_UNPACKING) conv += out->ms[p];
    }
    out->operation_ms = op;
    out->convolution_ms = conv;
    out->total_ms = a.total_ms;
    out->total_calls = a.total_calls;
    return hst;
}

int conv2d_breakdown_reset(conv2d_desc* d) {
    if (!d) return CONV2D_E_NULL;
    const int st = harvest(d);
    std::memset(d->acc, 0, sizeof(d->acc));
    d->last_algo = -1;
    return st;
}

int conv2d_set_timing(conv2d_desc* d, int mode) {
    if (!d) return CONV2D_E_NULL;
    if (mode < CONV2D_TIMING_OFF || mode > CONV2D_TIMING_PHASES) return CONV2D_E_INVALID;
    const int st = harvest(d);
    d->timing = mode;
    return st;
}

int conv2d_plan_query(const conv2d_desc* d, int algo, conv2d_plan_info* out) {
    if (!d || !out) return CONV2D_E_NULL;
    if (algo < 0 || algo >= CONV2D_ALGO_COUNT) return CONV2D_E_INVALID;
    if (algo == CONV2D_ALGO_AUTO) algo = d->auto_algo;
    std::memset(out, 0, sizeof(*out));
    const Geometry& g = d->g;
    out->algo = algo;
    out->kred = (int32_t)g.Kred;
    const int bk = algo == CONV2D_ALGO_IM2COL_GEMM ? d->expl.gemm.bk : d->implicit.bk;
    out->kred_pad = (int32_t)(ceil_div(g.Kred, bk) * bk);
    out->needs_reorder = g.layout == CONV2D_NHWC ? 1 : 0;
    if (algo == CONV2D_ALGO_IMPLICIT_GEMM && d->implicit_nhwc && !d->implicit_slice)
        out->needs_reorder = implicit_writes_nhwc(d) ? 0 : 1;
    if (algo == CONV2D_ALGO_WINOGRAD && g.xdt == CONV2D_BF16) out->needs_reorder = 1;
    if (algo == CONV2D_ALGO_DIRECT && d->direct_nhwc) out->needs_reorder = 0;
    out->op_class = (int32_t)d->opclass;
    out->chunks = 1;
    if (algo == CONV2D_ALGO_IMPLICIT_GEMM) {
        out->tile_m = d->implicit.bm;
        out->tile_n = d->implicit.bn;
        out->kernel = CONV2D_KERNEL_GEMM;
        out->ksplit = d->implicit.ksplit;
        if (d->implicit.ksplit > 1) out->workspace_bytes = d->implicit.ksplit * g.G * g.Kg * g.P * 4;
        out->tail_tiles = d->implicit.tail_tiles;
        out->tail_pieces = d->implicit.tail_pieces;
        if (d->implicit.tail_tiles > 0) out->workspace_bytes = tail_part_bytes(d->implicit);
        if (d->implicit_slice) {
            out->tile_m = 64;
            out->tile_n = 32 * d->slice.nw;
            out->kred_pad = 2 * d->slice.kh;
            out->kernel = CONV2D_KERNEL_SLICE;
            out->ksplit = 1;
            out->tail_tiles = out->tail_pieces = 0;
            out->workspace_bytes = 0;
        }
        if (!d->implicit_ok) return CONV2D_E_UNSUPPORTED;
    } else if (algo == CONV2D_ALGO_IM2COL_GEMM) {
        out->tile_m = d->expl.gemm.bm;
        out->tile_n = d->expl.gemm.bn;
        out->workspace_bytes = d->expl.col_bytes + d->expl.c_bytes;
        out->chunks = d->expl.chunks;
        if (d->expl.status != CONV2D_OK) return d->expl.status;
    } else if (algo == CONV2D_ALGO_WINOGRAD) {
        out->tile_m = d->wino.gemm.bm;
        out->tile_n = d->wino.gemm.bn;
        out->kred = (int32_t)g.C;  // the GEMMs reduce over the input channels
        out->kred_pad = (int32_t)(ceil_div(g.C, d->wino.gemm.bk) * d->wino.gemm.bk);
        out->workspace_bytes = d->wino.u_bytes + d->wino.v_bytes + d->wino.m_bytes;
        out->chunks = d->wino.chunks;
        out->wino_tile = d->wino.mt;
        if (!d->wino.ok) return d->wino.status;
    } else {
        out->kernel = CONV2D_KERNEL_DIRECT;
        if (d->smallk_ranges > 1) {
            out->ksplit = d->smallk_ranges;
            out->workspace_bytes = (int64_t)d->smallk_ranges * g.K * g.P * 4;
        }
        if (!d->direct_ok) return CONV2D_E_UNSUPPORTED;
    }
    return CONV2D_OK;
}

const char* conv2d_status_string(int status) {
    switch (status) {
        case CONV2D_OK: return "ok";
        case CONV2D_E_INVALID: return "invalid parameter";
        case CONV2D_E_SHAPE: return "filter window does not fit the padded input";
        case CONV2D_E_UNSUPPORTED: return "unsupported combination";
        case CONV2D_E_NULL: return "null pointer";
        case CONV2D_E_ALLOC: return "workspace allocation failed or exceeds the limit";
        case CONV2D_E_HIP: return "HIP runtime error";
        case CONV2D_E_NO_DATA: return "no timing data recorded";
        case CONV2D_E_SCRATCH: return "workspace exceeds the no-allocation scratch array";
        default: return "unknown status";
    }
}

int conv2d_runtime_version(int* v) {
    if (!v) return CONV2D_E_NULL;
    return hipRuntimeGetVersion(v) == hipSuccess ? CONV2D_OK : CONV2D_E_HIP;
}

}  // extern "C"
