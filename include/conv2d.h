/*
 * conv2d.h -- C ABI of the MI355X (gfx950) conv2d forward library.
 *
 * The library computes the 2D convolution forward primitive that ConvBench
 * benchmarks (Sec. I, Sec. III-B: the Conv2d layers of TIMM / torchvision
 * models, with stride, zero padding, dilation, groups and rectangular
 * filters), on one GPU, with three algorithm families and a per-phase time
 * breakdown in the nomenclature of ConvBench's timing tool (Sec. III-A):
 *
 *   y[n,k,ho,wo] = b[k] + sum_{c<C/g, r<R, s<S}
 *                  x[n, gi*C/g + c, ho*sh - ph + r*dh, wo*sw - pw + s*dw] * w[k,c,r,s]
 *   gi = k / (K/g); taps outside the input read zero (no filter flip);
 *   Ho = floor((H + 2*ph - dh*(R-1) - 1)/sh) + 1, likewise Wo.
 *
 * Conventions for every function below:
 *   - The return value is a status: CONV2D_OK (0) or a negative CONV2D_E_*.
 *     No function aborts or prints.
 *   - Device pointers (x, w, bias, y) are owned by the caller, must stay valid
 *     until the work queued on `stream` has finished, and hold dense,
 *     contiguous tensors in the layouts stated below.
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *   - A descriptor must not be used by two host threads at once; distinct
 *     descriptors are independent.
 *   - Calls on one descriptor are ordered: a conv2d_fwd (or probe) queued on
 *     another stream than the previous call on that descriptor first makes its
 *     stream wait (hipStreamWaitEvent) for an event recorded on that previous
 *     stream, behind the previous call, since both use the descriptor's
 *     workspaces.  The previous call's stream must therefore still exist when
 *     the next call names another one.  Calls on the same stream every time
 *     record no event and cost nothing extra.
 */
#ifndef CONV2D_H
#define CONV2D_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
    CONV2D_OK = 0,
    CONV2D_E_INVALID = -1,     /* a parameter is out of range (dims < 1, C % g != 0, ...) */
    CONV2D_E_SHAPE = -2,       /* the filter window does not fit: Ho < 1 or Wo < 1 */
    CONV2D_E_UNSUPPORTED = -3, /* valid convolution, but this dtype / layout / algo / size is not offered */
    CONV2D_E_NULL = -4,        /* a required pointer is NULL */
    CONV2D_E_ALLOC = -5,       /* workspace could not be allocated within the limit */
    CONV2D_E_HIP = -6,         /* a HIP runtime call or kernel launch failed */
    CONV2D_E_NO_DATA = -7,     /* breakdown (or pack probe) requested before any call that feeds it */
    CONV2D_E_SCRATCH = -8      /* conv2d_fwd_noalloc: the call needs more workspace than its static
                                  scratch array holds (CONV2D_NOALLOC_SCRATCH_BYTES) */
};

/* Layout of x and y.  w is always K x C/g x R x S (row-major). */
enum { CONV2D_NCHW = 0, CONV2D_NHWC = 1 };

/* Element types.  x and w share a type; bias is always fp32. */
enum { CONV2D_F32 = 0, CONV2D_BF16 = 1 };

/* Algorithm families (ConvBench's main and baseline methods, Sec. III-C). */
enum {
    CONV2D_ALGO_AUTO = 0,          /* planner's choice */
    CONV2D_ALGO_IMPLICIT_GEMM = 1, /* sliced direct convolution: im2col slices gathered into LDS, MFMA */
    CONV2D_ALGO_IM2COL_GEMM = 2,   /* explicit im2col pack, MFMA GEMM, unpack (ConvBench's default baseline) */
    CONV2D_ALGO_DIRECT = 3,        /* direct VALU kernels: depthwise (NCHW, or NHWC read and written
                                      as it is when C is a multiple of 4), small groups, K <= 4 */
    CONV2D_ALGO_WINOGRAD = 4,      /* Winograd F(2x2,3x3) / F(4x4,3x3): 3x3, stride 1, dilation 1, one group;
                                      fp32, or bf16 with F(2x2) only and C a multiple of 8 */
    CONV2D_ALGO_COUNT = 5
};
/* Winograd's phases: PRE_REORDER the filter transform, IN_PACKING the input
 * transform, IN_MICROKERNEL the (m+2)^2 GEMMs of the transformed domain (16 for
 * m = 2, 36 for m = 4), IN_UNPACKING the output transform with the bias (Sec. I
 * names the family; the minimal filtering algorithm is Lavin and Gray's).  The
 * planner picks the output tile m (conv2d_plan_info.wino_tile).  Its workspace
 * (transformed filters, then inputs and products per chunk of m x m output
 * tiles) obeys CONV2D_WORKSPACE_LIMIT_BYTES like the explicit path's. */

/* Processing steps of the timing tool (Sec. III-A): pre-convolution analysis and
 * reordering; in-convolution tiling, packing, microkernel and unpacking;
 * post-convolution reordering. */
enum {
    CONV2D_PH_PRE_ANALYSIS = 0,
    CONV2D_PH_PRE_REORDER = 1,
    CONV2D_PH_IN_TILING = 2,
    CONV2D_PH_IN_PACKING = 3,
    CONV2D_PH_IN_MICROKERNEL = 4,
    CONV2D_PH_IN_UNPACKING = 5,
    CONV2D_PH_POST_REORDER = 6,
    CONV2D_PH_COUNT = 7
};

/* Timing modes of a descriptor (the timing tool of Sec. III-A).  OFF records
 * nothing; TOTAL records one event pair around each conv2d_fwd (Operation Time
 * only); PHASES records one event pair around every phase launch, which costs a
 * few microseconds per phase on the GPU.  The initial mode comes from the
 * environment variable CONV2D_TIMING = off | total | phases (default: off). */
enum { CONV2D_TIMING_OFF = 0, CONV2D_TIMING_TOTAL = 1, CONV2D_TIMING_PHASES = 2 };

typedef struct conv2d_desc conv2d_desc; /* opaque, owned by the library */

/* One convolution.  n,c,h,w: input dims; k: output channels; r,s: filter
 * height and width.  Padding is symmetric zero padding (pad_h rows above and
 * below, pad_w columns left and right).  has_bias != 0 means a K-element fp32
 * bias is added once per output channel. */
typedef struct {
    int64_t n, c, h, w, k, r, s;
    int32_t stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, groups;
    int32_t layout;   /* CONV2D_NCHW or CONV2D_NHWC, for x and y */
    int32_t x_dtype;  /* CONV2D_F32 or CONV2D_BF16; the type of x and w */
    int32_t y_dtype;  /* CONV2D_F32, or CONV2D_BF16 when x_dtype is BF16 */
    int32_t has_bias;
} conv2d_params;

/* Accumulated phase times of one algorithm on one descriptor.  ms[p] is the
 * summed GPU time (hipEvent) of phase p over `calls[p]` launches, except
 * PRE_ANALYSIS, which is the host time of conv2d_desc_create (calls = 1).
 * fused_mask has bit p set when phase p runs inside another phase's kernel
 * (its time is included there).  operation_ms is the sum of all phases
 * (the timing tool's Operation Time); convolution_ms is the sum of the
 * in-convolution phases (its Convolution Time).  pack_is_preconv = 1 marks
 * that the explicit path's im2col is booked as IN_PACKING although the paper
 * also calls it a pre-convolution reordering.  total_ms / total_calls hold
 * the event pairs of TIMING_TOTAL mode (whole conv2d_fwd calls). */
typedef struct {
    double ms[CONV2D_PH_COUNT];
    int64_t calls[CONV2D_PH_COUNT];
    uint32_t fused_mask;
    int32_t algo;
    int32_t pack_is_preconv;
    int64_t fwd_calls;
    double operation_ms;
    double convolution_ms;
    double total_ms;
    int64_t total_calls;
} conv2d_breakdown_t;

/* Microkernels behind the algorithms.  IMPLICIT_GEMM runs either the tiled MFMA
 * GEMM that gathers im2col slices into LDS (GEMM) or, for short reductions
 * (C/g * R * S), the sliced direct kernel that keeps the input rows of a run of
 * output pixels in LDS and reads the columns from there (SLICE). */
enum { CONV2D_KERNEL_GEMM = 0, CONV2D_KERNEL_SLICE = 1, CONV2D_KERNEL_DIRECT = 2 };

/* What the planner decided for one algorithm (for reports and tests). */
typedef struct {
    int32_t algo;             /* resolved algorithm (never AUTO) */
    int32_t tile_m, tile_n;   /* GEMM block tile (output channels x output pixels); 0 for DIRECT */
    int32_t kred, kred_pad;   /* reduction length (C/g)*R*S and its padded length */
    int64_t workspace_bytes;  /* device workspace this algorithm uses per chunk (explicit) or for the
                                 partial sums of the split reduction or the tail split (implicit) */
    int64_t chunks;           /* explicit path: number of pack/GEMM/unpack chunks */
    int32_t needs_reorder;    /* 1 when a pre- or post-convolution layout reorder runs (x or y in the
                                 other layout than the kernel reads or writes) */
    int32_t op_class;         /* bit 0 pointwise, 1 grouped, 2 depthwise, 3 dilated, 4 rectangular, 5 strided */
    int32_t kernel;           /* microkernel that runs: CONV2D_KERNEL_* */
    int32_t ksplit;           /* implicit GEMM: reduction split into this many parts (1 = none);
                                 the parts' fp32 partial sums are added by the unpack phase.
                                 DIRECT with K <= 4 (ungrouped, square 1/3/5/7 filter): the input
                                 channels' ranges of the few-output-channel kernel, likewise */
    int32_t tail_tiles;       /* implicit GEMM: output tiles computed in tail_pieces parts by extra
                                 blocks of the same launch, so that every CU gets the same share
                                 of tile work (0 = none); the last part of a tile to finish adds
                                 the parts in order (fp32 partials in the workspace) */
    int32_t tail_pieces;
    int32_t wino_tile;        /* WINOGRAD: output tile edge m of F(m x m, 3x3), 2 or 4 */
} conv2d_plan_info;

/* Validate params, compute the output size, classify the operation and plan
 * every algorithm (operation analysis, Sec. III-A).  Host only: needs no GPU.
 * On success *out receives a new descriptor.  Errors: E_NULL, E_INVALID,
 * E_SHAPE, E_UNSUPPORTED (fp32 x with bf16 y, unknown layout/dtype). */
int conv2d_desc_create(const conv2d_params* params, conv2d_desc** out);

/* Free the descriptor, its events and its workspace.  Waits for nothing:
 * the caller must make sure no work using it is still queued.  NULL is OK. */
int conv2d_desc_destroy(conv2d_desc* desc);

/* Output dimensions of the operation: out_nkhw = {N, K, Ho, Wo} with
 * Ho = floor((H + 2*pad_h - dil_h*(R-1) - 1)/stride_h) + 1, likewise Wo (the
 * Conv2d layers of Sec. III-B; logical dims, the memory layout is the
 * descriptor's layout).  E_NULL only. */
int conv2d_output_shape(const conv2d_desc* desc, int64_t out_nkhw[4]);

/* Queue one forward convolution (the operation ConvBench times, Sec. III-B / III-C:
 * convolution() and convolution_baseline() of the harness are this call with an
 * implicit/direct algo and with CONV2D_ALGO_IM2COL_GEMM) on `stream` and return
 * without waiting.
 *   x    : N x C x H x W (NCHW) or N x H x W x C (NHWC), x_dtype
 *   w    : K x C/g x R x S, x_dtype
 *   bias : K floats, or NULL when has_bias == 0 (ignored then)
 *   y    : N x K x Ho x Wo (NCHW) or N x Ho x Wo x K (NHWC), y_dtype
 *   algo : CONV2D_ALGO_*; AUTO lets the planner choose.
 * NHWC x and y go to an NCHW kernel through library-owned reordered copies (the
 * pre- and post-convolution reordering phases) unless the kernel reads or writes
 * NHWC itself: conv2d_plan_info.needs_reorder tells which.
 * Errors: E_NULL (x, w, y or a required bias missing), E_INVALID (bad algo),
 * E_UNSUPPORTED (algo cannot run this op), E_ALLOC (explicit or Winograd
 * workspace over CONV2D_WORKSPACE_LIMIT_BYTES, default 1 GiB, even after chunking),
 * E_HIP (a launch failed).  Faults inside kernels surface at the next
 * synchronisation.  Results are bitwise reproducible for a fixed algo. */
int conv2d_fwd(conv2d_desc* desc, const void* x, const void* w, const float* bias, void* y,
               int algo, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): conv2d_fwd without any
 * allocation.  Same arguments, layouts, algorithms and results (bit for bit) as
 * conv2d_fwd; the workspaces (reordered copies, tap-major filters, split and
 * tail-split partial sums and counters, the tap table, the explicit path's
 * columns) come from one static device array of CONV2D_NOALLOC_SCRATCH_BYTES
 * per GPU, which the library holds from its first use on that GPU until the
 * process ends.  The first call on a device looks the array up and clears its
 * counter region (queued on `stream`).  No events are recorded (the
 * descriptor's timing mode is ignored) and the descriptor is not modified.
 * Every call on a GPU shares that GPU's array and overwrites what the previous
 * call left there: calls that can overlap on one GPU (other streams, other host
 * threads) race and must be serialised by the caller; conv2d_fwd calls on the
 * same descriptor are independent of it.  Errors as conv2d_fwd, plus
 * E_SCRATCH when the call needs more than the array holds (kernels of the call
 * that came before the workspace that did not fit may already be queued; y is
 * then undefined). */
#define CONV2D_NOALLOC_SCRATCH_BYTES (64LL << 20)
int conv2d_fwd_noalloc(const conv2d_desc* desc, const void* x, const void* w, const float* bias, void* y,
                       int algo, void* stream);

/* Pack probe (measurement of the fused packing, Sec. III-C breakdown): queue the
 * implicit algorithm's microkernel on `stream` with its loader only -- the im2col
 * gather into LDS with stride, padding and dilation resolved, the filter loads
 * and the barriers, but no MFMA and no output.  Its duration (timed by the
 * caller's events around the call, one kernel launch) over the full
 * microkernel's estimates the share of the packing fused into the implicit
 * algorithm.  x and w: the device pointers of a conv2d_fwd call; y and bias are
 * neither read nor written.  The probe reads the internal copies the last
 * implicit conv2d_fwd on this descriptor made (tap-major weights, a reordered
 * x), so it needs one such call first: E_NO_DATA otherwise.  E_NULL, E_UNSUPPORTED
 * (no implicit algorithm for this shape, or another device), E_HIP. */
int conv2d_pack_probe(conv2d_desc* desc, const void* x, const void* w, void* stream);

/* Kernel probe (measurement of the microkernel's own duration, Sec. III-A's
 * microkernel step): queue only the implicit algorithm's microkernel launch --
 * the tiled MFMA GEMM with its fused gather and epilogue, or the sliced kernel --
 * on `stream`, without the steps around it (filter repack, layout reorders, the
 * split reduction's unpack).  Back-to-back calls timed by the caller's events
 * give the kernel's average duration with no other launch in between.  x, w,
 * bias, y: the pointers of a conv2d_fwd call; y (or the internal NCHW result of
 * an NHWC operation, or the split partial sums) is written as that call's
 * microkernel writes it.  Reads the internal copies the last implicit conv2d_fwd
 * on this descriptor made: E_NO_DATA before such a call.  E_NULL, E_UNSUPPORTED
 * (no implicit algorithm, or another device), E_HIP. */
int conv2d_kernel_probe(conv2d_desc* desc, const void* x, const void* w, const float* bias, void* y, void* stream);

/* Roofline probes (measurement; no descriptor).  Each queues one kernel on
 * `stream` and returns at once; the caller times it with its own events.
 * conv2d_probe_mfma: an MFMA issue loop on register operands over every CU (two
 * blocks of four waves per CU, four independent accumulators per wave, `iters`
 * iterations); dtype CONV2D_F32 runs the 32x32x2 fp32 MFMA, CONV2D_BF16 the
 * 32x32x16 bf16 one.  *flops receives the floating-point operations the launch
 * performs.  sink: device buffer of at least 2 * CUs * 256 * 4 bytes that
 * receives one float per thread (their values carry no meaning).
 * conv2d_probe_copy: dst[0:bytes] = src[0:bytes] with 16-byte accesses (bytes a
 * positive multiple of 16, below 2^43; the buffers must not overlap): the device
 * copy rate, and the cache flush before a cold-cache run.
 * Errors: E_NULL, E_INVALID (dtype, iters < 1, sink too small, bytes), E_HIP. */
int conv2d_probe_mfma(int dtype, int64_t iters, void* sink, int64_t sink_bytes, void* stream, double* flops);
int conv2d_probe_copy(void* dst, const void* src, int64_t bytes, void* stream);

/* The timing tool's breakdown (Sec. III-A, Fig. 1: elapsed time and call count
 * per processing step; Operation Time = all steps, Convolution Time = the
 * in-convolution steps).  Synchronises on the descriptor's recorded events,
 * folds them into the per-algorithm totals and copies the totals of `algo`
 * (AUTO: the algorithm of the last conv2d_fwd) into *out.  With timing OFF the
 * times stay zero and only fwd_calls counts.  E_NULL, E_INVALID (algo),
 * E_NO_DATA when that algorithm has never been run, E_HIP. */
int conv2d_breakdown(conv2d_desc* desc, int algo, conv2d_breakdown_t* out);

/* Discard all accumulated phase times (PRE_ANALYSIS is kept). */
int conv2d_breakdown_reset(conv2d_desc* desc);

/* Set the timing mode (CONV2D_TIMING_*).  Pending events are folded first. */
int conv2d_set_timing(conv2d_desc* desc, int mode);

/* Planner decisions for `algo` (AUTO: the algorithm AUTO resolves to). */
int conv2d_plan_query(const conv2d_desc* desc, int algo, conv2d_plan_info* out);

/* Static text for a status code; never NULL. */
const char* conv2d_status_string(int status);

/* Version of the HIP runtime this library is bound to (hipRuntimeGetVersion). */
int conv2d_runtime_version(int* hip_runtime_version);

#ifdef __cplusplus
}
#endif

#endif /* CONV2D_H */
