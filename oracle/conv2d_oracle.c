/*
 * conv2d_oracle.c -- CPU oracle for the 2D convolution forward primitive.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The GPU library never
 * links, calls or includes anything from here, and this file includes nothing
 * from the GPU library.
 *
 * What it computes: the conv2d operation that ConvBench times (Sec. I and
 * Sec. III-B: the operations are the Conv2d layers of TIMM / torchvision
 * models, with stride, zero padding, dilation, groups and rectangular
 * filters).  The paper prints no formula; the definition written out here is
 * the zero-padded, unflipped (cross-correlation) convolution of those layers:
 *
 *   Ho = floor((H + 2*ph - dh*(R-1) - 1) / sh) + 1        (likewise Wo)
 *   y[n,k,ho,wo] = b[k] + sum_{c<C/g, r<R, s<S} x[n, gi*C/g + c, hi, wi] * w[k,c,r,s]
 *       hi = ho*sh - ph + r*dh,  wi = wo*sw - pw + s*dw,  gi = k / (K/g),
 *   taps with hi or wi outside the input contribute zero.
 *
 * It is the plain seven-loop nest (n, k, ho, wo, c, r, s), accumulated in
 * fp64.  Next to y it returns A[n,k,ho,wo] = |b[k]| + sum |x*w| over the
 * same taps, the denominator of the normalised error used by the tests.
 * Inputs are fp32 arrays holding the exact values the GPU reads (bf16 data
 * arrives already rounded, and bf16 -> fp32 -> fp64 is exact).  x and y are
 * NCHW, w is K x C/g x R x S.  Parallelism: OpenMP over (n, k) planes only;
 * each output is summed by one thread in the fixed loop order, so results do
 * not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int64_t n, c, h, w, k, r, s;
    int64_t stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, groups;
    int64_t has_bias;
} oracle_conv_t;

enum { ORACLE_OK = 0, ORACLE_E_INVALID = -1, ORACLE_E_SHAPE = -2, ORACLE_E_NULL = -4 };

/* One output extent with floor rounding; returns 0 when no window fits. */
static int64_t out_extent(int64_t in, int64_t pad, int64_t dil, int64_t ext, int64_t stride) {
    int64_t span = in + 2 * pad - dil * (ext - 1) - 1; /* last valid window start */
    if (span < 0) return 0;
    return span / stride + 1;
}

static int check_params(const oracle_conv_t* p) {
    if (!p) return ORACLE_E_NULL;
    if (p->n < 1 || p->c < 1 || p->h < 1 || p->w < 1 || p->k < 1 || p->r < 1 || p->s < 1)
        return ORACLE_E_INVALID;
    if (p->stride_h < 1 || p->stride_w < 1 || p->dil_h < 1 || p->dil_w < 1) return ORACLE_E_INVALID;
    if (p->pad_h < 0 || p->pad_w < 0 || p->groups < 1) return ORACLE_E_INVALID;
    if (p->c % p->groups != 0 || p->k % p->groups != 0) return ORACLE_E_INVALID;
    return ORACLE_OK;
}

int oracle_output_dims(const oracle_conv_t* p, int64_t* ho, int64_t* wo) {
    int st = check_params(p);
    if (st) return st;
    if (!ho || !wo) return ORACLE_E_NULL;
    *ho = out_extent(p->h, p->pad_h, p->dil_h, p->r, p->stride_h);
    *wo = out_extent(p->w, p->pad_w, p->dil_w, p->s, p->stride_w);
    if (*ho < 1 || *wo < 1) return ORACLE_E_SHAPE;
    return ORACLE_OK;
}

/* The innermost three loops for one output point. */
static void one_output(const oracle_conv_t* p, const float* x, const float* w, const float* b,
                       int64_t n, int64_t k, int64_t ho, int64_t wo, double* y_out, double* a_out) {
    const int64_t cg = p->c / p->groups, kg = p->k / p->groups;
    const int64_t gi = k / kg;
    double acc = 0.0, absacc = 0.0;
    for (int64_t c = 0; c < cg; ++c) {
        for (int64_t r = 0; r < p->r; ++r) {
            for (int64_t s = 0; s < p->s; ++s) {
                int64_t hi = ho * p->stride_h - p->pad_h + r * p->dil_h;
                int64_t wi = wo * p->stride_w - p->pad_w + s * p->dil_w;
                if (hi < 0 || hi >= p->h || wi < 0 || wi >= p->w) continue;
                double xv = (double)x[((n * p->c + gi * cg + c) * p->h + hi) * p->w + wi];
                double wv = (double)w[((k * cg + c) * p->r + r) * p->s + s];
                double t = xv * wv;
                acc += t;
                absacc += fabs(t);
            }
        }
    }
    if (p->has_bias) {
        acc += (double)b[k];
        absacc += fabs((double)b[k]);
    }
    *y_out = acc;
    if (a_out) *a_out = absacc;
}

/* Full evaluation: y and (optionally) A are N x K x Ho x Wo fp64 arrays. */
int oracle_conv2d(const oracle_conv_t* p, const float* x, const float* w, const float* b,
                  double* y, double* a, int nthreads) {
    int64_t ho_n, wo_n;
    int st = oracle_output_dims(p, &ho_n, &wo_n);
    if (st) return st;
    if (!x || !w || !y || (p->has_bias && !b)) return ORACLE_E_NULL;
    const int64_t planes = p->n * p->k;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t pl = 0; pl < planes; ++pl) {
        const int64_t n = pl / p->k, k = pl % p->k;
        for (int64_t ho = 0; ho < ho_n; ++ho) {
            for (int64_t wo = 0; wo < wo_n; ++wo) {
                const int64_t o = (pl * ho_n + ho) * wo_n + wo;
                one_output(p, x, w, b, n, k, ho, wo, &y[o], a ? &a[o] : NULL);
            }
        }
    }
    return ORACLE_OK;
}

/* Point-sampled evaluation of the same definition: idx holds npts rows of
 * (n, k, ho, wo); y[i] and a[i] receive the value at row i. */
int oracle_conv2d_points(const oracle_conv_t* p, const float* x, const float* w, const float* b,
                         int64_t npts, const int64_t* idx, double* y, double* a, int nthreads) {
    int64_t ho_n, wo_n;
    int st = oracle_output_dims(p, &ho_n, &wo_n);
    if (st) return st;
    if (!x || !w || !y || !idx || (p->has_bias && !b)) return ORACLE_E_NULL;
    for (int64_t i = 0; i < npts; ++i) {
        const int64_t* q = idx + 4 * i;
        if (q[0] < 0 || q[0] >= p->n || q[1] < 0 || q[1] >= p->k || q[2] < 0 || q[2] >= ho_n ||
            q[3] < 0 || q[3] >= wo_n)
            return ORACLE_E_INVALID;
    }
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
    for (int64_t i = 0; i < npts; ++i) {
        const int64_t* q = idx + 4 * i;
        one_output(p, x, w, b, q[0], q[1], q[2], q[3], &y[i], a ? &a[i] : NULL);
    }
    return ORACLE_OK;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
