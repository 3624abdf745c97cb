/*
 * Oracle: plain fp64 direct 2-D convolution on the CPU.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the correctness reference for the
 * GPU kernels. Only the tests, the smoke check and the benchmark's CPU
 * baseline leg may build, load or call it; no product code path uses it.
 * It shares no code, header or constant with the GPU library.
 *
 * What it computes: the convolution operator that the paper's autotuner
 * optimises (paper, section 2.1: operators such as 2D convolution are tuned
 * for a target device). The paper never writes the operator out; this file
 * takes the reading used by DNN frameworks and by the tuner's conv2d tasks:
 * cross-correlation (no filter flip), zero padding, floor output size,
 * grouped channels:
 *
 *   OH = floor((H + 2*ph - dh*(R-1) - 1) / sh) + 1   (same for OW)
 *   y[n,k,p,q] = sum_{c<Cg} sum_{r<R} sum_{t<S}
 *                x[n, g(k)*Cg + c, p*sh - ph + r*dh, q*sw - pw + t*dw] * w[k,c,r,t]
 *   with Cg = C/groups, Kg = K/groups, g(k) = floor(k/Kg), x = 0 off the image.
 *
 * The sum runs in fp64 in the fixed order (c, r, t) for every output. The
 * optional second output a[] is the same operator on |x| and |w|, used to
 * state rounding-error bounds.
 *
 * Layouts: layout 0 = x NCHW, w K x Cg x R x S, y NCHW.
 *          layout 1 = x NHWC, w K x R x S x Cg, y NHWC (for R = S = 1 this is
 *          the K x C weight matrix of a pointwise layer).
 *
 * nthreads > 1 spreads the (n, k) pairs over OpenMP threads; each output is
 * still summed by one thread in the same order, so the result does not
 * depend on the thread count.
 *
 * Returns 0, or -1 when the shape is inconsistent (nothing is written).
 */
#include <stdint.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int64_t out_extent(int64_t in, int64_t pad, int64_t dil, int64_t ker, int64_t stride)
{
    int64_t span = in + 2 * pad - dil * (ker - 1) - 1;
    if (span < 0) return 0;
    return span / stride + 1;
}

int oracle_out_size(int64_t in, int64_t pad, int64_t dil, int64_t ker, int64_t stride)
{
    return (int)out_extent(in, pad, dil, ker, stride);
}

/* Flat position of x[n][c][h][w] in the chosen layout. */
static int64_t x_at(int layout, int64_t n, int64_t c, int64_t h, int64_t w,
                    int64_t C, int64_t H, int64_t W)
{
    if (layout == 0) return ((n * C + c) * H + h) * W + w;
    return ((n * H + h) * W + w) * C + c;
}

/* Flat position of w[k][c][r][t] (c within the group) in the chosen layout. */
static int64_t w_at(int layout, int64_t k, int64_t c, int64_t r, int64_t t,
                    int64_t Cg, int64_t R, int64_t S)
{
    if (layout == 0) return ((k * Cg + c) * R + r) * S + t;
    return ((k * R + r) * S + t) * Cg + c;
}

static int64_t y_at(int layout, int64_t n, int64_t k, int64_t p, int64_t q,
                    int64_t K, int64_t OH, int64_t OW)
{
    if (layout == 0) return ((n * K + k) * OH + p) * OW + q;
    return ((n * OH + p) * OW + q) * K + k;
}

int oracle_conv2d_f64(int64_t N, int64_t C, int64_t H, int64_t W,
                      int64_t K, int64_t R, int64_t S,
                      int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                      int64_t dh, int64_t dw, int64_t groups, int layout,
                      const double *x, const double *w, double *y, double *a,
                      int nthreads)
{
    if (N < 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || R <= 0 || S <= 0) return -1;
    if (sh <= 0 || sw <= 0 || ph < 0 || pw < 0 || dh <= 0 || dw <= 0 || groups <= 0) return -1;
    if (C % groups != 0 || K % groups != 0 || (layout != 0 && layout != 1)) return -1;
    const int64_t Cg = C / groups, Kg = K / groups;
    const int64_t OH = out_extent(H, ph, dh, R, sh);
    const int64_t OW = out_extent(W, pw, dw, S, sw);
    const int64_t pairs = N * K;
    (void)nthreads;

#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1)
#endif
    for (int64_t nk = 0; nk < pairs; ++nk) {
        const int64_t n = nk / K, k = nk % K;
        const int64_t c0 = (k / Kg) * Cg;
        for (int64_t p = 0; p < OH; ++p) {
            for (int64_t q = 0; q < OW; ++q) {
                double acc = 0.0, aacc = 0.0;
                for (int64_t c = 0; c < Cg; ++c) {
                    for (int64_t r = 0; r < R; ++r) {
                        const int64_t hi = p * sh - ph + r * dh;
                        if (hi < 0 || hi >= H) continue;
                        for (int64_t t = 0; t < S; ++t) {
                            const int64_t wi = q * sw - pw + t * dw;
                            if (wi < 0 || wi >= W) continue;
                            const double xv = x[x_at(layout, n, c0 + c, hi, wi, C, H, W)];
                            const double wv = w[w_at(layout, k, c, r, t, Cg, R, S)];
                            acc += xv * wv;
                            aacc += fabs(xv) * fabs(wv);
                        }
                    }
                }
                y[y_at(layout, n, k, p, q, K, OH, OW)] = acc;
                if (a) a[y_at(layout, n, k, p, q, K, OH, OW)] = aacc;
            }
        }
    }
    return 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
