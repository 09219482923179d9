/*
 * ROCKET transform oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  The product path (the HIP library and its Python
 * binding) never calls it, and this file shares no code, header or table
 * with that path.
 *
 * What it computes (CUROCKET paper, Sec. 2.1 "ROCKET" and Sec. 3.2
 * "Implementing CUROCKET"):
 *   every kernel k has a length l, weights w[0..l-1], a bias b, a dilation d
 *   and a zero padding p.  Convolving it with a series x of length L is a
 *   run of dot products, one per output position t = 0 .. O-1 with
 *       O   = L + 2p - (l-1) d                (number of dot products)
 *       y_t = b + sum_j w[j] * xz[t - p + j d]
 *   where xz is x with zeros outside [0, L) (the zero padding of Sec. 2.1).
 *   Two features come out of the run of y_t:
 *       PPV = |{t : y_t > 0}| / O   (proportion of positive values, divided by
 *                                    the number of dot products as Sec. 3.2 says)
 *       MAX = max_t y_t.
 *   Feature layout: F[i, 2k] = PPV, F[i, 2k+1] = MAX, in kernel order.
 *
 * Readings where the paper is silent (listed with reasons in the design notes):
 *   - cross-correlation orientation: tap j multiplies xz[t - p + j d];
 *   - "positive" is strict (y > 0);
 *   - evaluation in fp64 on the fp32 inputs (the paper notes that rounding
 *     near zero moves PPV slightly between devices, Sec. 5).
 *
 * Besides F it returns, per (row, kernel), the integer positive count and a
 * certified interval for the count that any fp32 evaluation of the same sums
 * can produce, in any summation order, with or without fused multiply-add:
 *       beta_t = gamma_{l+1} * (|b| + sum_j |w[j] xz[..]|) + (l+1) * 2^-126
 *       cnt_lo = |{t : y_t >  beta_t}|,  cnt_hi = |{t : y_t > -beta_t}|
 * with gamma_m = m u / (1 - m u), u = 2^-24 (the standard error bound of a
 * floating-point dot product of m terms; the 2^-126 term covers flushing of
 * subnormal intermediates).  beta_max = max_t beta_t bounds the error of MAX.
 *
 * Optional third feature, MPV (mean of the positive values; Sec. 5 names it
 * as one that fuses into the same pass because it does not depend on where
 * in the series the values fall):
 *       MPV = sum_{t : y_t > 0} y_t / |{t : y_t > 0}|,  0 when no y_t > 0.
 * Its certified range for an fp32 evaluation (values within beta_t of y_t,
 * any of the outputs within beta_t of zero counted either way, the positive
 * values summed in fp32 in any order, then one rounded division):
 *       sure  = {t : y_t > beta_t},   maybe = {t : |y_t| <= beta_t}
 *       mpv_lo = sum_sure (y_t - beta_t) (1 - gamma_c) (1 - u) / cnt_hi
 *       mpv_hi = (sum_sure (y_t + beta_t) + sum_maybe 2 beta_t)
 *                (1 + gamma_c) (1 + u) / cnt_lo
 * with c = cnt_hi; when cnt_lo = 0 the range is [0, max_maybe 2 beta_t
 * (1 + gamma_c)(1 + u)].
 *
 * Multivariate series (Sec. 3.3): a series has C channels, x_c[0..L-1].
 * Each kernel reads its own subset of channels, channel_count[k] of them
 * with ids channel_index[k*C + s], s < channel_count[k], and has one row
 * of weights per channel it reads; its dot product sums over those channels
 * and taps:
 *       y_t = b + sum_s sum_j w[s][j] * xz_{c_s}[t - p + j d]
 * (a univariate set is the case C = 1, every kernel reading channel 0).
 * beta_t then counts all channel_count * l products:
 *       beta_t = gamma_{m+1} (|b| + sum |w x|) + (m+1) 2^-126,  m = count * l.
 *
 * Plain loops: rows -> kernels -> t -> channels -> j.  No SIMD intrinsics,
 * no fast-math.  OpenMP only splits rows across threads (for timing the CPU
 * baseline).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_OK = 0, ORACLE_ERR_ARG = -1, ORACLE_ERR_LENGTH = -2 };

static double gamma_m(int m) {
    const double u = ldexp(1.0, -24);
    return (m * u) / (1.0 - m * u);
}

/* Number of dot products of one kernel on a series of length L (Sec. 2.1). */
int64_t oracle_output_length(int32_t L, int32_t length, int32_t dilation, int32_t padding) {
    return (int64_t)L + 2 * (int64_t)padding - (int64_t)(length - 1) * (int64_t)dilation;
}

/*
 * X        : fp32 [n_rows_total, C, L] row-major (C = n_channels; C = 1 for
 *            univariate series, [n_rows_total, L]).
 * rows     : optional list of n_out row indices into X (NULL: rows 0..n_out-1).
 * kernels  : SoA arrays of K kernels; weights of kernel k, channel slot s,
 *            tap j at weights[(k*C + s)*wstride + j] (wstride >= length).
 * channel_count, channel_index : per kernel, the channels it reads (see
 *            above); both may be NULL when C == 1.
 * F        : fp64 [n_out, 2K]  (PPV, MAX interleaved per kernel).
 * cnt, cnt_lo, cnt_hi : int64 [n_out, K] (may be NULL).
 * beta_max : fp64 [n_out, K] (may be NULL).
 * mpv, mpv_lo, mpv_hi : fp64 [n_out, K] (may be NULL).
 * nthreads : OpenMP threads (<= 0: runtime default).
 */
int oracle_transform_mc(const float *X, int64_t n_rows_total, const int64_t *rows, int64_t n_out,
                        int32_t C, int32_t L, int32_t K, const int32_t *length,
                        const int32_t *dilation, const int32_t *padding, const float *bias,
                        const float *weights, int32_t wstride, const int32_t *channel_count,
                        const int32_t *channel_index, double *F, int64_t *cnt, int64_t *cnt_lo,
                        int64_t *cnt_hi, double *beta_max, double *mpv, double *mpv_lo,
                        double *mpv_hi, int nthreads) {
    if (!X || !length || !dilation || !padding || !bias || !weights || !F) return ORACLE_ERR_ARG;
    if (C < 1 || L < 1 || K < 1 || n_out < 0 || wstride < 1) return ORACLE_ERR_ARG;
    if (C > 1 && (!channel_count || !channel_index)) return ORACLE_ERR_ARG;
    for (int32_t k = 0; k < K; ++k) {
        if (length[k] < 1 || length[k] > wstride || dilation[k] < 1 || padding[k] < 0)
            return ORACLE_ERR_ARG;
        if (oracle_output_length(L, length[k], dilation[k], padding[k]) < 1) return ORACLE_ERR_LENGTH;
        if (C > 1) {
            if (channel_count[k] < 1 || channel_count[k] > C) return ORACLE_ERR_ARG;
            for (int32_t s = 0; s < channel_count[k]; ++s)
                if (channel_index[(int64_t)k * C + s] < 0 || channel_index[(int64_t)k * C + s] >= C)
                    return ORACLE_ERR_ARG;
        }
    }
    if (rows) {
        for (int64_t r = 0; r < n_out; ++r)
            if (rows[r] < 0 || rows[r] >= n_rows_total) return ORACLE_ERR_ARG;
    } else if (n_out > n_rows_total) {
        return ORACLE_ERR_ARG;
    }
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_out; ++r) {
        const int64_t row = rows ? rows[r] : r;
        const float *xrow = X + row * (int64_t)C * L;
        for (int32_t k = 0; k < K; ++k) {
            const int32_t len = length[k], d = dilation[k], p = padding[k];
            const int32_t nch = C > 1 ? channel_count[k] : 1;
            const double b = (double)bias[k];
            const int64_t O = oracle_output_length(L, len, d, p);
            const double g = gamma_m(nch * len + 1);
            const double tiny = (nch * len + 1) * ldexp(1.0, -126);
            int64_t positive = 0, lo = 0, hi = 0;
            double mx = -INFINITY, bmax = 0.0;
            double pos_sum = 0.0, sure_lo = 0.0, sure_hi = 0.0, maybe = 0.0, maybe_max = 0.0;
            for (int64_t t = 0; t < O; ++t) {
                double y = b;
                double mag = fabs(b);
                for (int32_t s = 0; s < nch; ++s) {
                    const int32_t c = C > 1 ? channel_index[(int64_t)k * C + s] : 0;
                    const float *x = xrow + (int64_t)c * L;
                    const float *w = weights + ((int64_t)k * C + s) * wstride;
                    for (int32_t j = 0; j < len; ++j) {
                        const int64_t m = t - p + (int64_t)j * d;
                        const double xv = (m >= 0 && m < L) ? (double)x[m] : 0.0;
                        y += (double)w[j] * xv;
                        mag += fabs((double)w[j] * xv);
                    }
                }
                const double beta = g * mag + tiny;
                if (y > 0.0) {
                    ++positive;
                    pos_sum += y;
                }
                if (y > beta) {
                    ++lo;
                    sure_lo += y - beta;
                    sure_hi += y + beta;
                } else if (y > -beta) {
                    maybe += 2.0 * beta;
                    if (2.0 * beta > maybe_max) maybe_max = 2.0 * beta;
                }
                if (y > -beta) ++hi;
                if (y > mx) mx = y;
                if (beta > bmax) bmax = beta;
            }
            F[r * 2 * (int64_t)K + 2 * k] = (double)positive / (double)O;
            F[r * 2 * (int64_t)K + 2 * k + 1] = mx;
            if (cnt) cnt[r * (int64_t)K + k] = positive;
            if (cnt_lo) cnt_lo[r * (int64_t)K + k] = lo;
            if (cnt_hi) cnt_hi[r * (int64_t)K + k] = hi;
            if (beta_max) beta_max[r * (int64_t)K + k] = bmax;
            if (mpv) mpv[r * (int64_t)K + k] = positive > 0 ? pos_sum / (double)positive : 0.0;
            if (mpv_lo || mpv_hi) {
                const double u = ldexp(1.0, -24);
                const double gs = gamma_m((int)(hi > 0 ? hi : 1));
                double mlo, mhi;
                if (lo > 0) {
                    mlo = sure_lo * (1.0 - gs) * (1.0 - u) / (double)hi;
                    mhi = (sure_hi + maybe) * (1.0 + gs) * (1.0 + u) / (double)lo;
                } else {
                    mlo = 0.0;
                    mhi = maybe_max * (1.0 + gs) * (1.0 + u);
                }
                if (mpv_lo) mpv_lo[r * (int64_t)K + k] = mlo;
                if (mpv_hi) mpv_hi[r * (int64_t)K + k] = mhi;
            }
        }
    }
    return ORACLE_OK;
}

/* Univariate series [n_rows_total, L]: the multichannel loop with C = 1. */
int oracle_transform(const float *X, int64_t n_rows_total, const int64_t *rows, int64_t n_out,
                     int32_t L, int32_t K, const int32_t *length, const int32_t *dilation,
                     const int32_t *padding, const float *bias, const float *weights,
                     int32_t wstride, double *F, int64_t *cnt, int64_t *cnt_lo,
                     int64_t *cnt_hi, double *beta_max, double *mpv, double *mpv_lo,
                     double *mpv_hi, int nthreads) {
    return oracle_transform_mc(X, n_rows_total, rows, n_out, 1, L, K, length, dilation, padding,
                               bias, weights, wstride, NULL, NULL, F, cnt, cnt_lo, cnt_hi, beta_max,
                               mpv, mpv_lo, mpv_hi, nthreads);
}

/* Threads the OpenMP runtime would use (reported with the CPU baseline). */
int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
