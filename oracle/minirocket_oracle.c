/*
 * MINIROCKET transform oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  The product path never calls it, and this file
 * shares no code, header or table with that path.
 *
 * The CUROCKET paper (Sec. 5) names MINIROCKET (Dempster, Schmidt and Webb,
 * "MiniRocket: A Very Fast (Almost) Deterministic Transform for Time Series
 * Classification", KDD 2021) as a ROCKET variant that its principle carries
 * over to.  The paper does not restate MINIROCKET, so this follows the
 * published definition:
 *   - 84 fixed kernels of 9 taps, one per choice of 3 of the 9 taps
 *     (the choices in lexicographic order); weight 2 on the chosen taps and
 *     -1 on the other six (so the weights sum to 0);
 *   - for each dilation d of a fitted list (dilation index i) and kernel k,
 *     the dilated dot products  C_t = sum_j w[j] * xz[t - p + j d]  with the
 *     zero-padded series xz;  the pair (i, k) is padded (p = 4d, O = L
 *     outputs) when i + k is even, else unpadded (p = 0, O = L - 8d);
 *   - the pair has its own fitted biases b_q, q = 0 .. nf(i) - 1, and each
 *     gives one feature, the proportion of positive values of C_t - b_q:
 *         PPV = |{t : C_t > b_q}| / O;
 *   - feature order: dilation index, then kernel, then q.
 * Evaluation is in fp64 on the fp32 inputs.  Besides F it returns, per
 * feature, the count and a certified range for the count that any fp32
 * evaluation of the sums C_t (9 products, any order, with or without fused
 * multiply-add) followed by the exact comparison with b_q can give:
 *       beta_t = gamma_9 * sum_j |w[j] xz[..]| + 9 * 2^-126
 *       cnt_lo = |{t : C_t - b_q > beta_t}|,  cnt_hi = |{t : C_t - b_q > -beta_t}|
 * with gamma_m = m u / (1 - m u), u = 2^-24.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define MR_TAPS 9
#define MR_KERNELS 84

static double mr_gamma(int m) {
    const double u = ldexp(1.0, -24);
    return m * u / (1.0 - m * u);
}

/* The 3-of-9 tap choice of kernel k, in lexicographic order of (a, b, c). */
static void mr_choice(int k, int *a, int *b, int *c) {
    int idx = 0;
    for (int x = 0; x < MR_TAPS; ++x)
        for (int y = x + 1; y < MR_TAPS; ++y)
            for (int z = y + 1; z < MR_TAPS; ++z) {
                if (idx == k) {
                    *a = x;
                    *b = y;
                    *c = z;
                    return;
                }
                ++idx;
            }
}

/* Weights of kernel k: 2 on its three chosen taps, -1 elsewhere. */
void oracle_minirocket_weights(int k, double *w) {
    int a = 0, b = 0, c = 0;
    mr_choice(k, &a, &b, &c);
    for (int j = 0; j < MR_TAPS; ++j) w[j] = (j == a || j == b || j == c) ? 2.0 : -1.0;
}

/*
 * X: fp32 [n_rows_total, L]; rows: the m rows to evaluate (NULL: all).
 * dilations [n_dil], feats [n_dil] (features per kernel at that dilation),
 * biases [84 * sum(feats)] in feature order.
 * Outputs per evaluated row and feature: F (fp64 PPV), cnt, cnt_lo, cnt_hi.
 * Returns 0, -1 on bad arguments, -2 if a dilation leaves an unpadded pair
 * without outputs (L - 8d < 1).
 */
int oracle_minirocket_transform(const float *X, int64_t n_rows_total, const int64_t *rows, int64_t m,
                                int32_t L, int32_t n_dil, const int32_t *dilations, const int32_t *feats,
                                const float *biases, double *F, int64_t *cnt, int64_t *cnt_lo,
                                int64_t *cnt_hi, int threads) {
    if (!X || L < 1 || n_dil < 1 || !dilations || !feats || !biases || !F || !cnt || !cnt_lo || !cnt_hi)
        return -1;
    int64_t n_feat = 0;
    for (int32_t i = 0; i < n_dil; ++i) {
        if (dilations[i] < 1 || feats[i] < 0) return -1;
        if ((int64_t)L - 8 * (int64_t)dilations[i] < 1) return -2;
        n_feat += (int64_t)MR_KERNELS * feats[i];
    }
    if (threads > 0) {
#ifdef _OPENMP
        extern void omp_set_num_threads(int);
        omp_set_num_threads(threads);
#endif
    }
    const double g = mr_gamma(MR_TAPS);
    const double tiny = MR_TAPS * ldexp(1.0, -126);
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < m; ++r) {
        const int64_t row = rows ? rows[r] : r;
        const float *x = X + row * (int64_t)L;
        double *Fr = F + r * n_feat;
        int64_t *cr = cnt + r * n_feat, *lr = cnt_lo + r * n_feat, *hr = cnt_hi + r * n_feat;
        int64_t f0 = 0;
        for (int32_t i = 0; i < n_dil; ++i) {
            const int64_t d = dilations[i];
            for (int k = 0; k < MR_KERNELS; ++k) {
                double w[MR_TAPS];
                oracle_minirocket_weights(k, w);
                const int padded = ((i + k) % 2) == 0;
                const int64_t p = padded ? 4 * d : 0;
                const int64_t O = (int64_t)L + 2 * p - 8 * d;
                const int nf = feats[i];
                for (int q = 0; q < nf; ++q) cr[f0 + q] = lr[f0 + q] = hr[f0 + q] = 0;
                for (int64_t t = 0; t < O; ++t) {
                    double C = 0.0, a = 0.0;
                    for (int j = 0; j < MR_TAPS; ++j) {
                        const int64_t idx = t - p + j * d;
                        const double xv = (idx >= 0 && idx < L) ? (double)x[idx] : 0.0;
                        C += w[j] * xv;
                        a += fabs(w[j] * xv);
                    }
                    const double beta = g * a + tiny;
                    for (int q = 0; q < nf; ++q) {
                        const double y = C - (double)biases[f0 + q];
                        if (y > 0.0) ++cr[f0 + q];
                        if (y > beta) ++lr[f0 + q];
                        if (y > -beta) ++hr[f0 + q];
                    }
                }
                for (int q = 0; q < nf; ++q) Fr[f0 + q] = (double)cr[f0 + q] / (double)O;
                f0 += nf;
            }
        }
    }
    return 0;
}
