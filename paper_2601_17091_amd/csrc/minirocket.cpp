// MINIROCKET (Dempster, Schmidt and Webb, KDD 2021), the ROCKET variant the
// CUROCKET paper (Sec. 5) names as one its principle carries over to: the
// host-side fit (dilations and quantile biases) and the host tables of a
// MINIROCKET plan.  Pure host code; no HIP calls.
//
// The 84 kernels have 9 taps, weight 2 on one choice of 3 taps and -1 on the
// other six (the choices in lexicographic order).  Pair (dilation index i,
// kernel k) is padded (p = 4d) when i + k is even, else unpadded.  Features
// run over dilation index, kernel, bias.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <new>
#include <vector>

#include "rocket_internal.h"

namespace {

// The 3-of-9 tap choices in lexicographic order.
struct Choices {
    int tap[rocket::kMrKernels][3];
    Choices() {
        int k = 0;
        for (int a = 0; a < rocket::kMrTaps; ++a)
            for (int b = a + 1; b < rocket::kMrTaps; ++b)
                for (int c = b + 1; c < rocket::kMrTaps; ++c) {
                    tap[k][0] = a;
                    tap[k][1] = b;
                    tap[k][2] = c;
                    ++k;
                }
    }
};

const Choices &choices() {
    static const Choices c;
    return c;
}

void kernel_weights(int k, double w[rocket::kMrTaps]) {
    for (int j = 0; j < rocket::kMrTaps; ++j) w[j] = -1.0;
    for (int s = 0; s < 3; ++s) w[choices().tap[k][s]] = 2.0;
}

// Dilations and features per kernel at each dilation: F features per kernel
// over T = min(F, 32) grid points floor(2^e), e evenly spaced on
// [0, log2((L-1)/8)], equal values merged and their counts scaled by F / T.
void fit_dilations(int32_t L, int32_t num_features, std::vector<int32_t> &dil,
                   std::vector<int32_t> &feats) {
    const int64_t F = num_features / rocket::kMrKernels;
    const int64_t T = std::min<int64_t>(F, 32);
    const double multiplier = (double)F / (double)T;
    const double max_exponent = std::log2((double)(L - 1) / (double)(rocket::kMrTaps - 1));
    std::vector<int32_t> raw;
    for (int64_t i = 0; i < T; ++i) {
        double e = 0.0;
        if (T > 1) e = (i == T - 1) ? max_exponent : (double)i * (max_exponent / (double)(T - 1));
        raw.push_back((int32_t)std::pow(2.0, e));
    }
    std::vector<int32_t> sorted = raw;
    std::sort(sorted.begin(), sorted.end());
    dil.clear();
    feats.clear();
    for (size_t i = 0; i < sorted.size();) {
        size_t j = i;
        while (j < sorted.size() && sorted[j] == sorted[i]) ++j;
        dil.push_back(sorted[i]);
        feats.push_back((int32_t)((double)(j - i) * multiplier));
        i = j;
    }
    int64_t rem = F;
    for (int32_t f : feats) rem -= f;
    for (size_t i = 0; rem > 0; i = (i + 1) % feats.size(), --rem) ++feats[i];
}

// Quantile position m (1-based): frac(m * golden ratio), rounded to fp32.
float quantile_position(int64_t m) {
    const double phi = (std::sqrt(5.0) + 1.0) / 2.0;
    const double v = (double)m * phi;
    return (float)(v - std::floor(v));
}

// Quantile of sorted values by linear interpolation between order
// statistics: position h = q (n - 1).
double quantile_linear(const std::vector<double> &s, double q) {
    const int64_t n = (int64_t)s.size();
    const double h = (double)(n - 1) * q;
    const int64_t lo = (int64_t)std::floor(h);
    if (lo >= n - 1) return s[n - 1];
    const double frac = h - (double)lo;
    return s[lo] + frac * (s[lo + 1] - s[lo]);
}

}  // namespace

extern "C" rocket_status rocket_minirocket_fit(const float *X_train, int64_t n_train, int32_t L,
                                               int32_t num_features, uint64_t seed,
                                               rocket_minirocket_params *out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    if (!X_train || n_train < 1 || L < rocket::kMrTaps || num_features < rocket::kMrKernels)
        return ROCKET_ERR_INVALID_ARG;
    try {
        std::vector<int32_t> dil, feats;
        fit_dilations(L, num_features, dil, feats);
        int64_t total = 0;
        for (int32_t f : feats) total += (int64_t)rocket::kMrKernels * f;
        std::vector<float> biases((size_t)total);
        std::vector<double> xz((size_t)L + 8 * (size_t)dil.back()), C((size_t)L);
        int64_t f = 0;
        for (size_t i = 0; i < dil.size(); ++i) {
            const int64_t d = dil[i];
            for (int k = 0; k < rocket::kMrKernels; ++k) {
                // the pair's training series and its padded dot products,
                // summed in fp64 tap by tap
                const uint64_t v = rocket::splitmix64_at(seed, (uint64_t)i * rocket::kMrKernels + (uint64_t)k);
                const int64_t e = (int64_t)(((unsigned __int128)n_train * (v >> 11)) >> 53);
                const float *x = X_train + e * (int64_t)L;
                std::fill(xz.begin(), xz.end(), 0.0);
                for (int32_t t = 0; t < L; ++t) xz[(size_t)(4 * d + t)] = (double)x[t];
                double w[rocket::kMrTaps];
                kernel_weights(k, w);
                std::fill(C.begin(), C.end(), 0.0);
                for (int j = 0; j < rocket::kMrTaps; ++j)
                    for (int32_t t = 0; t < L; ++t) C[(size_t)t] = C[(size_t)t] + w[j] * xz[(size_t)(j * d + t)];
                std::vector<double> s = C;
                std::sort(s.begin(), s.end());
                for (int32_t q = 0; q < feats[i]; ++q, ++f)
                    biases[(size_t)f] = (float)quantile_linear(s, (double)quantile_position(f + 1));
            }
        }
        out->dilations = (int32_t *)std::malloc(dil.size() * sizeof(int32_t));
        out->features_per_dilation = (int32_t *)std::malloc(feats.size() * sizeof(int32_t));
        out->biases = (float *)std::malloc(std::max<size_t>(1, biases.size()) * sizeof(float));
        if (!out->dilations || !out->features_per_dilation || !out->biases) {
            rocket_minirocket_free(out);
            return ROCKET_ERR_OOM;
        }
        std::memcpy(out->dilations, dil.data(), dil.size() * sizeof(int32_t));
        std::memcpy(out->features_per_dilation, feats.data(), feats.size() * sizeof(int32_t));
        std::memcpy(out->biases, biases.data(), biases.size() * sizeof(float));
        out->input_length = L;
        out->n_dilations = (int32_t)dil.size();
        out->n_features = (int32_t)total;
        return ROCKET_OK;
    } catch (const std::bad_alloc &) {
        rocket_minirocket_free(out);
        return ROCKET_ERR_OOM;
    } catch (...) {
        rocket_minirocket_free(out);
        return ROCKET_ERR_INTERNAL;
    }
}

extern "C" void rocket_minirocket_free(rocket_minirocket_params *p) {
    if (!p) return;
    std::free(p->dilations);
    std::free(p->features_per_dilation);
    std::free(p->biases);
    std::memset(p, 0, sizeof(*p));
}

namespace rocket {

rocket_status validate_minirocket(const rocket_minirocket_params *m) {
    if (!m || !m->dilations || !m->features_per_dilation || !m->biases) return ROCKET_ERR_INVALID_ARG;
    if (m->input_length < kMrTaps || m->n_dilations < 1) return ROCKET_ERR_INVALID_ARG;
    int64_t total = 0;
    for (int32_t i = 0; i < m->n_dilations; ++i) {
        if (m->dilations[i] < 1 || m->features_per_dilation[i] < 0) return ROCKET_ERR_INVALID_ARG;
        if (i > 0 && m->dilations[i] <= m->dilations[i - 1]) return ROCKET_ERR_INVALID_ARG;
        total += (int64_t)kMrKernels * m->features_per_dilation[i];
    }
    if (total != (int64_t)m->n_features || total < 1) return ROCKET_ERR_INVALID_ARG;
    if (m->input_length >= kMaxOutputs) return ROCKET_ERR_LENGTH;
    for (int32_t i = 0; i < m->n_dilations; ++i)
        if ((int64_t)m->input_length - 8 * (int64_t)m->dilations[i] < 1) return ROCKET_ERR_LENGTH;
    return ROCKET_OK;
}

rocket_status build_minirocket_plan(const rocket_minirocket_params *m, HostPlan *out) {
    try {
        HostPlan P;
        P.minirocket = true;
        P.L = m->input_length;
        P.n_kernels = kMrKernels;
        P.n_features = m->n_features;
        const int64_t L = m->input_length;
        const int64_t dmax = m->dilations[m->n_dilations - 1];
        // padded pairs reach 4d on each side; lanes past O read up to 63
        // positions further (tail_pad)
        if (L + 8 * dmax > ((int64_t)1 << 30)) {
            P.halo_lo = P.halo_hi = P.row_stride = 0;
        } else {
            // rows share their zero margins, as in ROCKET plans
            P.halo_lo = P.halo_hi = (int32_t)(4 * dmax);
            P.row_stride = (int32_t)(L + 4 * dmax);
        }
        P.tail_pad = P.halo_hi + kTile;
        P.n_buckets = 2 * (int64_t)m->n_dilations;
        const float inf = std::numeric_limits<float>::infinity();
        int64_t fstart = 0;  // first feature of the current dilation
        for (int32_t i = 0; i < m->n_dilations; ++i) {
            const int32_t d = m->dilations[i];
            const int32_t nf = m->features_per_dilation[i];
            for (int padded = 1; padded >= 0 && nf > 0; --padded) {
                const int32_t p = padded ? 4 * d : 0;
                const int64_t O = L + 2 * (int64_t)p - 8 * (int64_t)d;
                const int64_t n_tiles = (O + kTile - 1) / kTile;
                // kernels k = 2 kappa + par have i + k even (padded) or odd
                const int par = padded ? (i & 1) : ((i + 1) & 1);
                for (int32_t q0 = 0; q0 < nf;) {
                    // chunks of 8 biases; a remainder of 4 takes a chunk of 4,
                    // one of 1..3 a chunk of 3 (5..7: 8)
                    const int32_t rest = nf - q0;
                    const int32_t nq = rest > kMrQSmall ? kMrQLarge : (rest == kMrQSmall ? kMrQSmall : kMrQTiny);
                    ItemDesc it;
                    std::memset(&it, 0, sizeof(it));
                    it.variant = mr_variant(par, nq);
                    it.d = d;
                    it.p = p;
                    it.O = (int32_t)O;
                    it.n_tiles = (int32_t)n_tiles;
                    it.w_off = (int32_t)fstart;
                    it.k_off = q0;
                    it.n_ch = nf;
                    // per series: one compare per (kernel, bias, output)
                    // plus the shared dot products (about 3 per kernel)
                    it.cost = (int32_t)std::min<int64_t>(n_tiles * kMrKappa * (nq + 3), INT32_MAX);
                    it.t_off = (int32_t)P.thr.size();
                    it.nq = nq;
                    it.inv_O = 1.0 / (double)O;
                    // biases [kappa][q]; +inf for the dummies past nf
                    for (int kappa = 0; kappa < kMrKappa; ++kappa)
                        for (int32_t q = 0; q < nq; ++q)
                            P.thr.push_back(q0 + q < nf ? m->biases[fstart + (int64_t)(2 * kappa + par) * nf + q0 + q]
                                                        : inf);
                    P.items.push_back(it);
                    q0 += std::min(nq, rest);
                }
            }
            fstart += (int64_t)kMrKernels * nf;
        }
        P.n_variants = kMrNumVariants;
        build_item_orders(P);
        *out = std::move(P);
        return ROCKET_OK;
    } catch (const std::bad_alloc &) {
        return ROCKET_ERR_OOM;
    } catch (...) {
        return ROCKET_ERR_INTERNAL;
    }
}

}  // namespace rocket
