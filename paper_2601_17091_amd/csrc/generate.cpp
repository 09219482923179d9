// Seeded ROCKET kernel generator (Sec. 2.1 of the CUROCKET paper) and the
// small host-only entry points of the C ABI.
//
// Random numbers: SplitMix64 (Steele, Lea, Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014) used as a counter-based
// generator: element i of the sequence started at `seed` is
// mix64(seed + (i + 1) * 0x9E3779B97F4A7C15).  Kernel k owns elements
// [16k, 16k + 16), so kernels are independent of each other and of K.
// Normals: Box-Muller transform (Box and Muller, 1958).
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>

#include "rocket_internal.h"

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr int kDrawsPerKernel = 16;

uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// uniform on [0, 1) from the top 53 bits
double unit_closed_open(uint64_t v) { return (double)(v >> 11) * 0x1.0p-53; }
// uniform on (0, 1] (safe for log)
double unit_open_closed(uint64_t v) { return (double)((v >> 11) + 1) * 0x1.0p-53; }

}  // namespace

uint64_t rocket::splitmix64_at(uint64_t seed, uint64_t index) {
    return mix64(seed + (index + 1) * kGolden);
}

extern "C" rocket_status rocket_generate_kernels(uint64_t seed, int32_t n_kernels,
                                                 int32_t input_length, rocket_kernels *out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    if (n_kernels < 1 || input_length < ROCKET_MAX_KERNEL_LENGTH) return ROCKET_ERR_INVALID_ARG;
    const int32_t K = n_kernels, L = input_length, M = ROCKET_MAX_KERNEL_LENGTH;
    int32_t *length = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    int32_t *dilation = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    int32_t *padding = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    float *bias = (float *)std::calloc((size_t)K, sizeof(float));
    float *weights = (float *)std::calloc((size_t)K * M, sizeof(float));
    if (!length || !dilation || !padding || !bias || !weights) {
        std::free(length);
        std::free(dilation);
        std::free(padding);
        std::free(bias);
        std::free(weights);
        return ROCKET_ERR_OOM;
    }
    static const int32_t kLengths[3] = {7, 9, 11};
    const double two_pi = 6.283185307179586;  // nearest double to 2*pi
    for (int32_t k = 0; k < K; ++k) {
        uint64_t v[kDrawsPerKernel];
        for (int s = 0; s < kDrawsPerKernel; ++s)
            v[s] = mix64(seed + ((uint64_t)k * kDrawsPerKernel + (uint64_t)s + 1) * kGolden);
        // length: floor(3u) computed exactly on the 53-bit integer
        const int32_t len = kLengths[(3 * (v[0] >> 11)) >> 53];
        // weights: twelve normals from six Box-Muller pairs, first `len` used
        double z[12];
        for (int i = 0; i < 6; ++i) {
            const double u1 = unit_open_closed(v[1 + 2 * i]);
            const double u2 = unit_closed_open(v[2 + 2 * i]);
            const double r = std::sqrt(-2.0 * std::log(u1));
            const double th = two_pi * u2;
            z[2 * i] = r * std::cos(th);
            z[2 * i + 1] = r * std::sin(th);
        }
        double sum = 0.0;
        for (int j = 0; j < len; ++j) sum += z[j];
        const double mean = sum / len;
        for (int j = 0; j < len; ++j) weights[(int64_t)k * M + j] = (float)(z[j] - mean);
        // bias: uniform on [-1, 1)
        bias[k] = (float)(2.0 * unit_closed_open(v[13]) - 1.0);
        // dilation: floor(2^x), x ~ U(0, A), A = log2((L-1)/(len-1))
        const double A = std::log2((double)(L - 1) / (double)(len - 1));
        int64_t d = (int64_t)std::floor(std::pow(2.0, unit_closed_open(v[14]) * A));
        const int64_t dmax = (int64_t)(L - 1) / (len - 1);
        if (d > dmax) d = dmax;
        if (d < 1) d = 1;
        dilation[k] = (int32_t)d;
        // zero padding centring the kernel, with probability 1/2
        padding[k] = (v[15] >> 63) ? (int32_t)((len - 1) * d / 2) : 0;
        length[k] = len;
    }
    out->n_kernels = K;
    out->input_length = L;
    out->max_len = M;
    out->length = length;
    out->dilation = dilation;
    out->padding = padding;
    out->bias = bias;
    out->weights = weights;
    out->n_channels = 1;
    return ROCKET_OK;
}

// Multivariate kernels (Sec. 3.3): the stream layout of one kernel (element
// k*512 + slot of the SplitMix64 sequence started at `seed`).
namespace {
constexpr int kMcSlots = 512;
constexpr int kMcSubset = 2;    // slots 2 .. C+1: channel shuffle
constexpr int kMcNormals = 64;  // Box-Muller pairs of the weights
constexpr int kMcBias = 509, kMcDilation = 510, kMcPadding = 511;
}  // namespace

extern "C" rocket_status rocket_generate_kernels_multi(uint64_t seed, int32_t n_kernels,
                                                       int32_t input_length, int32_t n_channels,
                                                       rocket_kernels *out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    if (n_kernels < 1 || input_length < ROCKET_MAX_KERNEL_LENGTH || n_channels < 1 ||
        n_channels > ROCKET_MAX_CHANNELS)
        return ROCKET_ERR_INVALID_ARG;
    const int32_t K = n_kernels, L = input_length, M = ROCKET_MAX_KERNEL_LENGTH, C = n_channels;
    int32_t *length = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    int32_t *dilation = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    int32_t *padding = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    float *bias = (float *)std::calloc((size_t)K, sizeof(float));
    float *weights = (float *)std::calloc((size_t)K * C * M, sizeof(float));
    int32_t *count = (int32_t *)std::calloc((size_t)K, sizeof(int32_t));
    int32_t *index = (int32_t *)std::calloc((size_t)K * C, sizeof(int32_t));
    if (!length || !dilation || !padding || !bias || !weights || !count || !index) {
        std::free(length);
        std::free(dilation);
        std::free(padding);
        std::free(bias);
        std::free(weights);
        std::free(count);
        std::free(index);
        return ROCKET_ERR_OOM;
    }
    static const int32_t kLengths[3] = {7, 9, 11};
    const double two_pi = 6.283185307179586;  // nearest double to 2*pi
    const double log2_c1 = std::log2((double)(C + 1));
    for (int32_t k = 0; k < K; ++k) {
        auto draw = [&](int slot) {
            return mix64(seed + ((uint64_t)k * kMcSlots + (uint64_t)slot + 1) * kGolden);
        };
        const int32_t len = kLengths[(3 * (draw(0) >> 11)) >> 53];
        int64_t cnt = (int64_t)std::floor(std::pow(2.0, unit_closed_open(draw(1)) * log2_c1));
        if (cnt < 1) cnt = 1;
        if (cnt > C) cnt = C;
        // partial Fisher-Yates shuffle of 0..C-1, the first cnt entries ascending
        int32_t perm[ROCKET_MAX_CHANNELS];
        for (int32_t i = 0; i < C; ++i) perm[i] = i;
        for (int32_t i = 0; i < cnt; ++i) {
            const uint64_t v = draw(kMcSubset + i);
            const int32_t j = i + (int32_t)(((uint64_t)(C - i) * (v >> 11)) >> 53);
            const int32_t t = perm[i];
            perm[i] = perm[j];
            perm[j] = t;
        }
        std::sort(perm, perm + cnt);
        // normals: Box-Muller pairs; normal q is channel slot q / 11, tap q % 11
        const int n_pairs = (int)((cnt * M + 1) / 2);
        double z[ROCKET_MAX_CHANNELS * ROCKET_MAX_KERNEL_LENGTH + 1];
        for (int m = 0; m < n_pairs; ++m) {
            const double u1 = unit_open_closed(draw(kMcNormals + 2 * m));
            const double u2 = unit_closed_open(draw(kMcNormals + 2 * m + 1));
            const double r = std::sqrt(-2.0 * std::log(u1));
            const double th = two_pi * u2;
            z[2 * m] = r * std::cos(th);
            z[2 * m + 1] = r * std::sin(th);
        }
        for (int32_t s = 0; s < cnt; ++s) {
            double sum = 0.0;
            for (int j = 0; j < len; ++j) sum += z[s * M + j];
            const double mean = sum / len;
            for (int j = 0; j < len; ++j)
                weights[((int64_t)k * C + s) * M + j] = (float)(z[s * M + j] - mean);
        }
        bias[k] = (float)(2.0 * unit_closed_open(draw(kMcBias)) - 1.0);
        const double A = std::log2((double)(L - 1) / (double)(len - 1));
        int64_t d = (int64_t)std::floor(std::pow(2.0, unit_closed_open(draw(kMcDilation)) * A));
        const int64_t dmax = (int64_t)(L - 1) / (len - 1);
        if (d > dmax) d = dmax;
        if (d < 1) d = 1;
        dilation[k] = (int32_t)d;
        padding[k] = (draw(kMcPadding) >> 63) ? (int32_t)((len - 1) * d / 2) : 0;
        length[k] = len;
        count[k] = (int32_t)cnt;
        for (int32_t s = 0; s < C; ++s) index[(int64_t)k * C + s] = s < cnt ? perm[s] : -1;
    }
    out->n_kernels = K;
    out->input_length = L;
    out->max_len = M;
    out->length = length;
    out->dilation = dilation;
    out->padding = padding;
    out->bias = bias;
    out->weights = weights;
    out->n_channels = C;
    out->channel_count = count;
    out->channel_index = index;
    return ROCKET_OK;
}

extern "C" void rocket_free_kernels(rocket_kernels *k) {
    if (!k) return;
    std::free(k->length);
    std::free(k->dilation);
    std::free(k->padding);
    std::free(k->bias);
    std::free(k->weights);
    std::free(k->channel_count);
    std::free(k->channel_index);
    std::memset(k, 0, sizeof(*k));
}

extern "C" const char *rocket_status_string(rocket_status s) {
    switch (s) {
        case ROCKET_OK: return "ok";
        case ROCKET_ERR_INVALID_ARG: return "invalid argument";
        case ROCKET_ERR_LENGTH: return "a kernel has no dot products for this series length";
        case ROCKET_ERR_OOM: return "out of memory";
        case ROCKET_ERR_HIP: return "HIP runtime error";
        case ROCKET_ERR_INTERNAL: return "internal error";
        case ROCKET_ERR_SCRATCH: return "request exceeds the library's static scratch";
    }
    return "unknown status";
}
