// Seeded ROCKET kernel generator (Sec. 2.1 of the CUROCKET paper) and the
// small host-only entry points of the C ABI.
//
// Random numbers: SplitMix64 (Steele, Lea, Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014) used as a counter-based
// generator: element i of the sequence started at `seed` is
// mix64(seed + (i + 1) * 0x9E3779B97F4A7C15).  Kernel k owns elements
// [16k, 16k + 16), so kernels are independent of each other and of K.
// Normals: Box-Muller transform (Box and Muller, 1958).
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
    return ROCKET_OK;
}

extern "C" void rocket_free_kernels(rocket_kernels *k) {
    if (!k) return;
    std::free(k->length);
    std::free(k->dilation);
    std::free(k->padding);
    std::free(k->bias);
    std::free(k->weights);
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
    }
    return "unknown status";
}
