/*
 * rocket.h -- C ABI of the MI355X (gfx950) ROCKET transform library.
 *
 * ROCKET (CUROCKET paper, Sec. 2.1): n_kernels random convolution kernels,
 * each with its own length, weights, bias, dilation and zero padding, are
 * slid over every series; every (series, kernel) pair yields two features,
 * the proportion of positive values (PPV) and the maximum (MAX) of the run
 * of dot products.  Sec. 3.2 normalises the positive count by the number of
 * dot products.
 *
 * Definitions used throughout (Sec. 2.1):
 *   O_k   = L + 2 p_k - (l_k - 1) d_k                  number of dot products
 *   y_t   = b_k + sum_{j<l_k} w_k[j] * xz[t - p_k + j d_k],  t = 0 .. O_k-1,
 *           xz = the series with zeros outside [0, L)
 *   F[i, 2k]   = |{t : y_t > 0}| / O_k   (PPV, computed as (float)count/(float)O_k)
 *   F[i, 2k+1] = max_t y_t                (MAX)
 *
 * Memory and threading rules for every entry point:
 *   - X (n x L fp32, row-major, contiguous) and F (n x 2 n_kernels fp32,
 *     row-major; n x 3 n_kernels with the MPV feature) are caller-owned
 *     DEVICE memory on the current HIP device (rocket_transform_host takes
 *     host memory instead).
 *     The library never frees them.  F is fully overwritten.
 *   - Kernel sets (rocket_kernels) live in HOST memory.
 *   - Series values (X, and the training set of rocket_minirocket_fit) and
 *     kernel weights and biases must be finite: no NaN, no infinity.  The
 *     device code compares and takes maxima under that assumption, so the
 *     features of a series that holds a NaN or an infinity are unspecified
 *     (they may differ between row layouts and call sizes).  Nothing checks
 *     the values.
 *   - Every argument is validated on the host before any device work; an
 *     invalid call returns an error and touches nothing.
 *   - No C++ exception crosses this boundary.
 *   - Device work is asynchronous on the given HIP stream (NULL = the null
 *     stream) unless a function says otherwise.
 */
#ifndef ROCKET_MI355X_H
#define ROCKET_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ROCKET_OK = 0,
    ROCKET_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad kernel field */
    ROCKET_ERR_LENGTH = -2,      /* a kernel has O_k < 1 (or O_k >= 2^24) for this L */
    ROCKET_ERR_OOM = -3,         /* host or device allocation failed */
    ROCKET_ERR_HIP = -4,         /* a HIP runtime call or kernel launch failed */
    ROCKET_ERR_INTERNAL = -5,    /* should not happen; a bug */
    ROCKET_ERR_SCRATCH = -6      /* the request needs more than the library's static scratch
                                    (rocket_transform_plan_noalloc) */
} rocket_status;

#define ROCKET_MAX_KERNEL_LENGTH 11 /* longest kernel; weights row stride */

/*
 * A kernel set in structure-of-arrays form (Sec. 2.1 kernel parameters).
 *   length[k]   in [1, 11]       (generated kernels use 7, 9, 11)
 *   dilation[k] >= 1
 *   padding[k]  >= 0             (generated: 0 or (length-1)*dilation/2)
 *   bias[k]     fp32
 *   max_len     weights row stride, in [length max, 11]; generated sets use 11
 *   input_length the series length the set was generated for (informational
 *               for hand-built sets; the transform takes L explicitly)
 * Univariate sets (n_channels 0 or 1; channel_count and channel_index may be
 * NULL): weights[k*max_len + j], j < length[k]; entries beyond length[k] are
 * ignored (the generator writes zeros there).
 * Multivariate sets (Sec. 3.3; series have n_channels = C channels, C in
 * [2, 32]): kernel k reads channel_count[k] channels (in [1, C]) with ids
 * channel_index[k*C + s], s < channel_count[k] (distinct, in [0, C)), and
 * has one weight row per channel it reads: weights[(k*C + s)*max_len + j].
 * Its dot product sums over those channels and taps.
 */
typedef struct {
    int32_t n_kernels;
    int32_t input_length;
    int32_t max_len;
    int32_t *length;
    int32_t *dilation;
    int32_t *padding;
    float *bias;
    float *weights;
    int32_t n_channels;
    int32_t *channel_count;
    int32_t *channel_index;
} rocket_kernels;

#define ROCKET_MAX_CHANNELS 32

/*
 * Generate n_kernels ROCKET kernels for series of length input_length
 * (Sec. 2.1): length uniform on {7, 9, 11}; weights standard normal, then
 * the kernel's mean subtracted (fp64, stored fp32); bias uniform on [-1, 1);
 * dilation floor(2^x), x uniform on [0, A), A = log2((L-1)/(length-1)),
 * capped at (L-1)/(length-1); padding (length-1)*dilation/2 with
 * probability 1/2, else 0.
 * Random numbers: kernel k, draw slot s in 0..15, is element k*16 + s of the
 * SplitMix64 sequence started at `seed` (Steele, Lea, Flood 2014); uniforms
 * take the top 53 bits; normals come from the Box-Muller transform
 * (slots 1..12, six pairs).  Slot 0: length, 13: bias, 14: dilation,
 * 15: padding (top bit).  The result depends only on (seed, k, input_length),
 * so a set of K kernels is a prefix of the set of K' > K kernels.
 * Host only; never touches a GPU.
 *
 * out: filled with library-owned host arrays (max_len = 11); release them
 *      with rocket_free_kernels.  On error *out is zeroed.
 * Errors: ROCKET_ERR_INVALID_ARG for out == NULL, n_kernels < 1 or
 *         input_length < 11 (some length would have no admissible dilation);
 *         ROCKET_ERR_OOM.
 */
rocket_status rocket_generate_kernels(uint64_t seed, int32_t n_kernels, int32_t input_length,
                                      rocket_kernels *out);

/*
 * Generate n_kernels multivariate ROCKET kernels (Sec. 3.3) for series of
 * n_channels channels (in [1, 32]) and length input_length: length, bias,
 * dilation and padding as rocket_generate_kernels; each kernel also reads
 * floor(2^x) channels, x uniform on [0, log2(C + 1)), clamped to [1, C],
 * chosen uniformly at random (ascending ids), with one weight row per
 * channel, standard normal and mean-centred over the kernel's taps.
 * Random numbers: kernel k, slot s reads element k*512 + s of the SplitMix64
 * sequence started at `seed`: slot 0 length, slot 1 channel count, slots
 * 2 .. C+1 a partial Fisher-Yates shuffle of 0..C-1 (step i swaps positions
 * i and i + floor(u (C - i)), computed exactly on the integer), slots 64 ..
 * Box-Muller pairs for the weights (normal q is channel slot q / 11, tap
 * q % 11), slot 509 bias, 510 dilation, 511 padding.  The result depends
 * only on (seed, k, input_length, n_channels).  Host only.
 * out: library-owned arrays (weights [K * C * 11], channel_index [K * C],
 *      -1 past each kernel's count); release with rocket_free_kernels.
 * Errors: ROCKET_ERR_INVALID_ARG (out NULL, n_kernels < 1, input_length < 11,
 *         n_channels outside [1, 32]); ROCKET_ERR_OOM.
 */
rocket_status rocket_generate_kernels_multi(uint64_t seed, int32_t n_kernels, int32_t input_length,
                                            int32_t n_channels, rocket_kernels *out);

/* Release arrays allocated by rocket_generate_kernels(_multi) and zero *k.
 * NULL-safe and idempotent.  Do not call on caller-built sets. */
void rocket_free_kernels(rocket_kernels *k);

/*
 * Opaque execution plan for one kernel set and one series length L, on the
 * HIP device that is current when it is created.  Creating a plan validates
 * the set, groups the kernels by (length, dilation, padding), builds the
 * device work tables and uploads them (synchronously).  A plan's tables are
 * immutable afterwards: transforms on different streams may share it.  The
 * one mutable part is the series-lane layout's feature buffer (short
 * series, see rocket_plan_create_ex), which transforms take in turn.
 */
typedef struct rocket_plan rocket_plan;

/*
 * Errors: ROCKET_ERR_INVALID_ARG (null pointers, n_kernels < 1, L < 1,
 *         max_len outside [1, 11], a length outside [1, max_len], dilation < 1,
 *         padding < 0); ROCKET_ERR_LENGTH (some O_k < 1, or some O_k above
 *         2^24 - 1); ROCKET_ERR_OOM; ROCKET_ERR_HIP.
 * On error *out is NULL.
 */
rocket_status rocket_plan_create(const rocket_kernels *k, int32_t L, rocket_plan **out);

/* Plan flags for rocket_plan_create_ex. */
#define ROCKET_PLAN_DEFAULT 0u
#define ROCKET_PLAN_DIRECT 1u  /* use the plain one-wavefront-per-pair kernel */
#define ROCKET_PLAN_CLAMPED 2u /* fused kernel with the long-series row layout */
#define ROCKET_PLAN_MPV 4u     /* a third feature per kernel: mean of positive values */
#define ROCKET_PLAN_TILED 8u   /* fused kernel with position tiles, also for short series */
#define ROCKET_PLAN_SERIES 16u /* series-lane layout for every call (short univariate series) */

/*
 * rocket_plan_create with flags.  ROCKET_PLAN_DIRECT selects the plain
 * kernel: one wavefront per (series, kernel) pair reading the series from
 * global memory.  It is slower and serves as a second GPU reference; the
 * default plan also falls back to it when a series does not fit one
 * workgroup's LDS even in the long-series layout.  ROCKET_PLAN_CLAMPED
 * forces the layout the default plan picks for long series: rows staged with
 * 512 zeros on each side, and the series offset of each block of tiles
 * clamped into those margins on the scalar unit (same results).
 * Short univariate series (L <= 128): calls with at least 4,096 series run
 * by default in the series-lane layout.  The 64 lanes of a wavefront take 64
 * series, staged position-major in LDS, so every MFMA computes one output
 * position for 4 kernels x 64 series and each lane reduces its own series;
 * the features go through a plan-owned buffer in slot order (allocated on
 * first use, at most 1 GiB, freed with the plan) and a permutation kernel
 * writes F; it runs on a stream the plan owns (non-blocking, default
 * priority) beside the next chunk of rows, and the call still completes on
 * hip_stream.  Same results as the position-tiled layout, which serves calls
 * with fewer series.  Transforms of one plan on different streams take turns
 * on that buffer (each waits for the previous one on the device).
 * ROCKET_PLAN_TILED keeps every call in the position-tiled layout;
 * ROCKET_PLAN_SERIES runs every call in the series-lane layout
 * (ROCKET_ERR_INVALID_ARG for multivariate sets or L > 128).
 * ROCKET_PLAN_DIRECT together with ROCKET_PLAN_CLAMPED or ROCKET_PLAN_TILED,
 * and ROCKET_PLAN_SERIES together with any of ROCKET_PLAN_DIRECT,
 * ROCKET_PLAN_CLAMPED and ROCKET_PLAN_TILED, are ROCKET_ERR_INVALID_ARG.
 * ROCKET_PLAN_MPV adds a third feature per kernel, the mean of the positive
 * values (MPV; the CUROCKET paper, Sec. 5, names it as a feature that does
 * not depend on time positions and so fuses into the same pass):
 *     MPV = sum_{t : y_t > 0} y_t / |{t : y_t > 0}|, 0 when no y_t > 0,
 * computed as the fp32 sum of the positive values divided in fp32 by the
 * count.  The feature matrix is then F [n, 3 n_kernels], per kernel
 * (PPV, MAX, MPV), and every entry point that writes F writes that layout
 * for this plan.  Unknown flag bits give ROCKET_ERR_INVALID_ARG.  Same
 * errors as rocket_plan_create otherwise.
 */
rocket_status rocket_plan_create_ex(const rocket_kernels *k, int32_t L, uint32_t flags,
                                    rocket_plan **out);

/* Free a plan's host and device memory.  NULL-safe.  The caller must make
 * sure no transform using the plan is still running. */
void rocket_plan_destroy(rocket_plan *p);

/*
 * Transform n series with a plan: X_dev [n, L] -> F_dev [n, f n_kernels],
 * features in the ORIGINAL kernel order, interleaved (PPV, MAX) per kernel
 * (f = 2), or (PPV, MAX, MPV) for a plan made with ROCKET_PLAN_MPV (f = 3).
 * Asynchronous on hip_stream (a hipStream_t; NULL = null stream).
 * n == 0 is a no-op.  Rows are independent; any row range of X may be
 * passed (row batching is the caller's loop over pointer offsets).
 * X must be finite (see the rules at the top of this file).
 * Work may run on streams the plan owns (the Toeplitz items' kernel of a
 * plan that has them, the series-lane chunks); it starts after the work
 * queued on hip_stream before the call, and hip_stream waits for all of it,
 * so the call behaves as one stream-ordered operation on hip_stream.
 * A call that runs the series-lane layout (short series, n >= 4,096 or
 * ROCKET_PLAN_SERIES) allocates the plan's feature buffer on first use, or
 * grows it (hipMalloc, at most 1 GiB; growing first waits for the device),
 * and makes the stream wait on the device for the previous call that used
 * the buffer.
 * The plan's device must be the current HIP device.
 * Errors: ROCKET_ERR_INVALID_ARG (p, X_dev or F_dev NULL with n > 0, n < 0,
 *         the current device not the plan's); ROCKET_ERR_OOM (the feature
 *         buffer); ROCKET_ERR_HIP (launch failure).
 */
rocket_status rocket_transform_plan(const rocket_plan *p, const float *X_dev, int64_t n,
                                    float *F_dev, void *hip_stream);

/*
 * rocket_transform_plan without any device allocation, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, layout, results
 * and errors as rocket_transform_plan, and the same kernels; it calls no
 * hipMalloc, hipFree or other allocating routine.  The one layout that needs
 * device memory beyond X and F, the series-lane layout of short series
 * (the slot-ordered feature buffer), uses instead a static device array of
 * ROCKET_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on every GPU
 * it runs on until the process ends; the series go through it in chunks of
 * at most 32 MiB of features (rows rounded down to a multiple of 64, at most
 * 8,192).  Every call on a GPU shares that GPU's array: calls that overlap in
 * time on one GPU (other streams, other plans) race on it, so the caller
 * orders them, e.g. on one stream (each call ends, on hip_stream, after its
 * last use of the array).  Nothing in the array needs clearing between calls.
 * The plan's device must be the current device.  The array's address on a
 * device is looked up on the first call there.
 * Errors: those of rocket_transform_plan, plus ROCKET_ERR_INVALID_ARG when
 *         the current device is not the plan's, ROCKET_ERR_SCRATCH when the
 *         features of 64 short series (2 or 3 floats per kernel slot) exceed
 *         half of the array (more than about 65,000 kernels), before any
 *         device work; F is then untouched.
 */
#define ROCKET_NOALLOC_SCRATCH_BYTES (64u << 20)
rocket_status rocket_transform_plan_noalloc(const rocket_plan *p, const float *X_dev, int64_t n,
                                            float *F_dev, void *hip_stream);

/*
 * One-shot transform: plan create + transform + plan destroy.  Returns after
 * the work on hip_stream has completed (it synchronises the stream before
 * freeing the plan).  Same errors as rocket_plan_create and
 * rocket_transform_plan.
 */
rocket_status rocket_transform(const float *X_dev, int64_t n, int32_t L, const rocket_kernels *k,
                               float *F_dev, void *hip_stream);

/*
 * Transform series held in HOST memory: X_host [n, L] -> F_host [n, f K]
 * (same layout and feature order as rocket_transform_plan; X_host must be
 * finite).  Rows go
 * through the device in batches of batch_rows (0: about n/8 rows, at most
 * 256 MiB of staging per buffer).  Each
 * batch's copy in, transform and copy out run on three HIP streams (the
 * caller's stream for the transform, two of the library's own for the
 * copies), double-buffered, so copies overlap the transform of the
 * neighbouring batches.  Returns when F_host is complete.  For overlap the
 * host buffers should be pinned (hipHostMalloc, or torch pin_memory);
 * pageable buffers work but the copies then serialise.  The function
 * allocates and frees its own device staging buffers (2 x batch of X and
 * of F).  n == 0 is a no-op.
 * The plan's device must be the current HIP device.
 * Errors: ROCKET_ERR_INVALID_ARG (p NULL, n < 0, X_host or F_host NULL with
 *         n > 0, batch_rows < 0, the current device not the plan's);
 *         ROCKET_ERR_OOM; ROCKET_ERR_HIP.
 */
rocket_status rocket_transform_host(const rocket_plan *p, const float *X_host, int64_t n,
                                    float *F_host, int64_t batch_rows, void *hip_stream);

/*
 * Plan facts for benchmarks and tests (host only).
 *   n_items      number of work items (groups of kernels sharing one bucket)
 *   n_buckets    number of distinct (length, dilation, padding) buckets
 *   mfma_per_row MFMA instructions one series costs (4x4x1 fp32 blocks;
 *                in the series-lane layout one MFMA serves 64 series, and
 *                this is the rounded share of one series)
 *   lds_bytes    LDS one workgroup uses (0 for the direct kernel)
 *   direct       1 if the plan runs the direct kernel, else 0
 *   clamped      1 if the fused kernel stages rows with 512 zeros on each
 *                side and clamps each block's series offset into them
 *                (chosen when the full zero margins of the padded kernels
 *                would not fit in LDS, or forced by ROCKET_PLAN_CLAMPED),
 *                else 0
 *   features_per_kernel  2 (PPV, MAX) or 3 (PPV, MAX, MPV); 0 for a
 *                MINIROCKET plan
 *   rows_per_block       series staged per workgroup (0 for the direct kernel)
 *   n_features   columns of F
 *   minirocket   1 for a MINIROCKET plan, else 0
 *   series_lane  1 if the plan runs the series-lane layout (for calls of at
 *                least 4,096 series, or every call with ROCKET_PLAN_SERIES);
 *                lds_bytes, rows_per_block and mfma_per_row then describe
 *                that layout
 *   valu_fma_per_row  fp32 FMA instructions (64 lanes each) one series costs
 *                in VALU items: the one or two kernels left over in a bucket
 *                of a univariate plan for series longer than 128 samples,
 *                run without MFMA
 *   toeplitz_items  work items of the shifted-kernel (Toeplitz) form: the
 *                one or two kernels left over in a bucket at a large
 *                dilation, run in a second kernel launch of each call
 *                (0: one launch per call)
 */
typedef struct {
    int64_t n_items;
    int64_t n_buckets;
    int64_t mfma_per_row;
    int64_t lds_bytes;
    int32_t direct;
    int32_t clamped;
    int32_t features_per_kernel;
    int32_t rows_per_block;
    int64_t n_features;
    int32_t minirocket;
    int32_t series_lane;
    int64_t valu_fma_per_row;
    int64_t toeplitz_items;
} rocket_plan_facts;

/* Fill *out with the plan's facts.  Errors: ROCKET_ERR_INVALID_ARG if p or
 * out is NULL. */
rocket_status rocket_plan_info(const rocket_plan *p, rocket_plan_facts *out);

/*
 * Host-side work tables of the fused kernel, for tests and tools (no GPU is
 * touched).  rocket_plan_tables_build validates like rocket_plan_create and
 * fills *out with library-owned arrays; free them with
 * rocket_plan_tables_free (NULL-safe, idempotent).
 *   items        n_items x item_words (16) int32, one row per work item:
 *                [variant, dilation, padding, outputs O, tiles, w_off,
 *                 k_off, cost, n_ch, ch_off, 0, 0, mask_lo, mask_hi,
 *                 inv_O (words 14-15: 1/O as an IEEE double,
 *                 little-endian)];
 *                n_ch channels, listed in chan[ch_off .. ch_off + n_ch),
 *                are the union of the channels the item's kernels read
 *                (1 and channel 0 for univariate sets); mask_lo |
 *                mask_hi << 32 holds the same channels as a bit mask;
 *                variant = 2 * ell_index + (G - 1), ell_index 0/1/2 for
 *                7/9/11 taps, G kernel groups of 4 slots (MFMA items), or
 *                6 + 2 * ell_index + (nk - 1) for VALU items of nk = 1 or 2
 *                kernels in slots 0..nk-1 (G = 1 packing; univariate plans
 *                for series longer than 128 samples), or
 *                12 + 2 * ell_index + (nk - 1) for Toeplitz items: nk = 1 or
 *                2 leftover kernels at a large dilation d, slot s holding
 *                kernel s / sigma (sigma = 4 / nk) shifted by s % sigma taps
 *                over ell + sigma - 1 taps, tiles = ceil(d / 64) chunks per
 *                super-tile of sigma * d outputs;
 *                the O outputs are computed in tiles = ceil(O / 64) tiles
 *                of 64 consecutive positions (lane l of tile k computes
 *                output 64k + l; lanes past O compute nothing that counts);
 *                cost = MFMA instructions per series (tiles x taps x G x n_ch;
 *                VALU items: (tiles x taps x nk + 1) / 2)
 *   wpk          packed weights, per item [n_ch][G][taps][4 slots]
 *   slot_bias, slot_kernel  per item 4G slots (kernel -1 = empty slot)
 *   order, split_begin, layout_off  item orders for the split counts in
 *                split_counts[n_layouts]: the items of variant v in split s
 *                of layout i (ns = split_counts[i] splits) are
 *                order[split_begin[layout_off[i] + v*ns + s] ..
 *                      split_begin[layout_off[i] + v*ns + s + 1]), v = 0..17
 *   halo_lo, halo_hi, row_stride  zero margins and LDS row length (floats)
 *                of the padded layout: a staged row is halo_lo zeros then
 *                the series (row_stride floats in all), and its right
 *                margin of halo_hi <= halo_lo zeros is the next row's left
 *                margin (every tap of every real output reads the zero-
 *                padded series)
 *   tail_pad     zeros staged after the last row of a workgroup: its right
 *                margin, then room for the lanes past O of an item's last
 *                tile, so that every read stays inside the staged memory
 */
typedef struct {
    int64_t n_items;
    int32_t item_words;
    int32_t n_channels;
    const int32_t *items;
    int64_t n_chan;
    const int32_t *chan;
    int64_t n_wpk;
    const float *wpk;
    int64_t n_slots;
    const float *slot_bias;
    const int32_t *slot_kernel;
    int64_t n_order;
    const int32_t *order;
    int64_t n_split_begin;
    const int32_t *split_begin;
    int32_t n_layouts;
    const int32_t *layout_off;
    const int32_t *split_counts;
    int32_t halo_lo;
    int32_t halo_hi;
    int32_t row_stride;
    int32_t tail_pad;
    void *internal;
} rocket_plan_tables;

rocket_status rocket_plan_tables_build(const rocket_kernels *k, int32_t L, rocket_plan_tables *out);
void rocket_plan_tables_free(rocket_plan_tables *t);

/*
 * MINIROCKET (Dempster, Schmidt and Webb, KDD 2021), the ROCKET variant the
 * CUROCKET paper (Sec. 5) names as one its principle carries over to:
 *   - 84 fixed kernels of 9 taps, one per choice of 3 of the 9 taps
 *     (choices in lexicographic order), weight 2 on the chosen taps and -1
 *     on the other six;
 *   - a fitted list of dilations d_i (ascending) and, per dilation, a number
 *     nf_i of features per kernel;
 *   - pair (dilation index i, kernel k) is padded (p = 4 d_i, O = L outputs)
 *     when i + k is even, else unpadded (p = 0, O = L - 8 d_i); its dot
 *     products are C_t = sum_j w_k[j] * xz[t - p + j d_i];
 *   - the pair has nf_i fitted biases b; each gives one feature, the
 *     proportion of positive values of C_t - b:
 *         PPV = |{t : C_t > b}| / O   (computed as (float)count / (float)O);
 *   - feature order: dilation index, then kernel, then bias.
 * Parameters live in HOST memory:
 *   input_length           L the parameters were fitted for
 *   n_dilations            number of dilations (>= 1)
 *   n_features             84 * sum(features_per_dilation)
 *   dilations[i]           ascending, >= 1, with L - 8 d_i >= 1
 *   features_per_dilation[i]  >= 0
 *   biases[f]              fp32, feature order
 */
typedef struct {
    int32_t input_length;
    int32_t n_dilations;
    int32_t n_features;
    int32_t *dilations;
    int32_t *features_per_dilation;
    float *biases;
} rocket_minirocket_params;

/*
 * Fit MINIROCKET to a training set X_train [n_train, L] (fp32, HOST memory,
 * row-major), L >= 9, for num_features requested features (>= 84; the fit
 * keeps 84 * floor(num_features / 84)):
 *   - dilations: the per-kernel feature count F = num_features / 84 is
 *     spread over T = min(F, 32) grid points floor(2^e), e evenly spaced on
 *     [0, log2((L-1)/8)] (e_0 = 0, e_{T-1} = the end point); equal values
 *     merge, their counts are scaled by F / T and truncated, and what is left
 *     of F is dealt one by one from the smallest dilation;
 *   - biases: pair (i, k) draws one training series e = (n_train * (v >> 11))
 *     >> 53, v = element i*84 + k of the SplitMix64 sequence started at
 *     `seed`; its padded dot products C_t, t = 0..L-1 (summed in fp64, tap by
 *     tap) are sorted, and the pair's biases are the quantiles at the
 *     positions q_m = frac(m * golden ratio) (m = 1, 2, ... over the whole
 *     feature list, rounded to fp32), by linear interpolation between order
 *     statistics, rounded to fp32.
 * X_train must be finite (see the rules at the top of this file).
 * Host only; never touches a GPU.
 * out: library-owned arrays; release with rocket_minirocket_free.  On error
 *      *out is zeroed.
 * Errors: ROCKET_ERR_INVALID_ARG (X_train or out NULL, n_train < 1, L < 9,
 *         num_features < 84); ROCKET_ERR_OOM.
 */
rocket_status rocket_minirocket_fit(const float *X_train, int64_t n_train, int32_t L,
                                    int32_t num_features, uint64_t seed,
                                    rocket_minirocket_params *out);

/* Release arrays allocated by rocket_minirocket_fit and zero *p.  NULL-safe
 * and idempotent.  Do not call on caller-built parameters. */
void rocket_minirocket_free(rocket_minirocket_params *p);

/*
 * Plan of the MINIROCKET transform for series of length m->input_length on
 * the current HIP device.  rocket_transform_plan and rocket_transform_host
 * with this plan write F [n, n_features] (PPV only, feature order above).
 * The plan groups the 4 kernels of a work item by (dilation, padding) and
 * computes each pair's dot products once for all of its biases.
 * flags: ROCKET_PLAN_DEFAULT or ROCKET_PLAN_CLAMPED (the long-series row
 *        layout, same results); anything else is ROCKET_ERR_INVALID_ARG.
 * Errors: ROCKET_ERR_INVALID_ARG (null pointers, a field outside the ranges
 *         above, n_features != 84 * sum(features_per_dilation));
 *         ROCKET_ERR_LENGTH (L - 8 d_i < 1 for some i, or L >= 2^24);
 *         ROCKET_ERR_OOM; ROCKET_ERR_HIP.  On error *out is NULL.
 */
rocket_status rocket_minirocket_plan_create(const rocket_minirocket_params *m, uint32_t flags,
                                            rocket_plan **out);

/* Static, human-readable name of a status code ("unknown status" otherwise). */
const char *rocket_status_string(rocket_status s);

/*
 * Checked builds, for debugging (a second library, librocket_checked.so,
 * compiled with ROCKET_CHECKED=1; the Python binding loads it when the
 * environment sets ROCKET_DEBUG=1).  Every entry point works as documented
 * above; in addition the device code checks every LDS tile read against the
 * bytes its workgroup staged, every feature store of the workgroup kernels
 * against the rows and columns of its launch, and every slot column the
 * series-lane permutation reads against the plan's slots.  A failed check
 * sets a flag and the access is redirected inside its buffer or skipped (the
 * features are then wrong, but no memory outside the buffers is touched).
 *   rocket_checked_build  1 in a checked build, 0 in the product library.
 *   rocket_check_flags    waits for the current device, stores the checks
 *                         that failed there since the last call in *flags
 *                         (bit 0: an LDS read, bit 1: a feature store,
 *                         bit 2: a slot column read; 0 = none) and clears
 *                         them.  The product library
 *                         stores 0 and touches no device.
 *                         Errors: ROCKET_ERR_INVALID_ARG (flags NULL);
 *                         ROCKET_ERR_HIP.
 */
int32_t rocket_checked_build(void);
rocket_status rocket_check_flags(uint32_t *flags);

#ifdef __cplusplus
}
#endif

#endif /* ROCKET_MI355X_H */
