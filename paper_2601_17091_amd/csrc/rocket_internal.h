// Internal layout shared by the host planner (plan.cpp) and the gfx950
// kernels (transform.hip).  Not part of the public ABI.
#pragma once

#include <cstdint>
#include <vector>

#include "rocket.h"

namespace rocket {

// The fused MFMA path keeps the three kernel lengths ROCKET draws
// (Sec. 2.1: 7, 9, 11).  A hand-built kernel of another length is run as the
// next supported length with zero weights on the extra taps.
constexpr int kNumEll = 3;
constexpr int kEllValues[kNumEll] = {7, 9, 11};

inline int ell_index_for(int length) { return length <= 7 ? 0 : (length <= 9 ? 1 : 2); }

// Wavefront size on CDNA4 and the number of kernel slots one
// v_mfma_f32_4x4x1_16b_f32 block holds (its 4 A-matrix rows).
constexpr int kWave = 64;
constexpr int kSlotsPerGroup = 4;
constexpr int kMaxGroups = 2;  // a work item holds 4 or 8 kernels of one bucket

// Outputs are computed in tiles of 64 consecutive positions: lane l of a
// wavefront computes output 64*k + l of tile k for every kernel slot of the
// item.  A block runs kTilesPerBlock[G-1] tiles at once (the independent
// MFMA accumulation chains of a wavefront: tiles x groups = 8).
constexpr int kTile = kWave;
constexpr int kTilesPerBlock[kMaxGroups] = {8, 4};
constexpr int kMaxTilesPerBlock = 8;

// Clamped row layout (long series): each staged row carries this many zeros
// on each side; the series index of a block's first lane is clamped into
// [-kClampMargin, L] on the scalar unit, so a block whose 64*NT positions all
// fall outside the series reads zeros from a margin.
constexpr int kClampMargin = kTile * kMaxTilesPerBlock;

// The fused kernel runs multichannel items over a 64-bit channel mask.
static_assert(ROCKET_MAX_CHANNELS <= 64, "channel masks are 64 bits");

// Every output of an item is computed by exactly one lane of one tile; lanes
// of the last tile past O start from -inf and change no feature.
constexpr int64_t kMaxOutputs = (int64_t)1 << 24;  // O must stay below 2^24

// One work item: up to 4*G kernels that share (length, dilation, padding),
// so every slot has the same O outputs and reads the same series values.
// MINIROCKET items use d, p, O, n_tiles, cost, t_off, nq and inv_O as named,
// and three fields for their feature numbering: w_off = the first feature of
// the item's dilation, k_off = the item's first bias (of each kernel), n_ch =
// the dilation's features per kernel; variant = mr_variant(parity, nq).
struct alignas(16) ItemDesc {
    int32_t variant;   // ell_index * 2 + (G - 1)
    int32_t d;         // dilation
    int32_t p;         // padding
    int32_t O;         // number of dot products (outputs)
    int32_t n_tiles;   // ceil(O / 64); Toeplitz items: chunks per super-tile, ceil(d / 64)
    int32_t w_off;     // first packed weight: [n_ch][G][ell][4] floats
    int32_t k_off;     // first slot entry: kernel ids and biases, [4G]
    int32_t cost;      // MFMA instructions per series (scheduling weight)
    int32_t n_ch;      // channels the item's kernels read (their union; 1 if univariate)
    int32_t ch_off;    // first entry of the item's channel list
    int32_t t_off;     // MINIROCKET: first threshold, [kMrKappa][nq] floats
    int32_t nq;        // MINIROCKET: thresholds per kernel in this item (kMrQTiny, kMrQSmall or kMrQLarge)
    uint32_t ch_mask[2];  // multichannel: the item's channels as a bit mask (lo, hi words)
    double inv_O;      // 1 / O rounded to double (exact PPV, see transform.hip)
};
static_assert(sizeof(ItemDesc) == 64, "ItemDesc must stay 64 bytes");
constexpr int kItemWords = (int)(sizeof(ItemDesc) / sizeof(int32_t));

// Item orders for a few split counts.  Within a layout with `nsplit` splits
// the items are grouped by variant, so that every workgroup runs one code
// variant: the items of variant v in split s are
// order[split_begin[v*nsplit + s] .. split_begin[v*nsplit + s + 1]).
// Variants 0..5 are MFMA items, 2 * ell_index + (G - 1).  Variants 6..11 are
// VALU items: the one or two leftover kernels of a bucket (nk of them), run
// with plain fp32 FMA instead of a 4-slot MFMA group that would be mostly
// empty, 6 + 2 * ell_index + (nk - 1); their weights keep the 4-slot packing
// of a one-group item.
constexpr int kNumMfmaVariants = 2 * kNumEll;
constexpr int kNumVariants = 6 * kNumEll;
constexpr int kValuVariant0 = kNumMfmaVariants;

// Variants 12..17 are Toeplitz items: the one or two kernels left over in a
// bucket at a large dilation d, 12 + 2 * ell_index + (nk - 1).  The 4 slots
// of one MFMA group hold the same kernel shifted by sigma = 4 / nk taps:
// slot s is kernel s / sigma at shift h = s % sigma, whose weight at tap m is
// w[m - h], over ell + sigma - 1 taps; lane l of chunk c of super-tile st
// then computes, in slot s, the output at position
//     st * sigma * d + 64 c + l + h * d,
// valid when 64 c + l < d (the chunks of a super-tile cover d positions per
// shift) and the position is below O.  A super-tile covers sigma * d
// consecutive outputs per kernel in ceil(d / 64) chunks; each chunk is one
// tile of 64 consecutive series reads per tap, as in an MFMA item.
constexpr int kToepVariant0 = 4 * kNumEll;

// Series of at most this length can run in the series-lane layout, which
// takes MFMA items only; VALU items are made for longer series.
constexpr int kSeriesMaxL = 128;
constexpr int kNumSplitLayouts = 6;  // 1, 2, 4, 8, 16, 32 splits
constexpr int kSplitCounts[kNumSplitLayouts] = {1, 2, 4, 8, 16, 32};

// MINIROCKET (Sec. 5 names it): 84 kernels of 9 taps.  Pair (dilation i,
// kernel k) is padded when i + k is even, so at one (dilation, padding) the
// kernels are those of one parity of k: an item holds those 42 kernels and
// kMrQTiny, kMrQSmall or kMrQLarge of each kernel's biases (dummy biases of
// +inf fill the last chunk; C > +inf never holds).  Variant = 3 * parity +
// bias class (0: kMrQSmall, 1: kMrQLarge, 2: kMrQTiny).
constexpr int kMrKernels = 84;
constexpr int kMrTaps = 9;
constexpr int kMrKappa = kMrKernels / 2;
constexpr int kMrQTiny = 3;
constexpr int kMrQSmall = 4;
constexpr int kMrQLarge = 8;
constexpr int kMrNumVariants = 6;  // parity x {kMrQSmall, kMrQLarge, kMrQTiny}
constexpr int mr_variant(int parity, int nq) {
    return 3 * parity + (nq == kMrQLarge ? 1 : (nq == kMrQTiny ? 2 : 0));
}

struct HostPlan {
    bool minirocket = false;
    int64_t n_features = 0;  // columns of F
    int32_t n_kernels = 0;
    int32_t L = 0;
    int32_t halo_lo = 0;     // padded layout: zeros staged before the series
    int32_t halo_hi = 0;     // padded layout: zeros staged after the series
    int32_t row_stride = 0;  // padded layout: floats per staged row (0: does not fit 32 bits)
    int32_t tail_pad = 0;    // zeros staged after the last row (reads of lanes past O)
    int32_t n_channels = 1;  // channels per series
    int64_t n_buckets = 0;
    int64_t mfma_per_row = 0;
    int64_t series_mfma_64 = 0;  // MFMAs for 64 series in the series-lane layout (O x taps x G)
    int64_t valu_fma_per_row = 0;  // VALU items: fp32 FMA instructions (64 lanes) per series
    std::vector<ItemDesc> items;
    std::vector<float> wpk;       // packed A-operand weights
    std::vector<float> bias;      // per slot
    std::vector<int32_t> kid;     // per slot, -1 = empty
    std::vector<int32_t> chan;    // per item, its channel list (ascending)
    std::vector<float> thr;       // MINIROCKET: per item [nq][4] thresholds
    std::vector<int32_t> order;   // kNumSplitLayouts concatenated item orders
    int32_t n_variants = kNumVariants;  // code variants of the plan's kernel (kMrNumVariants for MINIROCKET)
    std::vector<int32_t> split_begin;  // per layout: n_variants*nsplit + 1 offsets into order
    std::vector<int32_t> layout_off;   // per layout: offset into split_begin
};

// Validate a kernel set for series length L (host only, no device calls).
rocket_status validate_kernels(const rocket_kernels *k, int32_t L);

// Build the host-side tables of a plan.  Assumes validate_kernels passed.
rocket_status build_host_plan(const rocket_kernels *k, int32_t L, HostPlan *out);

// MINIROCKET parameters: validation and the plan's host tables.
rocket_status validate_minirocket(const rocket_minirocket_params *m);
rocket_status build_minirocket_plan(const rocket_minirocket_params *m, HostPlan *out);

// Item orders: per variant (0 .. n_variants - 1), longest-processing-time
// split of the items into every layout's split count (fills order,
// split_begin, layout_off).
void build_item_orders(HostPlan &P);

// Element `index` of the SplitMix64 sequence started at `seed`.
uint64_t splitmix64_at(uint64_t seed, uint64_t index);

}  // namespace rocket
