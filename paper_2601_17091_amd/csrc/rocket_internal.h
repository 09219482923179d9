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

// One work item: up to 4*G kernels that share (length, dilation, padding).
// The 64 lanes of a wavefront each own a chunk of consecutive outputs along
// one dilation residue class (positions q, q+d, q+2d, ...).  Each residue
// class is split into nc chunks of balanced length, S or S-1 outputs.  A
// "round" hands 64 chunks to the 64 lanes and runs a fixed number of steps
// for all of them: the chunks of S outputs come first, so the first
// rounds_long rounds run S steps and the rest S-1.  In a round of S steps a
// lane holding an (S-1)-output chunk computes one extra output past its
// chunk, and a lane without a chunk computes junk; both start those
// accumulations from -inf (lane-table flags), so they change neither the
// count nor the max.  Every real output is computed by exactly one lane.
struct alignas(16) ItemDesc {
    int32_t variant;      // ell_index * 2 + (G - 1)
    int32_t d;            // dilation
    int32_t p;            // padding
    int32_t O;            // number of dot products (outputs)
    int32_t S;            // steps of a long chunk (short chunks: S - 1)
    int32_t rounds;       // rounds per series
    int32_t lane_off;     // first lane-table entry (rounds * 64 entries)
    int32_t w_off;        // first packed weight: [n_ch][G][ell][4] floats
    int32_t k_off;        // first slot entry: kernel ids and biases, [4G]
    int32_t cost;         // MFMA instructions per series (scheduling weight)
    int32_t n_long;       // chunks of S outputs
    int32_t n_short;      // chunks of S - 1 outputs
    int32_t rounds_long;  // rounds that run S steps: ceil(n_long / 64)
    int32_t n_ch;         // channels the item's kernels read (their union; 1 if univariate)
    int32_t ch_off;       // first entry of the item's channel list
    int32_t reserved0;
    double inv_O;         // 1 / O rounded to double (exact PPV, see transform.hip)
    int32_t reserved1[2];
};
static_assert(sizeof(ItemDesc) == 80, "ItemDesc must stay 80 bytes");
constexpr int kItemWords = (int)(sizeof(ItemDesc) / sizeof(int32_t));

// Lane-table entry: the output position of the lane's first step (below
// 2^24) and two flags.
constexpr int64_t kMaxOutputs = (int64_t)1 << 24;  // O must stay below 2^24
constexpr uint32_t kLanePosMask = 0x00FFFFFFu;
constexpr uint32_t kLaneShort = 1u << 31;  // chunk is one output short: last step discarded
constexpr uint32_t kLaneIdle = 1u << 30;   // no chunk: every step discarded

// Item orders for a few split counts.  Within a layout with `nsplit` splits
// the items are grouped by variant, so that every workgroup runs one code
// variant: the items of variant v in split s are
// order[split_begin[v*nsplit + s] .. split_begin[v*nsplit + s + 1]).
constexpr int kNumVariants = 2 * kNumEll;
constexpr int kNumSplitLayouts = 6;  // 1, 2, 4, 8, 16, 32 splits
constexpr int kSplitCounts[kNumSplitLayouts] = {1, 2, 4, 8, 16, 32};

struct HostPlan {
    int32_t n_kernels = 0;
    int32_t L = 0;
    int32_t halo_lo = 0;   // zeros staged before the series in LDS
    int32_t halo_hi = 0;   // zeros staged after the series in LDS
    int32_t row_stride = 0;  // floats per staged row
    int32_t tail_pad = 0;    // zeros staged after the last row (reads of discarded steps)
    int32_t n_channels = 1;  // channels per series
    int64_t n_buckets = 0;
    int64_t mfma_per_row = 0;
    std::vector<ItemDesc> items;
    std::vector<uint32_t> lanes;
    std::vector<float> wpk;       // packed A-operand weights
    std::vector<float> bias;      // per slot
    std::vector<int32_t> kid;     // per slot, -1 = empty
    std::vector<int32_t> chan;    // per item, its channel list (ascending)
    std::vector<int32_t> order;   // kNumSplitLayouts concatenated item orders
    std::vector<int32_t> split_begin;  // per layout: kNumVariants*nsplit + 1 offsets into order
    std::vector<int32_t> layout_off;   // per layout: offset into split_begin
};

// Validate a kernel set for series length L (host only, no device calls).
rocket_status validate_kernels(const rocket_kernels *k, int32_t L);

// Build the host-side tables of a plan.  Assumes validate_kernels passed.
rocket_status build_host_plan(const rocket_kernels *k, int32_t L, HostPlan *out);

// Chunking of one bucket: nc chunks per residue class, chunk lengths S and
// S-1, with n_long / n_short chunks of each; rounds of 64 chunks, the first
// rounds_long of them running S steps.  Chosen to minimise an estimate of
// the cycles one series costs (MFMA steps, reductions, round set-up).
struct Chunking {
    int64_t nc = 1, S = 1, n_long = 0, n_short = 0, rounds = 0, rounds_long = 0;
    int64_t steps() const { return rounds_long * S + (rounds - rounds_long) * (S - 1); }
};
Chunking choose_chunking(int64_t O, int64_t d, int ell);

}  // namespace rocket
