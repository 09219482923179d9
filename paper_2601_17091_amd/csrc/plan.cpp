// Host-side planning: validation, bucketing of kernels by (length, dilation,
// padding), work items, packed weights and item orders for the fused MFMA
// kernel.  Pure host code; no HIP calls.
#include <algorithm>
#include <array>
#include <climits>
#include <cstring>
#include <map>
#include <new>
#include <tuple>
#include <utility>
#include <vector>

#include "rocket_internal.h"

namespace rocket {

static int64_t output_length(int64_t L, int64_t len, int64_t dil, int64_t pad) {
    return L + 2 * pad - (len - 1) * dil;
}

static int popcount64(uint64_t m) { return __builtin_popcountll(m); }

// Multivariate kernel lists: cut into groups of 4 kernels whose channel
// unions stay small.  Every channel in a group's union costs the group one
// MFMA chain pass (a kernel that does not read the channel has zero weights
// there), so the issued work is the sum over groups of |union| x taps x
// tiles.  Greedy: each group starts from the remaining kernel that reads the
// most channels and adds, one at a time, the kernel that adds the fewest new
// channels (ties: the one reading more channels, then list order); then
// pairwise swaps between groups are applied while they shrink the sum of the
// two unions, and finally 100 random swaps per kernel are tried, each kept
// when it does not grow the sum (moves across equal sums let the search
// leave the plateaus where no single swap shrinks it).  Deterministic (a
// fixed SplitMix64 sequence); the swap passes are skipped for lists above
// 1,024 kernels (the first one's cost is quadratic in the group count).
using KernelSlot = std::pair<int32_t, int32_t>;  // (kernel, first frame tap)
template <typename MaskOf>
static std::vector<std::vector<KernelSlot>> group_by_channels(std::vector<KernelSlot> ks,
                                                              const MaskOf &mask_of) {
    std::vector<std::vector<KernelSlot>> groups;
    std::vector<char> used(ks.size(), 0);
    size_t left = ks.size();
    while (left > 0) {
        size_t seed = ks.size();
        for (size_t i = 0; i < ks.size(); ++i)
            if (!used[i] && (seed == ks.size() ||
                             popcount64(mask_of(ks[i].first)) > popcount64(mask_of(ks[seed].first))))
                seed = i;
        std::vector<KernelSlot> g{ks[seed]};
        used[seed] = 1;
        --left;
        uint64_t u = mask_of(ks[seed].first);
        while (g.size() < (size_t)kSlotsPerGroup && left > 0) {
            size_t best = ks.size();
            int best_add = 0, best_cnt = 0;
            for (size_t i = 0; i < ks.size(); ++i) {
                if (used[i]) continue;
                const uint64_t m = mask_of(ks[i].first);
                const int add = popcount64(u | m) - popcount64(u), cnt = popcount64(m);
                if (best == ks.size() || add < best_add || (add == best_add && cnt > best_cnt)) {
                    best = i;
                    best_add = add;
                    best_cnt = cnt;
                }
            }
            g.push_back(ks[best]);
            used[best] = 1;
            --left;
            u |= mask_of(ks[best].first);
        }
        groups.push_back(std::move(g));
    }
    if (ks.size() > 1024) return groups;
    auto uni = [&](const std::vector<KernelSlot> &g) {
        uint64_t u = 0;
        for (const KernelSlot &e : g) u |= mask_of(e.first);
        return popcount64(u);
    };
    for (int pass = 0; pass < 4; ++pass) {
        bool improved = false;
        for (size_t a = 0; a < groups.size(); ++a)
            for (size_t b = a + 1; b < groups.size(); ++b) {
                int base = uni(groups[a]) + uni(groups[b]);
                for (size_t ia = 0; ia < groups[a].size(); ++ia)
                    for (size_t ib = 0; ib < groups[b].size(); ++ib) {
                        std::swap(groups[a][ia], groups[b][ib]);
                        const int c = uni(groups[a]) + uni(groups[b]);
                        if (c < base) {
                            base = c;
                            improved = true;
                        } else {
                            std::swap(groups[a][ia], groups[b][ib]);
                        }
                    }
            }
        if (!improved) break;
    }
    if (groups.size() < 2) return groups;
    uint64_t state = 0x243F6A8885A308D3ull ^ (uint64_t)ks.size();
    auto next = [&state]() {  // SplitMix64
        uint64_t z = (state += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    };
    std::vector<int> cost(groups.size());
    for (size_t g = 0; g < groups.size(); ++g) cost[g] = uni(groups[g]);
    const size_t tries = 100 * ks.size();
    for (size_t t = 0; t < tries; ++t) {
        const size_t a = next() % groups.size();
        size_t b = next() % (groups.size() - 1);
        if (b >= a) ++b;
        const size_t ia = next() % groups[a].size(), ib = next() % groups[b].size();
        std::swap(groups[a][ia], groups[b][ib]);
        const int ca = uni(groups[a]), cb = uni(groups[b]);
        if (ca + cb <= cost[a] + cost[b]) {
            cost[a] = ca;
            cost[b] = cb;
        } else {
            std::swap(groups[a][ia], groups[b][ib]);
        }
    }
    return groups;
}

rocket_status validate_kernels(const rocket_kernels *k, int32_t L) {
    if (!k || L < 1 || k->n_kernels < 1) return ROCKET_ERR_INVALID_ARG;
    if (!k->length || !k->dilation || !k->padding || !k->bias || !k->weights)
        return ROCKET_ERR_INVALID_ARG;
    if (k->max_len < 1 || k->max_len > ROCKET_MAX_KERNEL_LENGTH) return ROCKET_ERR_INVALID_ARG;
    for (int32_t i = 0; i < k->n_kernels; ++i) {
        const int32_t len = k->length[i], d = k->dilation[i], p = k->padding[i];
        if (len < 1 || len > k->max_len || d < 1 || p < 0) return ROCKET_ERR_INVALID_ARG;
    }
    const int32_t C = k->n_channels < 1 ? 1 : k->n_channels;
    if (C > ROCKET_MAX_CHANNELS) return ROCKET_ERR_INVALID_ARG;
    if (C > 1) {
        if (!k->channel_count || !k->channel_index) return ROCKET_ERR_INVALID_ARG;
        for (int32_t i = 0; i < k->n_kernels; ++i) {
            const int32_t cc = k->channel_count[i];
            if (cc < 1 || cc > C) return ROCKET_ERR_INVALID_ARG;
            uint64_t seen = 0;
            for (int32_t s = 0; s < cc; ++s) {
                const int32_t c = k->channel_index[(int64_t)i * C + s];
                if (c < 0 || c >= C || (seen >> c) & 1u) return ROCKET_ERR_INVALID_ARG;
                seen |= (uint64_t)1 << c;
            }
        }
    }
    for (int32_t i = 0; i < k->n_kernels; ++i) {
        const int64_t O = output_length(L, k->length[i], k->dilation[i], k->padding[i]);
        if (O < 1 || O >= kMaxOutputs) return ROCKET_ERR_LENGTH;
    }
    return ROCKET_OK;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

void build_item_orders(HostPlan &P) {
    // per variant, largest cost first (longest-processing-time first), dealt
    // to splits greedily by accumulated cost
    std::vector<int32_t> by_cost(P.items.size());
    for (size_t i = 0; i < by_cost.size(); ++i) by_cost[i] = (int32_t)i;
    std::stable_sort(by_cost.begin(), by_cost.end(),
                     [&](int32_t a, int32_t b) { return P.items[a].cost > P.items[b].cost; });
    for (int li = 0; li < kNumSplitLayouts; ++li) {
        const int ns = kSplitCounts[li];
        P.layout_off.push_back((int32_t)P.split_begin.size());
        for (int v = 0; v < P.n_variants; ++v) {
            std::vector<std::vector<int32_t>> lists(ns);
            std::vector<int64_t> load(ns, 0);
            for (int32_t it : by_cost) {
                if (P.items[it].variant != v) continue;
                int best = 0;
                for (int sp = 1; sp < ns; ++sp)
                    if (load[sp] < load[best]) best = sp;
                lists[best].push_back(it);
                load[best] += P.items[it].cost;
            }
            for (int sp = 0; sp < ns; ++sp) {
                P.split_begin.push_back((int32_t)P.order.size());
                P.order.insert(P.order.end(), lists[sp].begin(), lists[sp].end());
            }
        }
        P.split_begin.push_back((int32_t)P.order.size());
    }
}

// Toeplitz items (variants kToepVariant0..): the one (sigma = 4) or two
// (sigma = 2) leftover kernels of a bucket at dilation d.  Per super-tile of
// sigma * d outputs per kernel: ceil(d / 64) chunks of ell + sigma - 1 MFMAs,
// each computing 4 x 64 outputs; the last super-tile covers what is left of
// O.  A VALU item costs ell fp32 FMAs per kernel per 64 outputs.
struct ToepShape {
    int sigma;
    int64_t nc;       // chunks per super-tile
    int64_t s_full;   // whole super-tiles
    int64_t n_last;   // chunks of the last, partial super-tile
    int64_t chunks;   // chunks per series
};
static ToepShape toeplitz_shape(int nk, int32_t d, int64_t O) {
    ToepShape t;
    t.sigma = 4 / nk;
    t.nc = ceil_div(d, kTile);
    const int64_t span = (int64_t)t.sigma * d;
    t.s_full = O / span;
    const int64_t rest = O - t.s_full * span;
    t.n_last = rest > 0 ? ceil_div(std::min<int64_t>(rest, d), kTile) : 0;
    t.chunks = t.s_full * t.nc + t.n_last;
    return t;
}

template <typename KS>
static bool toeplitz_pays(const KS &ks, size_t pos, size_t nk, int ell, int32_t d, int64_t O,
                          const rocket_kernels *k) {
    // the kernels must fill their frame (first frame tap 0, full length)
    for (size_t s = 0; s < nk; ++s)
        if (ks[pos + s].second != 0 || k->length[ks[pos + s].first] != ell) return false;
    const ToepShape t = toeplitz_shape((int)nk, d, O);
    // issue cycles per series: fp32 FMA 4.5, 4x4x1 fp32 MFMA 8.7, 1.5 vector
    // instructions to reduce a result register; the chunks of the last
    // super-tile also build their per-slot start values (about 10 more)
    const double valu = (double)ceil_div(O, kTile) * nk * (ell * 4.5 + 1.5 * 4.5);
    const double toep = (double)t.chunks * ((ell + t.sigma - 1) * 8.7 + 4 * 1.5 * 4.5) + (double)t.n_last * 45.0;
    return toep < 0.9 * valu;
}

template <typename KS>
static void add_toeplitz_item(HostPlan &P, const KS &ks, size_t pos, int nk, int eidx, int32_t d, int32_t p,
                              int64_t O, int32_t L, const rocket_kernels *k) {
    const int ell = kEllValues[eidx];
    const ToepShape t = toeplitz_shape(nk, d, O);
    const int taps = ell + t.sigma - 1;
    ItemDesc it;
    std::memset(&it, 0, sizeof(it));
    it.variant = kToepVariant0 + eidx * 2 + (nk - 1);
    it.d = d;
    it.p = p;
    it.O = (int32_t)O;
    it.n_tiles = (int32_t)t.nc;
    it.w_off = (int32_t)P.wpk.size();
    it.k_off = (int32_t)P.kid.size();
    it.cost = (int32_t)std::min<int64_t>(t.chunks * taps, INT32_MAX);
    it.n_ch = 1;
    it.ch_off = (int32_t)P.chan.size();
    P.chan.push_back(0);
    it.ch_mask[0] = 1u;
    it.inv_O = 1.0 / (double)O;
    // weights [tap m][slot s]: kernel s / sigma at shift s % sigma
    for (int m = 0; m < taps; ++m)
        for (int s = 0; s < 4; ++s) {
            const int32_t kk = ks[pos + (size_t)(s / t.sigma)].first;
            const int j = m - s % t.sigma;
            P.wpk.push_back(j >= 0 && j < ell ? k->weights[(int64_t)kk * k->max_len + j] : 0.0f);
        }
    // slots: the kernel id on the first slot of each kernel (its writer),
    // every slot carries its kernel's bias
    for (int s = 0; s < 4; ++s) {
        const int32_t kk = ks[pos + (size_t)(s / t.sigma)].first;
        P.kid.push_back(s % t.sigma == 0 ? kk : -1);
        P.bias.push_back(k->bias[kk]);
    }
    P.items.push_back(it);
    P.mfma_per_row += t.chunks * taps;
    (void)L;
}

static rocket_status build_plan(const rocket_kernels *k, int32_t L, bool allow_toeplitz, HostPlan *out);

// Toeplitz items run in a launch of their own, which stages every row group
// again: they are kept only where they carry a real share of the work (at
// least kToepMinShare of the items' cost), else their kernels stay in VALU
// items.
constexpr double kToepMinShare = 0.03;

rocket_status build_host_plan(const rocket_kernels *k, int32_t L, HostPlan *out) {
    rocket_status st = build_plan(k, L, true, out);
    if (st != ROCKET_OK) return st;
    double toep = 0.0, total = 0.0;
    for (const ItemDesc &it : out->items) {
        total += it.cost;
        if (it.variant >= kToepVariant0) toep += it.cost;
    }
    if (toep > 0.0 && toep < kToepMinShare * total) st = build_plan(k, L, false, out);
    return st;
}

static rocket_status build_plan(const rocket_kernels *k, int32_t L, bool allow_toeplitz, HostPlan *out) {
    try {
        HostPlan P;
        P.n_kernels = k->n_kernels;
        P.L = L;
        const int32_t C = k->n_channels < 1 ? 1 : k->n_channels;
        P.n_channels = C;
        // channels kernel i reads, as a bit mask (bit 0 for univariate sets)
        auto mask_of = [&](int32_t i) -> uint64_t {
            if (C == 1) return 1u;
            uint64_t m = 0;
            for (int32_t s = 0; s < k->channel_count[i]; ++s)
                m |= (uint64_t)1 << k->channel_index[(int64_t)i * C + s];
            return m;
        };
        // weight row of kernel i for channel c (nullptr if it does not read c)
        auto row_of = [&](int32_t i, int32_t c) -> const float * {
            if (C == 1) return k->weights + (int64_t)i * k->max_len;
            for (int32_t s = 0; s < k->channel_count[i]; ++s)
                if (k->channel_index[(int64_t)i * C + s] == c)
                    return k->weights + ((int64_t)i * C + s) * k->max_len;
            return nullptr;
        };
        // bucket kernels by (length, dilation, padding); kernels keep their
        // original order inside a bucket
        std::map<std::tuple<int32_t, int32_t, int32_t>, std::vector<int32_t>> buckets;
        // the taps of real outputs reach from position -p to L-1+p, plus
        // (ell - length) taps of zero weight for kernels run at a longer
        // code length; lanes past O in an item's last tile read up to 63
        // positions further (the next row's data, or after the last row the
        // tail, tail_pad below: those lanes start from -inf, so what they
        // read changes no feature)
        int64_t halo_lo = 0, halo_hi = 0;
        for (int32_t i = 0; i < k->n_kernels; ++i) {
            const int32_t len = k->length[i], d = k->dilation[i], p = k->padding[i];
            buckets[std::make_tuple(len, d, p)].push_back(i);
            const int64_t ell_eff = kEllValues[ell_index_for(len)];
            halo_lo = std::max<int64_t>(halo_lo, p);
            halo_hi = std::max<int64_t>(halo_hi, (int64_t)p + (ell_eff - len) * (int64_t)d);
        }
        P.n_buckets = (int64_t)buckets.size();
        // Consecutive staged rows share their zero margins: each row is a
        // left margin of h zeros and the series, and its right margin is the
        // next row's left margin (after the last row, the tail), so
        // h = max(halo_lo, halo_hi).  The margin is rounded so that the
        // series starts, and every staged row spans, a whole number of
        // 16-byte words: rows are then staged with 16-byte loads and LDS
        // writes (for series lengths divisible by 4).
        const int64_t h = (std::max(halo_lo, halo_hi) + 3) / 4 * 4;
        const int64_t stride = (h + L + 3) / 4 * 4;
        if (stride + h > (int64_t)1 << 30) {
            // cannot be staged; the plan will use the direct kernel
            P.halo_lo = P.halo_hi = P.row_stride = 0;
        } else {
            P.halo_lo = (int32_t)h;
            P.halo_hi = (int32_t)h;
            P.row_stride = (int32_t)stride;
        }

        // Frame lists: the kernels one run of items covers, each with the
        // frame tap its first weight sits on.  A bucket is one list; but
        // centred kernels (padding (len-1)*d/2) of every length at one
        // dilation compute the same O = L outputs around the same centre, so
        // a shorter one also runs in a longer frame with zero weights on the
        // outer taps.  The empty slots of a bucket's last 4-slot group are
        // filled that way when it saves a group of a shorter frame
        // (univariate sets; every group costs frame taps x tiles).
        struct Frame {
            int eidx;   // frame length class
            int32_t d, p;
            std::vector<std::pair<int32_t, int32_t>> ks;  // (kernel, first frame tap)
        };
        std::vector<Frame> frames;
        std::map<int32_t, std::array<std::vector<int32_t>, kNumEll>> centred;  // by dilation
        for (auto &kv : buckets) {
            const int32_t len = std::get<0>(kv.first), d = std::get<1>(kv.first),
                          p = std::get<2>(kv.first);
            const int e = ell_index_for(len);
            if (C == 1 && len == kEllValues[e] && (int64_t)p * 2 == (int64_t)(len - 1) * d) {
                centred[d][e] = kv.second;
                continue;
            }
            Frame f{e, d, p, {}};
            for (int32_t i : kv.second) f.ks.emplace_back(i, 0);
            frames.push_back(std::move(f));
        }
        for (auto &kv : centred) {
            const int32_t d = kv.first;
            auto &ids = kv.second;
            const int64_t n7 = (int64_t)ids[0].size(), n9 = (int64_t)ids[1].size(),
                          n11 = (int64_t)ids[2].size();
            auto groups = [](int64_t n) { return ceil_div(n, kSlotsPerGroup); };
            auto freeslots = [](int64_t n) { return (kSlotsPerGroup - n % kSlotsPerGroup) % kSlotsPerGroup; };
            // a9 9s and a7 7s ride in the last 11-group, b7 7s in the last 9-group
            int64_t best = -1, ba9 = 0, ba7 = 0, bb7 = 0;
            const int64_t f11 = n11 > 0 ? freeslots(n11) : 0;
            for (int64_t a9 = 0; a9 <= std::min(n9, f11); ++a9)
                for (int64_t a7 = 0; a7 <= std::min(n7, f11 - a9); ++a7) {
                    const int64_t m9 = n9 - a9;
                    const int64_t f9 = m9 > 0 ? freeslots(m9) : 0;
                    for (int64_t b7 = 0; b7 <= std::min(n7 - a7, f9); ++b7) {
                        const int64_t cost = 11 * groups(n11 + a9 + a7) + 9 * groups(m9 + b7) +
                                             7 * groups(n7 - a7 - b7);
                        if (best < 0 || cost < best) {
                            best = cost;
                            ba9 = a9;
                            ba7 = a7;
                            bb7 = b7;
                        }
                    }
                }
            // the fillers are the last kernels of their own lists
            Frame f11l{2, d, 5 * d, {}}, f9l{1, d, 4 * d, {}}, f7l{0, d, 3 * d, {}};
            for (int32_t i : ids[2]) f11l.ks.emplace_back(i, 0);
            for (int64_t q = n9 - ba9; q < n9; ++q) f11l.ks.emplace_back(ids[1][q], 1);
            for (int64_t q = n7 - ba7; q < n7; ++q) f11l.ks.emplace_back(ids[0][q], 2);
            for (int64_t q = 0; q < n9 - ba9; ++q) f9l.ks.emplace_back(ids[1][q], 0);
            for (int64_t q = n7 - ba7 - bb7; q < n7 - ba7; ++q) f9l.ks.emplace_back(ids[0][q], 1);
            for (int64_t q = 0; q < n7 - ba7 - bb7; ++q) f7l.ks.emplace_back(ids[0][q], 0);
            for (Frame *f : {&f11l, &f9l, &f7l})
                if (!f->ks.empty()) frames.push_back(std::move(*f));
        }

        for (Frame &fr : frames) {
            const int32_t d = fr.d, p = fr.p;
            auto &ks = fr.ks;
            // multivariate: items of one 4-kernel group each, grouped so that
            // the channel unions stay small (an 8-kernel item would run both
            // of its groups over the union of all 8 channel sets)
            std::vector<int32_t> item_sizes;
            if (C > 1) {
                std::vector<KernelSlot> flat;
                for (auto &g : group_by_channels(ks, mask_of)) {
                    item_sizes.push_back((int32_t)g.size());
                    flat.insert(flat.end(), g.begin(), g.end());
                }
                ks = std::move(flat);
            }
            size_t next_item = 0;
            const int eidx = fr.eidx;
            const int ell = kEllValues[eidx];
            // every kernel of a frame list has these outputs
            const int64_t O = output_length(L, k->length[ks[0].first], d, k->padding[ks[0].first]);
            const int64_t n_tiles = ceil_div(O, kTile);
            // univariate sets of long series: the one or two kernels left
            // after the 4- and 8-kernel items run as a VALU item (a 5-kernel
            // rest as 4 + 1): one kernel costs a quarter of a 4-slot MFMA
            // group's FMA work, two about half
            const bool valu_ok = C == 1 && L > kSeriesMaxL;
            size_t pos = 0;
            while (pos < ks.size()) {
                const size_t rem = ks.size() - pos;
                const int nk_valu = (valu_ok && rem <= 2) ? (int)rem : 0;
                if (nk_valu && allow_toeplitz && toeplitz_pays(ks, pos, (size_t)nk_valu, ell, d, O, k)) {
                    add_toeplitz_item(P, ks, pos, nk_valu, eidx, d, p, O, L, k);
                    pos += (size_t)nk_valu;
                    continue;
                }
                const int G = (C > 1 || rem <= 4 || (valu_ok && rem == 5)) ? 1 : 2;
                const size_t take = C > 1 ? (size_t)item_sizes[next_item++]
                                          : std::min<size_t>(rem, (size_t)(4 * G));
                ItemDesc it;
                std::memset(&it, 0, sizeof(it));
                it.variant = nk_valu ? kValuVariant0 + eidx * 2 + (nk_valu - 1) : eidx * 2 + (G - 1);
                it.d = d;
                it.p = p;
                it.O = (int32_t)O;
                it.n_tiles = (int32_t)n_tiles;
                it.w_off = (int32_t)P.wpk.size();
                it.k_off = (int32_t)P.kid.size();
                uint64_t umask = 0;
                for (size_t s = 0; s < take; ++s) umask |= mask_of(ks[pos + s].first);
                it.n_ch = 0;
                it.ch_off = (int32_t)P.chan.size();
                it.ch_mask[0] = (uint32_t)umask;
                it.ch_mask[1] = (uint32_t)(umask >> 32);
                for (int32_t c = 0; c < C; ++c)
                    if ((umask >> c) & 1u) {
                        P.chan.push_back(c);
                        ++it.n_ch;
                    }
                // MFMA instructions per series: ell taps per tile and group,
                // for every channel of the item (capped: it only orders work);
                // a VALU item's nk FMAs per tap and tile count as half an
                // MFMA each (4.5 against 8.7 cycles)
                it.cost = nk_valu ? (int32_t)std::min<int64_t>((n_tiles * ell * nk_valu + 1) / 2, INT32_MAX)
                                  : (int32_t)std::min<int64_t>(n_tiles * ell * G * it.n_ch, INT32_MAX);
                it.inv_O = 1.0 / (double)O;
                // A-operand weights: [channel][g][j][slot i]; zeros for empty
                // slots, for channels a slot's kernel does not read and for
                // frame taps outside the kernel's own taps
                for (int32_t ci = 0; ci < it.n_ch; ++ci) {
                    const int32_t c = P.chan[it.ch_off + ci];
                    for (int g = 0; g < G; ++g)
                        for (int j = 0; j < ell; ++j)
                            for (int i = 0; i < 4; ++i) {
                                const size_t s = (size_t)(4 * g + i);
                                float w = 0.0f;
                                if (s < take) {
                                    const int32_t kk = ks[pos + s].first, off = ks[pos + s].second;
                                    const float *row = row_of(kk, c);
                                    if (row && j >= off && j < off + k->length[kk]) w = row[j - off];
                                }
                                P.wpk.push_back(w);
                            }
                }
                for (int s = 0; s < 4 * G; ++s) {
                    if ((size_t)s < take) {
                        P.kid.push_back(ks[pos + s].first);
                        P.bias.push_back(k->bias[ks[pos + s].first]);
                    } else {
                        P.kid.push_back(-1);
                        P.bias.push_back(0.0f);
                    }
                }
                P.items.push_back(it);
                if (!nk_valu) {
                    P.mfma_per_row += n_tiles * ell * G * it.n_ch;
                    P.series_mfma_64 += O * ell * G;
                } else {
                    P.valu_fma_per_row += n_tiles * ell * nk_valu;
                }
                pos += take;
            }
        }

        // after the last row: its right margin, then the reads of lanes past
        // O in an item's last tile (up to 63 positions further)
        P.tail_pad = P.halo_hi + kTile;

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

extern "C" rocket_status rocket_plan_tables_build(const rocket_kernels *k, int32_t L,
                                                  rocket_plan_tables *out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    std::memset(out, 0, sizeof(*out));
    rocket_status st = rocket::validate_kernels(k, L);
    if (st != ROCKET_OK) return st;
    rocket::HostPlan *P = new (std::nothrow) rocket::HostPlan();
    if (!P) return ROCKET_ERR_OOM;
    st = rocket::build_host_plan(k, L, P);
    if (st != ROCKET_OK) {
        delete P;
        return st;
    }
    out->n_items = (int64_t)P->items.size();
    out->item_words = rocket::kItemWords;
    out->n_chan = (int64_t)P->chan.size();
    out->chan = P->chan.data();
    out->n_channels = P->n_channels;
    out->items = reinterpret_cast<const int32_t *>(P->items.data());
    out->n_wpk = (int64_t)P->wpk.size();
    out->wpk = P->wpk.data();
    out->n_slots = (int64_t)P->kid.size();
    out->slot_bias = P->bias.data();
    out->slot_kernel = P->kid.data();
    out->n_order = (int64_t)P->order.size();
    out->order = P->order.data();
    out->n_split_begin = (int64_t)P->split_begin.size();
    out->split_begin = P->split_begin.data();
    out->n_layouts = rocket::kNumSplitLayouts;
    out->layout_off = P->layout_off.data();
    out->split_counts = rocket::kSplitCounts;
    out->halo_lo = P->halo_lo;
    out->halo_hi = P->halo_hi;
    out->row_stride = P->row_stride;
    out->tail_pad = P->tail_pad;
    out->internal = P;
    return ROCKET_OK;
}

extern "C" void rocket_plan_tables_free(rocket_plan_tables *t) {
    if (!t) return;
    delete static_cast<rocket::HostPlan *>(t->internal);
    std::memset(t, 0, sizeof(*t));
}
