"""Host logic of the fused kernel, checked on the CPU.

The planner's tables (work items, packed weights, item orders) are read back
through rocket_plan_tables_build and walked here the way the GPU kernel walks
them: an item's O outputs are computed in ceil(O/64) tiles of 64 consecutive
positions, lane l of tile k computing output 64k + l; tiles run in blocks of
NT (8 for 4-kernel items, 4 for 8-kernel items); for tap j, lane l of tile u
of the block that starts at output t0 reads series index t0 - p + j*d +
64u + l.  In the padded layout that index is used as is (staged rows of
halo_lo zeros and the series, consecutive rows sharing their margins, so a
row's right margin of halo_hi zeros is the next row's left margin, and
tail_pad zeros after the last row); in the clamped layout the block's
offset t0 - p + j*d is clamped into [-512, L] first (512 zeros on each side
of the series).  Lanes past O start
from -inf on the GPU and change no feature.  The checks: every output of
every kernel is computed by exactly one lane, every load stays inside the
staged memory, every load of a real output reads the zero-padded series
value, the packed weights are the kernels' own, and an fp32 replay of the
walk lands inside the oracle's certified bounds.
"""
import numpy as np
import pytest

import paper_2601_17091_amd as rk
from _util import kernel_set

ELLS = (7, 9, 11)
TILE = 64
TILES_PER_BLOCK = {1: 8, 2: 4}
CLAMP_MARGIN = 512
N_VARIANTS = 18      # 0..5 MFMA items, 6..11 VALU items, 12..17 Toeplitz items
TOEP0 = 12
SERIES_MAX_L = 128   # VALU items only for longer series
SERIES_MARGIN = 8    # series-lane layout: zero positions staged on each side of a series


def variant_info(v):
    """(taps, MFMA groups G, VALU kernels nk) of an item variant: MFMA items
    2*ell_index + (G-1); VALU items 6 + 2*ell_index + (nk-1), packed as G = 1."""
    if v < 6:
        return ELLS[v // 2], v % 2 + 1, 0
    return ELLS[(v - 6) // 2], 1, (v - 6) % 2 + 1


def item_fields(row):
    (variant, d, p, O, n_tiles, w_off, k_off, cost, n_ch, ch_off) = (int(v) for v in row[:10])
    inv_O = row[14:16].astype(np.int32).view(np.float64)[0]
    return dict(variant=variant, d=d, p=p, O=O, n_tiles=n_tiles, w_off=w_off, k_off=k_off,
                cost=cost, n_ch=n_ch, ch_off=ch_off, inv_O=inv_O)


def kernel_row(kernels, k, c):
    """Weights of kernel k for channel c (None if it does not read c)."""
    C = int(kernels.get("n_channels", 1))
    if C == 1:
        return kernels["weights"][k] if c == 0 else None
    for s_ in range(int(kernels["channel_count"][k])):
        if int(kernels["channel_index"][k][s_]) == c:
            return kernels["weights"][k][s_]
    return None


def tile_reads(f, ell, L, clamped):
    """Series index every lane reads, [tile, lane, tap], in the given layout."""
    G = variant_info(f["variant"])[1]
    NT = TILES_PER_BLOCK[G]
    nt, d, p = f["n_tiles"], f["d"], f["p"]
    k = np.arange(nt)
    t0 = (k // NT) * NT * TILE                      # first output of the tile's block
    u = k % NT                                      # tile within its block
    off = t0[:, None] - p + np.arange(ell)[None, :] * d   # [tile, tap] block offset of the tap
    if clamped:
        off = np.clip(off, -CLAMP_MARGIN, L)
    return off[:, None, :] + (u * TILE)[:, None, None] + np.arange(TILE)[None, :, None]


def walk_toeplitz(f, tables, kernels, L, halo_lo, stride, pad, rows, clamped, cover, F, right_end):
    """A Toeplitz item (one or two leftover kernels at dilation d): slot s is
    kernel s // sigma shifted by h = s % sigma taps over ell + sigma - 1 taps;
    super-tiles of sigma*d outputs per kernel in ceil(d/64) chunks, run in
    blocks of 8 chunks (the last super-tile, if partial, one chunk at a
    time); lane l of the chunk at t0 reads t0 - p + m*d + l at tap m and, in
    slot s, computes the output at t0 + l + h*d, valid when it lies in the
    chunk's first d positions per shift and below O."""
    v = f["variant"] - TOEP0
    ell, nk = ELLS[v // 2], v % 2 + 1
    sigma = 4 // nk
    taps = ell + sigma - 1
    d, p, O = f["d"], f["p"], f["O"]
    nc = -(-d // TILE)
    assert f["n_tiles"] == nc and L > SERIES_MAX_L and f["n_ch"] == 1
    kid = tables["slot_kernel"][f["k_off"]:f["k_off"] + 4]
    bias = tables["slot_bias"][f["k_off"]:f["k_off"] + 4]
    W = tables["wpk"][f["w_off"]:f["w_off"] + taps * 4].reshape(taps, 4)
    kern = []
    for q in range(nk):
        k = int(kid[q * sigma])
        assert k >= 0 and np.all(kid[q * sigma + 1:(q + 1) * sigma] < 0)
        assert int(kernels["length"][k]) == ell and int(kernels["dilation"][k]) == d
        assert int(kernels["padding"][k]) == p
        assert L + 2 * p - (ell - 1) * d == O
        for h in range(sigma):
            s_ = q * sigma + h
            col = np.zeros(taps, np.float32)
            col[h:h + ell] = kernels["weights"][k][:ell]
            assert np.array_equal(W[:, s_], col) and bias[s_] == np.float32(kernels["bias"][k])
        kern.append(k)
    span = sigma * d
    s_full = O // span
    rest = O - s_full * span
    nlast = -(-min(rest, d) // TILE) if rest > 0 else 0
    assert f["cost"] == (s_full * nc + nlast) * taps
    # chunks as (t0, block offset of tap 0, tile within block, last super-tile)
    chunks = []
    for st in range(s_full):
        for c in range(nc):
            chunks.append((st * span + c * TILE, st * span + (c // 8) * 8 * TILE, c % 8, False))
    for c in range(nlast):
        t0 = s_full * span + c * TILE
        chunks.append((t0, t0, 0, True))
    t0 = np.array([c_[0] for c_ in chunks])
    boff = np.array([c_[1] for c_ in chunks])
    u = np.array([c_[2] for c_ in chunks])
    last = np.array([c_[3] for c_ in chunks])
    lane = np.arange(TILE)
    off = boff[:, None] - p + np.arange(taps)[None, :] * d          # [chunk, tap]
    if clamped:
        off = np.clip(off, -CLAMP_MARGIN, L)
    else:
        # the last super-tile's block offsets are clamped to at most L
        off = np.where(last[:, None], np.minimum(off, L), off)
    idx = off[:, None, :] + (u * TILE)[:, None, None] + lane[None, :, None]   # [chunk, lane, tap]
    assert (halo_lo + idx).min() >= 0 and (halo_lo + idx).max() < stride + pad, (d, p, O)
    for q, k in enumerate(kern):
        cov = np.zeros(O, np.int64)
        vals = []
        for h in range(sigma):
            s_ = q * sigma + h
            pos = t0[:, None] + lane[None, :] + h * d                 # [chunk, lane]
            within = ((t0 - (t0 // span) * span)[:, None] + lane[None, :]) < d
            real = within & (pos < O)
            np.add.at(cov, pos[real], 1)
            # taps with a weight for this slot read the zero-padded series at the true index
            ri = idx[real][:, h:h + ell]
            ti = pos[real][:, None] - p + np.arange(ell)[None, :] * d
            inside = (ti >= 0) & (ti < L)
            assert np.array_equal(ri[inside], ti[inside])
            assert np.all((ri[~inside] < 0) | (ri[~inside] >= L))
            assert (halo_lo + ri).max() < right_end
            vals.append((s_, real, pos))
        cover[k] = cov
        if rows is not None:
            n = rows.shape[0]
            ys, ms = [], []
            for s_, real, pos in vals:
                acc = np.full((n, int(real.sum())), bias[s_], np.float32)
                xr = rows[:, 0][:, halo_lo + idx[real]]                  # [n, output, tap]
                for m in range(taps):
                    acc = (acc + xr[..., m] * W[m, s_]).astype(np.float32)
                ys.append(acc)
            y = np.concatenate(ys, axis=1)
            F[:, 2 * k] = (y > 0).sum(axis=1) / O
            F[:, 2 * k + 1] = y.max(axis=1)


def walk(tables, kernels, L, X=None, clamped=False):
    """Replay the fused kernel's schedule; returns per-kernel coverage and,
    if X is given, fp32 features [n, 2K]."""
    K = len(kernels["length"])
    C = int(kernels.get("n_channels", 1))
    halo_lo, halo_hi, stride, pad = (tables["halo_lo"], tables["halo_hi"], tables["row_stride"],
                                     tables["tail_pad"])
    if clamped:
        # each row keeps both margins; TILE zeros after the last row
        halo_lo, halo_hi, stride, pad = CLAMP_MARGIN, CLAMP_MARGIN, L + 2 * CLAMP_MARGIN, TILE
        assert stride == halo_lo + L + halo_hi
    else:
        # consecutive rows share their margins: a row is halo_lo zeros and the
        # series; its right margin is the next row's left margin or, after the
        # last row, the first halo_hi zeros of the tail
        assert stride >= halo_lo + L and halo_hi <= halo_lo and stride % 4 == 0 and halo_lo % 4 == 0
        assert pad >= halo_hi + TILE - 1
    right_end = halo_lo + L + halo_hi   # end of the zeros right of a row's series
    cover = [np.zeros(0, np.int64)] * K
    F = None
    if X is not None:
        n = X.shape[0]
        F = np.full((n, 2 * K), np.nan, dtype=np.float64)
        Xc = X.reshape(n, C, L)
        rows = np.zeros((n, C, stride + pad), dtype=np.float32)
        rows[:, :, halo_lo:halo_lo + L] = Xc
    for row in tables["items"]:
        f = item_fields(row)
        if f["variant"] >= TOEP0:
            walk_toeplitz(f, tables, kernels, L, halo_lo, stride, pad, rows if X is not None else None, clamped,
                          cover, F, right_end)
            continue
        d, p, O = f["d"], f["p"], f["O"]
        ell, G, nk = variant_info(f["variant"])
        nslot = 4 * G
        kid = tables["slot_kernel"][f["k_off"]:f["k_off"] + nslot]
        bias = tables["slot_bias"][f["k_off"]:f["k_off"] + nslot]
        nch = f["n_ch"]
        chans = tables["chan"][f["ch_off"]:f["ch_off"] + nch].astype(np.int64)
        assert nch >= 1 and np.all(np.diff(chans) > 0) and chans.min() >= 0 and chans.max() < C
        W = tables["wpk"][f["w_off"]:f["w_off"] + nch * G * ell * 4].reshape(nch, G, ell, 4)
        # [channel, slot, tap]
        Wslot = np.stack([np.concatenate([W[ci, g].T for g in range(G)], axis=0) for ci in range(nch)])
        used = np.zeros(nch, bool)
        for s_, k in enumerate(kid):
            if k >= 0:
                ln = int(kernels["length"][k])
                # a kernel runs in the item's frame of ell taps from frame tap
                # off on: its padding is p - off*d and its outputs the item's
                assert int(kernels["dilation"][k]) == d
                off, r_ = divmod(p - int(kernels["padding"][k]), d)
                assert r_ == 0 and 0 <= off and off + ln <= ell
                assert L + 2 * int(kernels["padding"][k]) - (ln - 1) * d == O
                for ci, c in enumerate(chans):
                    wrow = kernel_row(kernels, k, c)
                    if wrow is None:
                        assert np.all(Wslot[ci, s_] == 0)
                    else:
                        used[ci] = True
                        assert np.array_equal(Wslot[ci, s_, off:off + ln], wrow[:ln])
                        assert np.all(Wslot[ci, s_, :off] == 0) and np.all(Wslot[ci, s_, off + ln:] == 0)
                assert bias[s_] == np.float32(kernels["bias"][k])
            else:
                assert np.all(Wslot[:, s_] == 0)
        assert used.all()     # the channel list is exactly the union
        assert f["n_tiles"] == -(-O // TILE)
        if nk:
            # VALU items: the first nk slots, univariate long series
            assert nch == 1 and L > SERIES_MAX_L and np.all(kid[:nk] >= 0) and np.all(kid[nk:] < 0)
            assert f["cost"] == (f["n_tiles"] * ell * nk + 1) // 2
        else:
            assert f["cost"] == f["n_tiles"] * ell * G * nch
        assert f["inv_O"] == 1.0 / O
        # outputs: lane l of tile k computes 64k + l; the real ones are < O
        t = (np.arange(f["n_tiles"])[:, None] * TILE + np.arange(TILE)[None, :])   # [tile, lane]
        real = t < O
        for k in kid[kid >= 0]:
            cover[k] = np.bincount(t[real], minlength=O)
        idx = tile_reads(f, ell, L, clamped)                                          # [tile, lane, tap]
        # every load inside the staged memory (lanes past O of the last row:
        # inside the tail pad)
        assert (halo_lo + idx).min() >= 0 and (halo_lo + idx).max() < stride + pad, (d, p, O)
        # loads of real outputs inside the row, at the zero-padded series value
        true_idx = t[:, :, None] - p + np.arange(ell)[None, None, :] * d
        ri, ti = idx[real], true_idx[real]
        assert (halo_lo + ri).max() < right_end
        inside = (ti >= 0) & (ti < L)
        assert np.array_equal(ri[inside], ti[inside])
        assert np.all((ri[~inside] < 0) | (ri[~inside] >= L))
        if X is not None:
            acc = np.broadcast_to(bias.astype(np.float32), (n, O, nslot)).copy()
            # channel by channel, tap by tap, in the kernel's order
            for ci, c in enumerate(chans):
                xv = rows[:, c][:, halo_lo + ri.reshape(O, ell)]                  # [n, output, tap]
                for j in range(ell):
                    acc = (acc + xv[..., j, None] * Wslot[ci][None, None, :, j]).astype(np.float32)
            cnt = (acc > 0).sum(axis=1)
            mxv = acc.max(axis=1)
            for s_, k in enumerate(kid):
                if k >= 0:
                    F[:, 2 * k] = cnt[:, s_] / O
                    F[:, 2 * k + 1] = mxv[:, s_]
    return cover, F


def check_tables(kernels, L, X=None, oracle=None):
    t = rk.plan_tables(kernels, L)
    K = len(kernels["length"])
    # every item appears exactly once in every split layout, in the list of
    # its own variant
    n_items = t["items"].shape[0]
    for li in range(len(t["layout_off"])):
        ns = t["split_counts"][li]
        beg = t["split_begin"][t["layout_off"][li]:t["layout_off"][li] + N_VARIANTS * ns + 1]
        ids = []
        for v in range(N_VARIANTS):
            for s_ in range(ns):
                part = t["order"][beg[v * ns + s_]:beg[v * ns + s_ + 1]]
                assert np.all(t["items"][part, 0] == v)
                ids.append(part)
        assert np.array_equal(np.sort(np.concatenate(ids)), np.arange(n_items))
    # every kernel sits in exactly one slot
    kid = t["slot_kernel"]
    assert np.array_equal(np.sort(kid[kid >= 0]), np.arange(K))
    r = oracle.transform(X, kernels) if X is not None else None
    for clamped in (False, True):
        cover, F = walk(t, kernels, L, X, clamped)
        for k in range(K):
            O = L + 2 * int(kernels["padding"][k]) - (int(kernels["length"][k]) - 1) * int(kernels["dilation"][k])
            assert cover[k].shape[0] == O and np.all(cover[k] == 1), k
        if X is not None:
            cnt = np.rint(F[:, 0::2] * r["O"][None, :]).astype(np.int64)
            assert np.all(r["cnt_lo"] <= cnt) and np.all(cnt <= r["cnt_hi"])
            assert np.all(np.abs(F[:, 1::2] - r["F"][:, 1::2]) <= r["beta"])
    return t


@pytest.mark.parametrize("seed,K,L", [(1, 300, 11), (2, 300, 30), (3, 400, 64), (4, 500, 128),
                                      (5, 400, 500), (6, 300, 1000), (7, 200, 3000)])
def test_generated_sets_cover_every_output(seed, K, L):
    check_tables(rk.generate_kernels(seed, K, L), L)


def _random_cases(n, seed=2024):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        L = int(np.exp(rng.uniform(np.log(11), np.log(20000))))
        cases.append((int(rng.integers(0, 1 << 30)), int(rng.integers(1, 1500)), L))
    return cases


@pytest.mark.parametrize("seed,K,L", _random_cases(40))
def test_random_sets_cover_every_output(seed, K, L):
    """Generated sets at random sizes (L log-uniform from 11 to 20,000, K up
    to 1,500): MFMA, VALU and Toeplitz items in every mix the planner makes;
    every output computed once and every load inside the staged memory in
    both row layouts."""
    check_tables(rk.generate_kernels(seed, K, L), L)


@pytest.mark.parametrize("seed,K,L", [(11, 120, 11), (12, 150, 64), (13, 200, 300)])
def test_emulated_walk_matches_oracle(oracle, seed, K, L):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((3, L)).cumsum(axis=1)
    X = ((X - X.mean(1, keepdims=True)) / X.std(1, keepdims=True)).astype(np.float32)
    check_tables(rk.generate_kernels(seed, K, L), L, X, oracle)


def test_hand_built_lengths_and_extremes(oracle):
    """Every length 1..11, dilations up to the largest admissible, and the
    O = 1 extreme, including lengths the generator never draws."""
    rng = np.random.default_rng(3)
    L = 40
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in range(1, 12):
        dmax = (L - 1) // max(1, ln - 1) if ln > 1 else 9
        for d in sorted({1, 2, dmax, max(1, dmax // 2)}):
            for padded in (0, 1):
                p = (ln - 1) * d // 2 if padded else 0
                lengths.append(ln)
                dil.append(d)
                pad.append(p)
                bias.append(float(rng.uniform(-1, 1)))
                weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    X = rng.standard_normal((2, L)).astype(np.float32)
    check_tables(ks, L, X, oracle)


def test_item_cost_and_groups():
    ks = rk.generate_kernels(203, 10000, 1000)
    t = rk.plan_tables(ks, 1000)
    toep = t["items"][:, 0] >= TOEP0       # Toeplitz items: checked by walk_toeplitz
    items = t["items"][~toep]
    info = np.array([variant_info(int(v)) for v in items[:, 0]])
    ell, G, nk = info[:, 0], info[:, 1], info[:, 2]
    O, n_tiles = items[:, 3], items[:, 4]
    np.testing.assert_array_equal(n_tiles, (O + TILE - 1) // TILE)
    mf = nk == 0
    np.testing.assert_array_equal(items[mf, 7], (n_tiles * ell * G * items[:, 8])[mf])
    np.testing.assert_array_equal(items[~mf, 7], ((n_tiles * ell * nk + 1) // 2)[~mf])
    # a bucket is split into groups of 8 with at most one smaller group,
    # whose one or two last kernels run as a VALU or a Toeplitz item
    assert (G[mf] == 2).sum() > (G[mf] == 1).sum() and (~mf).sum() > 0
    # FMA work issued (an MFMA: 4 slots x 64 lanes; a VALU FMA: 64 lanes;
    # a Toeplitz item's cost counts its MFMAs) stays within 12% of the
    # nominal taps x outputs
    nominal = (ks["length"] * (1000 + 2 * ks["padding"] - (ks["length"] - 1) * ks["dilation"])).sum()
    issued = ((n_tiles * ell * G * 256)[mf].sum() + (n_tiles * ell * nk * 64)[~mf].sum()
              + (t["items"][toep, 7] * 256).sum())
    assert issued < 1.12 * nominal


def test_centred_kernels_fill_longer_frames():
    """Centred kernels of a shorter length fill the empty slots of a longer
    frame at the same dilation when that saves a group: one 11-tap, two
    9-tap and one 7-tap kernel at d = 2 run as one 4-slot group of 11 taps."""
    rng = np.random.default_rng(8)
    L = 50
    lengths = [11, 9, 9, 7, 9]
    dil = [2, 2, 2, 2, 3]
    pad = [(ln - 1) * d // 2 for ln, d in zip(lengths, dil)]
    ks = kernel_set(lengths, dil, pad, rng.uniform(-1, 1, 5), [rng.standard_normal(n) for n in lengths])
    t = check_tables(ks, L)
    items = t["items"]
    assert items.shape[0] == 2
    by_d = {int(r[1]): r for r in items}
    assert ELLS[by_d[2][0] // 2] == 11 and by_d[2][0] % 2 == 0 and by_d[2][2] == 10
    assert ELLS[by_d[3][0] // 2] == 9


def test_ppv_through_double_reciprocal():
    """The kernel writes PPV as (float)(c * fl64(1/O)); for 0 <= c <= O < 2^24
    that equals the correctly rounded fp32 quotient (float)c / (float)O.
    Exhaustive for O < 1200, then random (c, O) pairs up to 2^24 - 1."""
    rng = np.random.default_rng(5)
    cs = []
    for O in range(1, 1200):
        cs.append(np.arange(O + 1))
    O_all = np.concatenate([np.full(O + 1, O) for O in range(1, 1200)])
    c_all = np.concatenate(cs)
    O_r = rng.integers(1, 1 << 24, size=2_000_000)
    c_r = (rng.random(O_r.shape[0]) * (O_r + 1)).astype(np.int64)
    O_all = np.concatenate([O_all, O_r, np.full(4, (1 << 24) - 1)])
    c_all = np.concatenate([c_all, c_r, [1, 2, (1 << 23), (1 << 24) - 2]])
    want = c_all.astype(np.float32) / O_all.astype(np.float32)
    got = (c_all.astype(np.float64) * (1.0 / O_all.astype(np.float64))).astype(np.float32)
    assert np.array_equal(want, got)


@pytest.mark.parametrize("seed,K,L,C", [(21, 200, 60, 3), (22, 300, 150, 6)])
def test_multichannel_walk_matches_oracle(oracle, seed, K, L, C):
    """Multivariate sets: every item's channel list is the union of its
    kernels' channels, the packed weights are each kernel's row for each
    channel (zero for channels it does not read), and the replay over
    channels then taps lands inside the oracle's bounds."""
    rng = np.random.default_rng(seed)
    ks = rk.generate_kernels_multi(seed, K, L, C)
    X = rng.standard_normal((3, C, L)).cumsum(axis=2)
    X = ((X - X.mean(2, keepdims=True)) / X.std(2, keepdims=True)).astype(np.float32)
    check_tables(ks, L, X, oracle)


def test_multichannel_generator_matches_oracle():
    from oracle import rocket_oracle as o
    for C in (2, 5, 32):
        a = rk.generate_kernels_multi(77, 300, 500, C)
        b = o.generate_kernels_multi(77, 300, 500, C)
        for key in ("length", "dilation", "padding", "bias", "channel_count", "channel_index", "weights"):
            assert np.array_equal(a[key], b[key]), (C, key)


def _multichannel_set(chan_sets, C, L, seed, length=9, dilation=1, padding=0):
    """A hand-built multivariate set: kernel i reads the channels chan_sets[i]."""
    rng = np.random.default_rng(seed)
    K = len(chan_sets)
    count = np.array([len(s) for s in chan_sets], dtype=np.int32)
    index = np.zeros((K, C), dtype=np.int32)
    W = np.zeros((K, C, 11), dtype=np.float32)
    for i, s in enumerate(chan_sets):
        index[i, :len(s)] = sorted(s)
        W[i, :len(s), :length] = rng.standard_normal((len(s), length))
    return dict(length=np.full(K, length, np.int32), dilation=np.full(K, dilation, np.int32),
                padding=np.full(K, padding, np.int32), bias=rng.uniform(-1, 1, K).astype(np.float32),
                weights=W, n_channels=C, channel_count=count, channel_index=index, input_length=L)


def test_multichannel_groups_share_channels():
    """Multivariate buckets are cut into 4-kernel items whose channel unions
    stay small: eight kernels of one bucket reading {0,1}, {2,3}, {0}, {2},
    {1}, {3}, {0,1}, {2,3} form two items, each over 2 channels (one item of
    eight would run both of its groups over all 4 channels)."""
    sets = [{0, 1}, {2, 3}, {0}, {2}, {1}, {3}, {0, 1}, {2, 3}]
    L = 40
    ks = _multichannel_set(sets, 4, L, 5)
    t = check_tables(ks, L)
    items = t["items"]
    assert items.shape[0] == 2
    assert (items[:, 0] % 2 == 0).all()          # 4-kernel items
    assert sorted(items[:, 8].tolist()) == [2, 2]  # two channels each
    unions = []
    for r in items:
        chans = set(int(c) for c in t["chan"][r[9]:r[9] + r[8]])
        kids = [int(x) for x in t["slot_kernel"][r[6]:r[6] + 4] if x >= 0]
        assert set().union(*(sets[k] for k in kids)) == chans
        # the channel mask the fused kernel iterates holds the same channels
        mask = int(r[12]) | (int(r[13]) << 32)
        assert mask == sum(1 << c for c in chans)
        unions.append(frozenset(chans))
    assert set(unions) == {frozenset({0, 1}), frozenset({2, 3})}


def test_multichannel_issued_work():
    """The multivariate benchmark's kernel set (10,000 kernels, 6 channels,
    L = 500): MFMA work issued over the channel unions stays within 1.5x of
    the valid (kernel, channel, tap, output) products."""
    from paper_2601_17091_amd.workloads import WORKLOADS
    w = WORKLOADS["multivariate"]
    ks = rk.generate_kernels_multi(w.kernel_seed, w.n_kernels, w.L, w.channels)
    items = rk.plan_tables(ks, w.L)["items"]
    assert (items[:, 0] % 2 == 0).all()
    valid = (ks["channel_count"].astype(np.int64) * ks["length"] *
             (w.L + 2 * ks["padding"] - (ks["length"] - 1) * ks["dilation"])).sum()
    assert items[:, 7].sum() * 256 < 1.42 * valid


def test_multichannel_grouping_is_deterministic():
    """The channel grouping's random swaps follow a fixed sequence: two
    builds of the same set give the same tables."""
    ks = rk.generate_kernels_multi(31, 2000, 300, 5)
    a, b = rk.plan_tables(ks, 300), rk.plan_tables(ks, 300)
    for key in ("items", "slot_kernel", "chan", "wpk", "order"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("seed,K,L", [(15, 300, 3000), (16, 400, 1500)])
def test_toeplitz_items_walk_matches_oracle(oracle, seed, K, L):
    """Long series: the one or two kernels left over in a bucket at a large
    dilation become Toeplitz items (one MFMA group, the kernel at 4 or 2 tap
    shifts); their walk covers every output once and lands in the oracle's
    certified bounds."""
    ks = rk.generate_kernels(seed, K, L)
    t = rk.plan_tables(ks, L)
    v = t["items"][:, 0]
    assert ((v >= 12) & (v % 2 == 0)).any() and ((v >= 12) & (v % 2 == 1)).any()
    X = np.random.default_rng(seed).standard_normal((3, L)).cumsum(axis=1).astype(np.float32)
    check_tables(ks, L, X, oracle)


def test_toeplitz_hand_built_dilations(oracle):
    """Singles and pairs at dilations around multiples of 64 (chunks filled
    exactly, or with 1 or 63 positions in the last chunk), padded and not,
    with O just above and below multiples of the super-tile span."""
    rng = np.random.default_rng(17)
    L = 1300
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in (7, 9, 11):
        for d in (60, 64, 65, 100, 127, 128, 129):
            if (ln - 1) * d >= L:
                continue
            for padded in (0, 1):
                for _ in range(1 + (d % 2)):          # singles and pairs
                    lengths.append(ln)
                    dil.append(d)
                    pad.append((ln - 1) * d // 2 if padded else 0)
                    bias.append(float(rng.uniform(-1, 1)))
                    weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    t = rk.plan_tables(ks, L)
    v = t["items"][:, 0]
    assert ((v >= 12) & (v % 2 == 0)).sum() >= 2 and ((v >= 12) & (v % 2 == 1)).sum() >= 2
    X = rng.standard_normal((4, L)).astype(np.float32)
    check_tables(ks, L, X, oracle)


def series_block_reads(b0j, n, L):
    """Positions read by a series-lane block of n positions under a tap whose
    first position is b0j, [tap, position]: the start is clamped into
    [-SERIES_MARGIN, L] (a block moved by the clamp lies wholly outside the
    series and reads margin zeros)."""
    b = np.clip(b0j, -SERIES_MARGIN, L)
    return b[:, None] + np.arange(n)[None, :]


@pytest.mark.parametrize("seed,K,L", [(21, 500, 11), (22, 800, 30), (23, 1000, 64), (24, 1000, 100),
                                      (25, 1000, 128)] + [(30 + i, 600, 11 + 13 * i) for i in range(9)])
def test_series_lane_reads_stay_staged(seed, K, L):
    """The series-lane kernel walks an item's O positions in blocks of NT
    (8 for 4-kernel items, 4 for 8-kernel items; the last block holds the
    rest), and for tap j a block starting at output t0 reads positions
    t0 - p + j*d onwards.  Every read stays inside the staged positions
    [-SERIES_MARGIN, L + SERIES_MARGIN), reads the series position itself
    where that lies inside the series, and a margin zero where not."""
    t = rk.plan_tables(rk.generate_kernels(seed, K, L), L)
    for row in t["items"]:
        f = item_fields(row)
        ell, G, nk = variant_info(f["variant"])
        assert nk == 0 and f["variant"] < 6  # series this short have MFMA items only
        NT = TILES_PER_BLOCK[G]
        assert NT <= SERIES_MARGIN
        for start in range(0, f["O"], NT):
            n = min(NT, f["O"] - start)
            b0j = start - f["p"] + np.arange(ell) * f["d"]
            pos = series_block_reads(b0j, n, L)
            assert pos.min() >= -SERIES_MARGIN and pos.max() < L + SERIES_MARGIN
            true = b0j[:, None] + np.arange(n)[None, :]
            inside = (true >= 0) & (true < L)
            assert np.array_equal(pos[inside], true[inside])
            assert np.all((pos[~inside] < 0) | (pos[~inside] >= L))
