"""Host logic of the fused kernel, checked on the CPU.

The planner's tables (work items, lane tables, packed weights, item orders)
are read back through rocket_plan_tables_build and walked here exactly the
way the GPU kernel walks them: in every round each active lane takes the
output positions q0, q0+d, ... (S or S-1 of them, by round) and loads the
series values at halo_lo - p + q + j*d from the zero-margined row; lanes
past the round's chunk count are discarded.  The checks: every position an
active lane computes is a real output, every output of every kernel is
computed exactly once, every load (idle lanes included) stays inside the
staged row, the packed weights are the kernels' own, and an fp32 replay of
the walk lands inside the oracle's certified bounds.
"""
import numpy as np
import pytest

import paper_2601_17091_amd as rk
from _util import kernel_set

ELLS = (7, 9, 11)


def walk(tables, kernels, L, X=None):
    """Replay the fused kernel's schedule; returns per-kernel coverage and,
    if X is given, fp32 features [n, 2K]."""
    K = len(kernels["length"])
    items = tables["items"]
    lanes = tables["lanes"].astype(np.int64)
    halo_lo, stride = tables["halo_lo"], tables["row_stride"]
    cover = [np.zeros(0, np.int64)] * K
    F = None
    if X is not None:
        n = X.shape[0]
        F = np.full((n, 2 * K), np.nan, dtype=np.float64)
        rows = np.zeros((n, stride), dtype=np.float32)
        rows[:, halo_lo:halo_lo + L] = X
    for it in items:
        (variant, d, p, O, S, rounds, lane_off, w_off, k_off, cost, n_long, n_short,
         rounds_long) = (int(v) for v in it[:13])
        ell = ELLS[variant // 2]
        G = variant % 2 + 1
        nslot = 4 * G
        kid = tables["slot_kernel"][k_off:k_off + nslot]
        bias = tables["slot_bias"][k_off:k_off + nslot]
        W = tables["wpk"][w_off:w_off + G * ell * 4].reshape(G, ell, 4)
        Wslot = np.concatenate([W[g].T for g in range(G)], axis=0)  # [slot, tap]
        for s_, k in enumerate(kid):
            if k >= 0:
                ln = int(kernels["length"][k])
                assert np.array_equal(Wslot[s_, :ln], kernels["weights"][k, :ln])
                assert np.all(Wslot[s_, ln:] == 0)
                assert bias[s_] == np.float32(kernels["bias"][k])
                assert (int(kernels["dilation"][k]), int(kernels["padding"][k])) == (d, p)
            else:
                assert np.all(Wslot[s_] == 0)
        assert rounds == rounds_long + -(-n_short // 64) and rounds_long == -(-n_long // 64)
        assert cost == (rounds_long * S + (rounds - rounds_long) * (S - 1)) * ell * G
        counted = []
        ys = [] if X is not None else None
        for rd in range(rounds):
            is_long = rd < rounds_long
            length = S if is_long else S - 1
            active = min(64, n_long - 64 * rd) if is_long else min(64, n_short - 64 * (rd - rounds_long))
            assert length >= 1 and active >= 1
            q0 = lanes[lane_off + 64 * rd:lane_off + 64 * rd + 64]
            q = q0[:, None] + np.arange(length)[None, :] * d        # [lane, step]
            # every lane's loads stay in the staged row, idle lanes included
            m = np.arange(length + ell - 1)
            idx = halo_lo - p + q0[:, None] + m[None, :] * d
            assert idx.min() >= 0 and idx.max() < stride, (d, p, O, S)
            qa = q[:active]
            assert qa.min() >= 0 and qa.max() < O                    # real outputs only
            counted.append(qa.ravel())
            if X is not None:
                tap_idx = halo_lo - p + qa[..., None] + np.arange(ell)[None, None, :] * d
                xv = rows[:, tap_idx]                                # [n, lane, step, tap]
                acc = np.broadcast_to(bias.astype(np.float32), xv.shape[:3] + (nslot,)).copy()
                for j in range(ell):
                    acc = (acc + xv[..., j, None] * Wslot[None, None, None, :, j]).astype(np.float32)
                ys.append(acc.reshape(acc.shape[0], -1, nslot))
        allq = np.concatenate(counted)
        for k in kid[kid >= 0]:
            cover[k] = np.bincount(allq, minlength=O)
        if X is not None:
            y = np.concatenate(ys, axis=1)                               # [n, outputs, slot]
            cnt = (y > 0).sum(axis=1)
            mxv = y.max(axis=1)
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
        beg = t["split_begin"][t["layout_off"][li]:t["layout_off"][li] + 6 * ns + 1]
        ids = []
        for v in range(6):
            for s_ in range(ns):
                part = t["order"][beg[v * ns + s_]:beg[v * ns + s_ + 1]]
                assert np.all(t["items"][part, 0] == v)
                ids.append(part)
        assert np.array_equal(np.sort(np.concatenate(ids)), np.arange(n_items))
    # every kernel sits in exactly one slot
    kid = t["slot_kernel"]
    assert np.array_equal(np.sort(kid[kid >= 0]), np.arange(K))
    cover, F = walk(t, kernels, L, X)
    for k in range(K):
        O = L + 2 * int(kernels["padding"][k]) - (int(kernels["length"][k]) - 1) * int(kernels["dilation"][k])
        assert cover[k].shape[0] == O and np.all(cover[k] == 1), k
    if X is not None:
        r = oracle.transform(X, kernels)
        cnt = np.rint(F[:, 0::2] * r["O"][None, :]).astype(np.int64)
        assert np.all(r["cnt_lo"] <= cnt) and np.all(cnt <= r["cnt_hi"])
        assert np.all(np.abs(F[:, 1::2] - r["F"][:, 1::2]) <= r["beta"])
    return t


@pytest.mark.parametrize("seed,K,L", [(1, 300, 11), (2, 300, 30), (3, 400, 64), (4, 500, 128),
                                      (5, 400, 500), (6, 300, 1000), (7, 200, 3000)])
def test_generated_sets_cover_every_output(seed, K, L):
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
    items = t["items"]
    G = items[:, 0] % 2 + 1
    ell = np.array(ELLS)[items[:, 0] // 2]
    S, rounds, rounds_long = items[:, 4], items[:, 5], items[:, 12]
    steps = rounds_long * S + (rounds - rounds_long) * (S - 1)
    np.testing.assert_array_equal(items[:, 9], steps * ell * G)
    # a bucket is split into groups of 8 with at most one smaller group
    assert (G == 2).sum() > (G == 1).sum()
