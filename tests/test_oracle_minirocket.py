"""MINIROCKET oracle pinned to closed forms, hand-worked fits, library
routines and the independent ROCKET oracle.

MINIROCKET is the variant the CUROCKET paper names in Sec. 5; its definition
is the published one (84 fixed 9-tap kernels with weights -1 and 2,
exponentially spaced dilations, quantile biases, PPV features).  Each check
targets a plausible slip: a wrong weight or tap choice, a padding flag on the
wrong pairs, a wrong output count, a quantile off by one order statistic, or
a bias drawn from the wrong series.
"""
import math

import numpy as np
import pytest
import torch

from _util import kernel_set


@pytest.fixture(scope="module")
def mo(oracle):
    from oracle import minirocket_oracle
    return minirocket_oracle


def test_kernels_are_the_84_choices(mo):
    w = mo.kernel_weights()
    assert w.shape == (84, 9)
    assert np.all((w == 2.0).sum(axis=1) == 3) and np.all((w == -1.0).sum(axis=1) == 6)
    np.testing.assert_array_equal(w.sum(axis=1), np.zeros(84))
    assert len({tuple(r) for r in w}) == 84
    ch = mo.kernel_choices()
    assert ch[0] == (0, 1, 2) and ch[1] == (0, 1, 3) and ch[-1] == (6, 7, 8) and ch == sorted(ch)


def test_kernel_outputs_sum_to_zero(mo):
    """Every tap is chosen by 28 of the 84 kernels, so summed over the 84
    kernels the dot products are -84 S + 3 * 28 S = 0 at every position (S the
    sum of the 9 series values under the taps)."""
    x = np.random.default_rng(1).standard_normal(60).astype(np.float32)
    for d in (1, 3, 7):
        tot = sum(mo.same_convolution(x, k, d) for k in range(84))
        assert np.abs(tot).max() <= 1e-12 * np.abs(x).sum() * 84


def test_same_convolution_matches_conv1d(mo):
    rng = np.random.default_rng(2)
    x = rng.standard_normal(50).astype(np.float32)
    w = mo.kernel_weights()
    for k in (0, 17, 83):
        for d in (1, 2, 6):
            ref = torch.nn.functional.conv1d(torch.from_numpy(x.astype(np.float64))[None, None],
                                             torch.from_numpy(w[k])[None, None], padding=4 * d,
                                             dilation=d)[0, 0].numpy()
            np.testing.assert_allclose(mo.same_convolution(x, k, d), ref, rtol=0, atol=1e-12)


def test_fit_dilations_hand_worked(mo):
    """L = 9: log2((L-1)/8) = 0, every one of the 32 grid points is 2^0 = 1:
    one dilation with all 119 features.  L = 17: exponents i/31, i = 0..31;
    only the last reaches 2, so counts (31, 1), scaled by 119/32 = 3.71875
    and truncated to (115, 3), the one left over going to the first."""
    d, f = mo.fit_dilations(9, 10000)
    assert d.tolist() == [1] and f.tolist() == [119]
    d, f = mo.fit_dilations(17, 10000)
    assert d.tolist() == [1, 2] and f.tolist() == [116, 3]
    # 840 features: 10 per kernel on 10 grid points 2^(7i/9) (multiplier 1):
    # 1, 1.71, 2.94, 5.04, 8.64, 14.8, 25.4, 43.5, 74.7, 128 -> the two 1s merge
    d, f = mo.fit_dilations(1025, 840)
    assert d.tolist() == [1, 2, 5, 8, 14, 25, 43, 74, 128] and f.tolist() == [2, 1, 1, 1, 1, 1, 1, 1, 1]


@pytest.mark.parametrize("L,nf", [(9, 84), (40, 1000), (500, 10000), (1000, 10000), (16384, 10000),
                                  (64, 10000), (2000, 50000)])
def test_fit_dilations_properties(mo, L, nf):
    d, f = mo.fit_dilations(L, nf)
    assert int(f.sum()) == nf // 84
    assert d[0] == 1 and np.all(np.diff(d) > 0) and d[-1] <= (L - 1) // 8
    assert len(d) <= 32 and np.all(f >= 1)


def test_quantile_positions_closed_form(mo):
    q = mo.quantile_positions(5)
    phi = (1 + 5 ** 0.5) / 2
    want = [m * phi - math.floor(m * phi) for m in range(1, 6)]
    np.testing.assert_allclose(q, want, rtol=0, atol=6e-8)
    assert abs(float(q[0]) - 0.6180339887) < 1e-7 and abs(float(q[1]) - 0.2360679775) < 1e-7


def test_quantile_linear_matches_numpy(mo):
    rng = np.random.default_rng(4)
    for n in (1, 2, 7, 100, 999):
        s = np.sort(rng.standard_normal(n))
        for q in np.concatenate([rng.random(20), [0.0, 1.0, 0.5]]):
            ref = float(np.quantile(s, q))
            assert abs(mo.quantile_linear(s, q) - ref) <= 1e-12 * (1 + abs(ref))


def _brute(mo, X, params):
    """Literal loops over pairs, positions and taps."""
    L = X.shape[1]
    w = mo.kernel_weights()
    out = []
    for x in X.astype(np.float64):
        row = []
        f = 0
        for i, d in enumerate(params["dilations"]):
            d = int(d)
            for k in range(84):
                p = 4 * d if (i + k) % 2 == 0 else 0
                O = L + 2 * p - 8 * d
                C = []
                for t in range(O):
                    s = 0.0
                    for j in range(9):
                        idx = t - p + j * d
                        s += w[k, j] * (x[idx] if 0 <= idx < L else 0.0)
                    C.append(s)
                for _ in range(int(params["features_per_dilation"][i])):
                    row.append(sum(c > float(params["biases"][f]) for c in C) / O)
                    f += 1
        out.append(row)
    return np.array(out)


def test_transform_matches_brute_force(mo):
    rng = np.random.default_rng(5)
    X = rng.standard_normal((4, 30)).astype(np.float32)
    params = mo.fit(X, 300, seed=9)
    # 3 per kernel on the grid 2^0, 2^0.929, 2^1.858 = 1, 1.90, 3.63
    assert params["dilations"].tolist() == [1, 3] and params["features_per_dilation"].tolist() == [2, 1]
    np.testing.assert_array_equal(mo.transform(X, params)["F"], _brute(mo, X, params))


def test_transform_matches_rocket_oracle(mo, oracle):
    """Feature (i, k, q) is the ROCKET PPV of the 9-tap kernel with weights
    w_k, bias -b, dilation d_i and padding 4 d_i (i + k even) or 0: the
    independent ROCKET oracle gives the same counts up to its certified
    rounding range."""
    rng = np.random.default_rng(6)
    X = rng.standard_normal((3, 120)).cumsum(axis=1).astype(np.float32)
    params = mo.fit(X, 2000, seed=1)
    lay = mo.feature_layout(params)
    w = mo.kernel_weights()
    d = params["dilations"][lay["dilation_index"]]
    ks = kernel_set([9] * len(d), d, np.where(lay["padded"], 4 * d, 0), -params["biases"].astype(np.float64),
                    [w[k] for k in lay["kernel"]])
    r_ro = oracle.transform(X, ks)
    r_mr = mo.transform(X, params)
    np.testing.assert_array_equal(r_mr["O"], r_ro["O"])
    assert np.all(r_mr["cnt"] >= r_ro["cnt_lo"]) and np.all(r_mr["cnt"] <= r_ro["cnt_hi"])
    assert np.mean(r_mr["cnt"] == r_ro["cnt"]) > 0.999


def test_fit_example_features_are_its_quantile_ranks(mo):
    """One training series: every pair's biases are quantiles of that
    series' own padded dot products.  Transforming it back, a padded pair's
    feature for position q counts the values above the q-quantile:
    L - 1 - floor(q (L - 1)) for distinct values (the fp32 rounding of the
    bias may move it by one)."""
    rng = np.random.default_rng(7)
    L = 80
    X = rng.standard_normal((1, L)).astype(np.float32)
    params = mo.fit(X, 840, seed=2)
    assert np.all(params["examples"] == 0)
    r = mo.transform(X, params)
    lay = mo.feature_layout(params)
    qpos = mo.quantile_positions(params["biases"].shape[0]).astype(np.float64)
    pad = lay["padded"]
    want = L - 1 - np.floor(qpos * (L - 1))
    got = r["cnt"][0]
    assert np.all(np.abs(got[pad] - want[pad]) <= 1)
    assert np.mean(got[pad] == want[pad]) > 0.95


def test_constant_series_unpadded_pairs(mo):
    """A constant series: unpadded pairs see only interior positions, where
    the dot products are c * sum(w) = 0, so their features are [0 > b]."""
    rng = np.random.default_rng(8)
    X = rng.standard_normal((5, 64)).astype(np.float32)
    params = mo.fit(X, 1000, seed=3)
    Xc = np.full((1, 64), 1.75, np.float32)
    r = mo.transform(Xc, params)
    lay = mo.feature_layout(params)
    un = ~lay["padded"]
    np.testing.assert_array_equal(r["F"][0, un], (params["biases"][un] < 0).astype(float))


def test_examples_drawn_from_the_counter_stream(mo):
    rng = np.random.default_rng(10)
    X = rng.standard_normal((37, 200)).astype(np.float32)
    a = mo.fit(X, 1000, seed=5)
    b = mo.fit(X, 1000, seed=5)
    np.testing.assert_array_equal(a["biases"], b["biases"])
    ex = a["examples"]
    assert ex.min() >= 0 and ex.max() < 37 and len(np.unique(ex)) > 20
    # the draw is element i*84 + k of the SplitMix64 stream, scaled to 37
    from oracle import rocket_oracle as ro
    v = ro.splitmix64_at(5, 2 * 84 + 11)
    assert ex[2, 11] == (37 * (v >> 11)) >> 53
    assert not np.array_equal(mo.fit(X, 1000, seed=6)["biases"], a["biases"])
