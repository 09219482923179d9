"""Oracle pinned to closed forms, invariants and library routines.

Each check targets a plausible slip in the oracle: a dropped bias, a wrong
sign or stride in the tap index, a wrong output count, a non-strict
positivity test, a wrong PPV denominator, or an error bound that real fp32
arithmetic escapes.
"""
import numpy as np
import pytest
import torch

from _util import fp32_features, kernel_set, random_kernels, z_norm


def _gen(oracle, seed, K, L):
    return oracle.generate_kernels(seed, K, L)


def test_zero_series_gives_bias(oracle):
    """X = 0: every dot product equals the bias (Sec. 2.1), so MAX = b exactly
    and PPV = [b > 0]."""
    ks = _gen(oracle, 3, 300, 200)
    X = np.zeros((2, 200), dtype=np.float32)
    r = oracle.transform(X, ks)
    b = ks["bias"].astype(np.float64)
    np.testing.assert_array_equal(r["F"][:, 1::2], np.broadcast_to(b, (2, 300)))
    np.testing.assert_array_equal(r["F"][:, 0::2], np.broadcast_to((b > 0).astype(float), (2, 300)))
    # MPV: the mean of O copies of b when b > 0, else no positive value
    np.testing.assert_array_equal(r["mpv"], np.broadcast_to(np.where(b > 0, b, 0.0), (2, 300)))


def test_zero_bias_zero_series_is_not_positive(oracle):
    """y = 0 exactly is not a positive value: PPV counts y > 0 strictly."""
    ks = kernel_set([9, 7], [1, 3], [4, 0], [0.0, 0.0], [[1.0] * 9, [-1.0] * 7])
    r = oracle.transform(np.zeros((1, 40), np.float32), ks)
    assert r["F"][0, 0] == 0.0 and r["F"][0, 2] == 0.0
    assert r["F"][0, 1] == 0.0 and r["F"][0, 3] == 0.0


def test_constant_series_unpadded(oracle):
    """Constant X = c, unpadded kernel: y_t = b + c * sum(w) for every t.  With
    mean-centred weights this is b up to fp32 rounding of the centring, so
    MAX = b within |c| * |sum w| and PPV = [b > 0]."""
    ks = _gen(oracle, 4, 500, 300)
    X = np.full((1, 300), 1.75, dtype=np.float32)
    r = oracle.transform(X, ks)
    unp = ks["padding"] == 0
    sw = ks["weights"].astype(np.float64).sum(axis=1)
    b = ks["bias"].astype(np.float64)
    exp_max = b + 1.75 * sw
    np.testing.assert_allclose(r["F"][0, 1::2][unp], exp_max[unp], rtol=0, atol=1e-14)
    assert np.all(np.abs(r["F"][0, 1::2][unp] - b[unp]) <= 1.75 * np.abs(sw[unp]) + 1e-15)
    assert np.all(np.abs(sw) < 1e-5)
    clear = unp & (np.abs(b) > 1e-4)
    np.testing.assert_array_equal(r["F"][0, 0::2][clear], (b[clear] > 0).astype(float))


def test_one_hot_closed_form(oracle):
    """X = a e_m: y_t = b + a w_j for the single tap j with t - p + j d = m,
    else y_t = b.  Written as a direct formula over t, not a tap loop."""
    rng = np.random.default_rng(11)
    L = 57
    ks = random_kernels(rng, 40, L)
    for m in (0, 13, 56):
        X = np.zeros((1, L), np.float32)
        X[0, m] = 2.5
        r = oracle.transform(X, ks)
        for k in range(40):
            ln, d, p = int(ks["length"][k]), int(ks["dilation"][k]), int(ks["padding"][k])
            b = float(ks["bias"][k])
            O = L + 2 * p - (ln - 1) * d
            t = np.arange(O)
            num = m - t + p
            j = num // d
            hit = (num % d == 0) & (j >= 0) & (j < ln)
            y = np.where(hit, b + 2.5 * ks["weights"][k][np.clip(j, 0, ln - 1)].astype(np.float64), b)
            assert r["F"][0, 2 * k + 1] == pytest.approx(y.max(), abs=1e-15)
            assert r["cnt"][0, k] == int((y > 0).sum())


def test_reverse_symmetry(oracle):
    """Reversing both the series and the weights reverses the run of dot
    products (t -> O-1-t), for padded and unpadded kernels alike."""
    ks = _gen(oracle, 8, 400, 150)
    rng = np.random.default_rng(8)
    X = z_norm(rng.standard_normal((3, 150)).cumsum(axis=1))
    rk = dict(ks)
    W = np.zeros_like(ks["weights"])
    for k in range(400):
        ln = int(ks["length"][k])
        W[k, :ln] = ks["weights"][k, :ln][::-1]
    rk["weights"] = W
    a = oracle.transform(X, ks)
    b = oracle.transform(np.ascontiguousarray(X[:, ::-1]), rk)
    np.testing.assert_allclose(a["F"][:, 1::2], b["F"][:, 1::2], rtol=0, atol=1e-12)
    np.testing.assert_array_equal(a["cnt"], b["cnt"])


def test_decimation_identity(oracle):
    """Unpadded dilation d on X equals dilation 1 on each residue subsequence
    X[r::d]: max of the maxima, sum of the counts and of the output lengths."""
    rng = np.random.default_rng(21)
    L = 200
    X = z_norm(rng.standard_normal((2, L)))
    for ln, d in ((7, 3), (9, 5), (11, 17), (7, 33)):
        w = rng.standard_normal(ln).astype(np.float32)
        b = float(rng.uniform(-1, 1))
        full = oracle.transform(X, kernel_set([ln], [d], [0], [b], [w]))
        cnt = np.zeros(2, dtype=np.int64)
        mx = np.full(2, -np.inf)
        total_O = 0
        for r in range(d):
            sub = np.ascontiguousarray(X[:, r::d])
            if sub.shape[1] - (ln - 1) < 1:
                continue
            part = oracle.transform(sub, kernel_set([ln], [1], [0], [b], [w]))
            cnt += part["cnt"][:, 0]
            mx = np.maximum(mx, part["F"][:, 1])
            total_O += int(part["O"][0])
        assert total_O == int(full["O"][0])
        np.testing.assert_array_equal(full["cnt"][:, 0], cnt)
        np.testing.assert_array_equal(full["F"][:, 1], mx)


def test_power_of_two_scaling(oracle):
    """b = 0: scaling X by 2^s scales every y_t exactly, so PPV is unchanged and
    MAX scales by 2^s."""
    ks = _gen(oracle, 9, 200, 120)
    ks = dict(ks)
    ks["bias"] = np.zeros_like(ks["bias"])
    rng = np.random.default_rng(9)
    X = z_norm(rng.standard_normal((2, 120)))
    a = oracle.transform(X, ks)
    for s in (-3, 5):
        b = oracle.transform((X * np.float32(2.0 ** s)).astype(np.float32), ks)
        np.testing.assert_array_equal(b["F"][:, 0::2], a["F"][:, 0::2])
        np.testing.assert_array_equal(b["F"][:, 1::2], a["F"][:, 1::2] * 2.0 ** s)
        np.testing.assert_array_equal(b["mpv"], a["mpv"] * 2.0 ** s)


def test_range_and_consistency(oracle):
    ks = _gen(oracle, 10, 1000, 256)
    rng = np.random.default_rng(10)
    X = z_norm(rng.standard_normal((4, 256)).cumsum(axis=1))
    r = oracle.transform(X, ks)
    ppv, mx = r["F"][:, 0::2], r["F"][:, 1::2]
    assert np.all((ppv >= 0) & (ppv <= 1))
    scaled = ppv * r["O"][None, :]
    np.testing.assert_array_equal(np.rint(scaled), r["cnt"])
    assert np.abs(scaled - r["cnt"]).max() < 1e-9
    np.testing.assert_array_equal(ppv > 0, mx > 0)
    assert np.all(r["cnt_lo"] <= r["cnt"]) and np.all(r["cnt"] <= r["cnt_hi"])
    # MPV is a mean of positive values: 0 exactly when PPV is 0, else in (0, MAX]
    mpv = r["mpv"]
    np.testing.assert_array_equal(mpv > 0, ppv > 0)
    assert np.all(mpv[ppv > 0] <= mx[ppv > 0] * (1 + 1e-15))
    assert np.all((r["mpv_lo"] <= mpv) & (mpv <= r["mpv_hi"]))


@pytest.mark.parametrize("seed", range(3))
def test_torch_conv1d_fp64(oracle, seed):
    """Library routine: torch conv1d (a cross-correlation) in fp64 with the
    kernel's padding and dilation gives the run of dot products."""
    rng = np.random.default_rng(30 + seed)
    L = int(rng.integers(60, 300))
    ks = oracle.generate_kernels(40 + seed, 60, L)
    X = z_norm(rng.standard_normal((3, L)).cumsum(axis=1))
    r = oracle.transform(X, ks)
    xt = torch.from_numpy(X.astype(np.float64))[:, None, :]
    for k in range(60):
        ln = int(ks["length"][k])
        w = torch.from_numpy(ks["weights"][k, :ln].astype(np.float64))[None, None, :]
        b = torch.tensor([float(ks["bias"][k])], dtype=torch.float64)
        y = torch.nn.functional.conv1d(xt, w, b, padding=int(ks["padding"][k]),
                                       dilation=int(ks["dilation"][k]))[:, 0, :].numpy()
        assert y.shape[1] == r["O"][k]
        assert np.abs(y).min() > 1e-9  # no value so close to 0 that order matters
        np.testing.assert_array_equal(r["cnt"][:, k], (y > 0).sum(axis=1))
        np.testing.assert_allclose(r["F"][:, 2 * k + 1], y.max(axis=1), rtol=0, atol=1e-12)


def test_numpy_correlate_dilation_one(oracle):
    """Dilation 1: 'valid' correlation is the unpadded kernel, 'same' the
    kernel padded by (l-1)/2."""
    rng = np.random.default_rng(44)
    x = z_norm(rng.standard_normal((1, 90)))
    for ln in (7, 9, 11):
        w = rng.standard_normal(ln).astype(np.float32)
        b = 0.1
        for p, mode in ((0, "valid"), ((ln - 1) // 2, "same")):
            r = oracle.transform(x, kernel_set([ln], [1], [p], [b], [w]))
            y = np.correlate(x[0].astype(np.float64), w.astype(np.float64), mode) + np.float64(np.float32(b))
            assert r["O"][0] == y.shape[0]
            assert r["cnt"][0, 0] == int((y > 0).sum())
            assert r["F"][0, 1] == pytest.approx(y.max(), abs=1e-12)


@pytest.mark.parametrize("order", ["ascending", "descending"])
def test_certified_bounds_hold_for_fp32(oracle, order):
    """Real fp32 evaluations, in two summation orders, land inside the oracle's
    certified count interval and MAX error bound."""
    rng = np.random.default_rng(50)
    L = 300
    ks = oracle.generate_kernels(51, 400, L)
    X = z_norm(rng.standard_normal((6, L)).cumsum(axis=1))
    r = oracle.transform(X, ks)
    cnt32, mx32, mpv32 = fp32_features(X, ks, order, with_mpv=True)
    assert np.all(r["cnt_lo"] <= cnt32) and np.all(cnt32 <= r["cnt_hi"])
    assert np.all(np.abs(mx32 - r["F"][:, 1::2]) <= r["beta"])
    assert np.all((r["mpv_lo"] <= mpv32) & (mpv32 <= r["mpv_hi"]))
    # and the MPV range is narrow where no output is within beta of zero
    tight = r["cnt_lo"] == r["cnt_hi"]
    width = (r["mpv_hi"] - r["mpv_lo"])[tight & (r["cnt"] > 0)] / r["mpv"][tight & (r["cnt"] > 0)]
    assert np.percentile(width, 99) < 2e-4 and width.max() < 1e-2
    # the interval is tight: it is a handful of outputs wide at most
    assert (r["cnt_hi"] - r["cnt_lo"]).max() <= 3
    assert r["beta"].max() < 1e-4
