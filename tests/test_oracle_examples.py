"""Oracle pinned to hand-computed worked examples (tests/golden/) and to a
literal brute-force loop on small random cases."""
import numpy as np
import pytest

from _util import brute_force, brute_force_mpv, kernel_set, load_golden, random_kernels

GOLDEN = load_golden()


@pytest.mark.parametrize("ex", GOLDEN, ids=[g["name"] for g in GOLDEN])
def test_worked_example(oracle, ex):
    X = np.asarray(ex["x"], dtype=np.float32)[None, :]
    assert X.shape[1] == int(ex["L"])
    ks = kernel_set([len(ex["w"])], [int(ex["dilation"])], [int(ex["padding"])], [ex["b"]], [ex["w"]])
    r = oracle.transform(X, ks)
    y = np.atleast_1d(np.asarray(ex["y"], dtype=np.float64))
    assert r["O"][0] == len(y)
    assert r["F"][0, 0] == pytest.approx(ex["ppv"], abs=1e-15)
    assert r["F"][0, 1] == ex["max"]
    assert r["cnt"][0, 0] == int((y > 0).sum())
    # MPV: the mean of the fixture's positive dot products (0 when none)
    pos = y[y > 0]
    assert r["mpv"][0, 0] == pytest.approx(pos.mean() if pos.size else 0.0, abs=1e-12)
    # the convolution (reversed-weight) reading must not reproduce these
    if (ex["flipped_ppv"], ex["flipped_max"]) != (ex["ppv"], ex["max"]):
        assert (r["F"][0, 0], r["F"][0, 1]) != pytest.approx((ex["flipped_ppv"], ex["flipped_max"]))


def test_worked_examples_flipped_reading(oracle):
    """Feeding reversed weights reproduces the fixture's 'flipped' features,
    which shows the fixtures discriminate the two orientations."""
    for ex in GOLDEN:
        X = np.asarray(ex["x"], dtype=np.float32)[None, :]
        ks = kernel_set([len(ex["w"])], [int(ex["dilation"])], [int(ex["padding"])], [ex["b"]],
                        [list(reversed(ex["w"]))])
        r = oracle.transform(X, ks)
        assert r["F"][0, 0] == pytest.approx(ex["flipped_ppv"], abs=1e-15), ex["name"]
        assert r["F"][0, 1] == ex["flipped_max"], ex["name"]


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_random(oracle, seed):
    rng = np.random.default_rng(1000 + seed)
    L = int(rng.integers(11, 33))
    n = int(rng.integers(1, 4))
    K = int(rng.integers(5, 50))
    X = rng.standard_normal((n, L)).astype(np.float32)
    ks = random_kernels(rng, K, L)
    r = oracle.transform(X, ks)
    ref = brute_force(X, ks)
    np.testing.assert_allclose(r["F"][:, 1::2], ref[:, 1::2], rtol=0, atol=1e-12)
    np.testing.assert_array_equal(r["F"][:, 0::2], ref[:, 0::2])
    np.testing.assert_allclose(r["mpv"], brute_force_mpv(X, ks), rtol=0, atol=1e-12)


def test_row_subset_matches_full(oracle):
    rng = np.random.default_rng(5)
    X = rng.standard_normal((9, 40)).astype(np.float32)
    ks = random_kernels(rng, 20, 40)
    full = oracle.transform(X, ks)
    rows = np.array([8, 0, 3, 3])
    sub = oracle.transform(X, ks, rows=rows)
    np.testing.assert_array_equal(sub["F"], full["F"][rows])
    np.testing.assert_array_equal(sub["cnt_lo"], full["cnt_lo"][rows])


def test_rejects_kernel_without_dot_products(oracle):
    X = np.zeros((1, 10), dtype=np.float32)
    ks = kernel_set([7], [2], [0], [0.0], [[1] * 7])  # O = 10 - 12 < 1
    with pytest.raises(ValueError):
        oracle.transform(X, ks)
