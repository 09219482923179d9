"""The oracle's kernel generator pinned to the published SplitMix64 outputs and
to the distributions of Sec. 2.1 (statistical checks, fixed seeds)."""
import math

import numpy as np
import pytest


def test_splitmix64_known_answers(oracle):
    # First outputs of SplitMix64 started at state 0 (Vigna's reference code).
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [oracle.splitmix64_at(0, i) for i in range(3)] == expect


def test_reproducible_and_prefix_stable(oracle):
    a = oracle.generate_kernels(123, 50, 500)
    b = oracle.generate_kernels(123, 80, 500)
    for key in ("length", "dilation", "padding", "bias", "weights"):
        np.testing.assert_array_equal(a[key], b[key][:50])
    c = oracle.generate_kernels(124, 50, 500)
    assert not np.array_equal(a["weights"], c["weights"])


@pytest.fixture(scope="module")
def big(oracle):
    return oracle.generate_kernels(2024, 30000, 1000)


def test_length_uniform(big):
    counts = np.array([(big["length"] == v).sum() for v in (7, 9, 11)])
    assert counts.sum() == 30000
    expected = 10000.0
    chi2 = ((counts - expected) ** 2 / expected).sum()
    assert chi2 < 13.8  # chi-square, 2 dof, p = 0.001


def test_weights_centred_normal(big):
    ln = big["length"]
    W = big["weights"].astype(np.float64)
    for k in range(0, 30000, 997):
        assert np.all(W[k, ln[k]:] == 0.0)
    sums = W.sum(axis=1)
    assert np.abs(sums).max() < 1e-5  # mean-centred (fp32 rounding only)
    # centred N(0,1) samples of size l have variance (l-1)/l per entry
    for v in (7, 9, 11):
        sel = W[ln == v][:, :v]
        var = sel.var()
        assert abs(var - (v - 1) / v) < 0.03, (v, var)
        kurt = ((sel / math.sqrt(var)) ** 4).mean()
        assert abs(kurt - 3.0) < 0.15, (v, kurt)


def test_bias_uniform(big):
    b = big["bias"].astype(np.float64)
    assert b.min() >= -1.0 and b.max() < 1.0
    assert abs(b.mean()) < 0.02
    assert abs(b.var() - 1.0 / 3.0) < 0.01
    hist, _ = np.histogram(b, bins=10, range=(-1, 1))
    assert ((hist - 3000) ** 2 / 3000).sum() < 27.9  # 9 dof, p = 0.001


def test_dilation_distribution(big):
    L = 1000
    for v in (7, 9, 11):
        d = big["dilation"][big["length"] == v].astype(np.float64)
        A = math.log2((L - 1) / (v - 1))
        assert d.min() >= 1 and d.max() <= (L - 1) // (v - 1)
        assert np.all(d == np.floor(d))
        # P(d >= m) = P(2^x >= m) = 1 - log2(m)/A for integer 1 <= m <= 2^A
        for m in (1, 2, 3, 5, 10, 40, 100):
            if m > 2 ** A:
                continue
            p = 1.0 - math.log2(m) / A
            emp = (d >= m).mean()
            sd = math.sqrt(max(p * (1 - p), 1e-12) / d.size)
            assert abs(emp - p) < 5 * sd + 1e-12, (v, m, emp, p)


def test_padding_rule(big):
    ln, d, p = big["length"], big["dilation"], big["padding"]
    padded = p != 0
    np.testing.assert_array_equal(p[padded], (ln[padded] - 1) * d[padded] // 2)
    frac = padded.mean()
    assert abs(frac - 0.5) < 5 * math.sqrt(0.25 / ln.size)
    O = 1000 + 2 * p - (ln - 1) * d
    assert O.min() >= 1
    np.testing.assert_array_equal(O[padded], 1000)


def test_small_input_length(oracle):
    k = oracle.generate_kernels(5, 200, 11)
    assert np.all(k["dilation"] == 1)
    with pytest.raises(ValueError):
        oracle.generate_kernels(5, 10, 10)
