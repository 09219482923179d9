"""Oracle pins for multivariate series (Sec. 3.3): every kernel reads its
own subset of channels, one weight row per channel, and its dot product sums
over those channels and taps.  Pinned to a literal Python loop, to torch's
multi-channel conv1d in fp64, to exact channel-relabelling invariance, to the
univariate transform where only one channel is non-zero, and to the
generator's distributions."""
import math

import numpy as np
import pytest

from _util import z_norm


def brute_force_mc(X, ks):
    """PPV, MAX, MPV of every (row, kernel) with plain Python floats."""
    n, C, L = X.shape
    K = len(ks["length"])
    F = np.zeros((n, 2 * K))
    M = np.zeros((n, K))
    for i in range(n):
        for k in range(K):
            ln, d, p = int(ks["length"][k]), int(ks["dilation"][k]), int(ks["padding"][k])
            b = float(ks["bias"][k])
            chans = [int(c) for c in ks["channel_index"][k][:int(ks["channel_count"][k])]]
            ys = []
            for t in range(L + 2 * p - (ln - 1) * d):
                acc = b
                for s, c in enumerate(chans):
                    for j in range(ln):
                        m = t - p + j * d
                        if 0 <= m < L:
                            acc += float(ks["weights"][k][s][j]) * float(X[i, c, m])
                ys.append(acc)
            pos = [y for y in ys if y > 0]
            F[i, 2 * k] = len(pos) / len(ys)
            F[i, 2 * k + 1] = max(ys)
            M[i, k] = sum(pos) / len(pos) if pos else 0.0
    return F, M


def test_brute_force_small(oracle):
    rng = np.random.default_rng(1)
    ks = oracle.generate_kernels_multi(3, 40, 24, 4)
    X = rng.standard_normal((2, 4, 24)).astype(np.float32)
    r = oracle.transform(X, ks)
    F, M = brute_force_mc(X, ks)
    np.testing.assert_array_equal(r["F"][:, 0::2], F[:, 0::2])
    np.testing.assert_allclose(r["F"][:, 1::2], F[:, 1::2], rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["mpv"], M, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(2))
def test_torch_conv1d_multichannel_fp64(oracle, seed):
    """The dot products are torch's conv1d over all C input channels in fp64,
    with zero weights on the channels a kernel does not read."""
    import torch
    rng = np.random.default_rng(20 + seed)
    C, L = 5, 90
    ks = oracle.generate_kernels_multi(40 + seed, 60, L, C)
    X = rng.standard_normal((3, C, L)).astype(np.float32)
    r = oracle.transform(X, ks)
    for k in range(len(ks["length"])):
        ln, d, p = int(ks["length"][k]), int(ks["dilation"][k]), int(ks["padding"][k])
        W = np.zeros((1, C, ln))
        for s in range(int(ks["channel_count"][k])):
            W[0, ks["channel_index"][k][s]] = ks["weights"][k][s][:ln]
        y = torch.nn.functional.conv1d(torch.from_numpy(X.astype(np.float64)), torch.from_numpy(W),
                                       torch.tensor([float(ks["bias"][k])], dtype=torch.float64),
                                       padding=p, dilation=d).numpy()[:, 0]
        assert y.shape[1] == r["O"][k]
        np.testing.assert_array_equal((y > 0).sum(axis=1), r["cnt"][:, k])
        np.testing.assert_allclose(y.max(axis=1), r["F"][:, 2 * k + 1], rtol=0, atol=1e-12)


def test_channel_relabelling(oracle):
    """Permuting the series' channels and relabelling every kernel's channel
    ids the same way leaves all features bit-identical."""
    rng = np.random.default_rng(3)
    C, L = 6, 120
    ks = oracle.generate_kernels_multi(9, 150, L, C)
    X = z_norm(rng.standard_normal((4 * C, L))).reshape(4, C, L)
    perm = rng.permutation(C)             # new channel q holds old channel perm[q]
    inv = np.argsort(perm)
    Xp = np.ascontiguousarray(X[:, perm, :])
    kp = dict(ks)
    idx = ks["channel_index"].copy()
    W = ks["weights"].copy()
    for k in range(idx.shape[0]):
        c = int(ks["channel_count"][k])
        new = inv[idx[k, :c]]
        order = np.argsort(new)           # keep channel ids ascending
        idx[k, :c] = new[order]
        W[k, :c] = ks["weights"][k, :c][order]
    kp["channel_index"], kp["weights"] = idx, W
    a, b = oracle.transform(X, ks), oracle.transform(Xp, kp)
    np.testing.assert_array_equal(a["cnt"], b["cnt"])
    np.testing.assert_allclose(a["F"], b["F"], rtol=0, atol=1e-12)


def test_single_live_channel_is_univariate(oracle):
    """With every channel zero except c, a kernel that reads c behaves as the
    univariate kernel made of its channel-c weight row; one that does not
    read c sees only its bias."""
    rng = np.random.default_rng(4)
    C, L, c = 4, 80, 2
    ks = oracle.generate_kernels_multi(11, 120, L, C)
    X = np.zeros((2, C, L), np.float32)
    X[:, c] = rng.standard_normal((2, L)).astype(np.float32)
    r = oracle.transform(X, ks)
    K = len(ks["length"])
    w1 = np.zeros((K, 11), np.float32)
    reads = np.zeros(K, bool)
    for k in range(K):
        hit = np.where(ks["channel_index"][k][:ks["channel_count"][k]] == c)[0]
        if hit.size:
            reads[k] = True
            w1[k] = ks["weights"][k][hit[0]]
    uni = dict(length=ks["length"], dilation=ks["dilation"], padding=ks["padding"], bias=ks["bias"],
               weights=w1)
    u = oracle.transform(np.ascontiguousarray(X[:, c]), uni)
    np.testing.assert_array_equal(r["F"][:, 0::2][:, reads], u["F"][:, 0::2][:, reads])
    np.testing.assert_array_equal(r["F"][:, 1::2][:, reads], u["F"][:, 1::2][:, reads])
    b = ks["bias"].astype(np.float64)
    np.testing.assert_array_equal(r["F"][:, 1::2][:, ~reads], np.broadcast_to(b[~reads], (2, (~reads).sum())))


def test_generator_channels():
    from oracle import rocket_oracle as o
    C = 7
    ks = o.generate_kernels_multi(123, 6000, 400, C)
    cc, idx, W = ks["channel_count"], ks["channel_index"], ks["weights"]
    assert cc.min() >= 1 and cc.max() <= C
    for k in range(0, 6000, 7):
        c = cc[k]
        ids = idx[k, :c]
        assert np.all(np.diff(ids) > 0) and ids.min() >= 0 and ids.max() < C
        assert np.all(idx[k, c:] == -1)
        assert np.all(W[k, c:] == 0)
        ln = ks["length"][k]
        assert np.all(np.abs(W[k, :c, :ln].astype(np.float64).sum(axis=1)) < 1e-5)
        assert np.all(W[k, :, ln:] == 0)
    # P(count = m) = log2((m+1)/m) / log2(C+1)
    want = np.array([math.log2((m + 1) / m) / math.log2(C + 1) for m in range(1, C + 1)])
    got = np.bincount(cc, minlength=C + 1)[1:] / cc.shape[0]
    assert np.abs(got - want).max() < 0.02
    # every channel is picked equally often
    per = np.bincount(idx[idx >= 0], minlength=C) / cc.sum()
    assert np.abs(per - 1.0 / C).max() < 0.01
    # reproducible, prefix-stable
    again = o.generate_kernels_multi(123, 50, 400, C)
    for key in ("length", "dilation", "padding", "bias", "channel_count"):
        np.testing.assert_array_equal(again[key], ks[key][:50])
    np.testing.assert_array_equal(again["weights"], W[:50])
