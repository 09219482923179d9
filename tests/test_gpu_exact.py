"""GPU parity where every dot product is exact in fp32.

With integer-valued series, weights and biases, every partial sum of a dot
product is a small integer (or a small multiple of 0.5), so any summation
order, with or without fused multiply-add, gives the exact value: the HIP
path must then equal the fp64 oracle exactly, feature by feature.  Many of
these dot products are exactly +0 or -0, and neither is positive (PPV counts
strictly positive values, Sec. 2.1), so these tests reach the positivity
test of every code path at y = +-0:
  * the ballot compares of the position-tiled MFMA blocks (padded and
    clamped row layouts, 4- and 8-kernel items) and of the VALU items;
  * the series-lane layout's sign-bit indicator, forced and by call size;
  * the direct kernel;
  * the MPV guard (a count of 0 gives MPV 0);
  * multichannel items;
  * MINIROCKET's C > b compare at equality (biases equal to exact dot
    products).
Biases of -0.0 and series of +-0 make y = -0 as well as +0.  Denormal
biases on a zero series sit inside the oracle's certified near-zero band
(either sign of count is correct there), and are checked against it."""
import sys

import numpy as np
import pytest

from _util import assert_mpv_parity, assert_parity, kernel_set

pytestmark = pytest.mark.gpu


def _log(msg):
    print("[gpu-exact] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def _int_bias(rng, size):
    b = rng.integers(-2, 3, size).astype(np.float32)
    # half of the zero biases are -0.0
    neg0 = (b == 0) & (rng.random(size) < 0.5)
    b[neg0] = np.float32(-0.0)
    return b


def _int_kernels(rng, L, buckets):
    """Hand-built kernels with integer weights in [-2, 2] and integer biases
    in [-2, 2] (zeros of both signs); buckets are (length, dilation, padded,
    size) and produce every item kind: 4- and 8-kernel MFMA items, the one or
    two leftover kernels (VALU items for series longer than 128), and shorter
    centred kernels moved into longer frames."""
    lengths, dil, pad, weights = [], [], [], []
    for ln, d, padded, size in buckets:
        d = min(d, (L - 1) // max(1, ln - 1)) if ln > 1 else d
        for _ in range(size):
            lengths.append(ln)
            dil.append(d)
            pad.append((ln - 1) * d // 2 if padded else 0)
            weights.append(rng.integers(-2, 3, ln).astype(np.float32))
    return kernel_set(lengths, dil, pad, _int_bias(rng, len(lengths)), weights)


BUCKETS = [(7, 1, 1, 8), (7, 3, 0, 5), (9, 1, 0, 9), (9, 2, 1, 4), (9, 7, 1, 1), (11, 1, 1, 12),
           (11, 5, 0, 2), (11, 29, 1, 3), (11, 29, 0, 1), (3, 4, 1, 2), (5, 9, 0, 6), (7, 40, 1, 2),
           (9, 37, 0, 1), (1, 1, 0, 3), (2, 6, 0, 2), (11, 2, 1, 1), (7, 2, 1, 3)]


def _int_series(rng, n, L):
    """Integer series in [-3, 3], plus a zero row, a -0 row and a constant
    1.5 row (all products and partial sums stay exact in fp32)."""
    X = rng.integers(-3, 4, (n, L)).astype(np.float32)
    X[1] = 0.0
    X[2] = np.float32(-0.0)
    X[3] = 1.5
    return X


def _assert_exact(F, ref, K, nf, what):
    """Every feature equal to the oracle's exact result."""
    F = np.asarray(F, dtype=np.float64)
    O = ref["O"][None, :].astype(np.float64)
    cnt = np.rint(F[:, 0::nf] * O).astype(np.int64)
    np.testing.assert_array_equal(cnt, ref["cnt"], err_msg=what + ": counts")
    np.testing.assert_array_equal(F[:, 1::nf], ref["F"][:, 1::2], err_msg=what + ": MAX")
    # PPV is (float)count / (float)O
    np.testing.assert_array_equal(F[:, 0::nf].astype(np.float32),
                                  (ref["cnt"].astype(np.float32) / ref["O"][None, :].astype(np.float32)),
                                  err_msg=what + ": PPV")
    if nf == 3:
        # the positive sum is an exact integer; one fp32 division by the count
        np.testing.assert_array_equal(F[:, 2::3].astype(np.float32), ref["mpv"].astype(np.float32),
                                      err_msg=what + ": MPV")


def _plan(rk, ks, L, mode, mpv):
    return rk.Plan(ks, L, direct=mode == "direct", clamped=mode == "clamped", tiled=mode == "tiled",
                   series=mode == "series", mpv=mpv)


def _transform(env, plan, X_np):
    torch, _ = env
    X = torch.from_numpy(np.ascontiguousarray(X_np)).cuda()
    F = plan.transform(X)
    torch.cuda.synchronize()
    return F.cpu().numpy()


@pytest.mark.parametrize("mpv", [False, True])
@pytest.mark.parametrize("mode,L", [("fused", 300), ("clamped", 300), ("direct", 300), ("fused", 100),
                                    ("tiled", 100), ("series", 100), ("direct", 100)])
def test_integer_series_exact(env, oracle, mode, L, mpv):
    torch, rk = env
    rng = np.random.default_rng(1000 + L)
    ks = _int_kernels(rng, L, BUCKETS)
    K = ks["length"].shape[0]
    X = _int_series(rng, 9, L)
    plan = _plan(rk, ks, L, mode, mpv)
    info = plan.info()
    assert info["direct"] == (mode == "direct") and info["clamped"] == (mode == "clamped")
    assert info["series_lane"] == (L <= 128 and mode in ("fused", "series"))
    if mode != "direct" and L > 128:
        # every VALU item variant beside the MFMA items
        t = rk.plan_tables(ks, L)
        assert (t["items"][:, 0] >= 6).any() and (t["items"][:, 0] < 6).any()
    _log("integer series mode=%s L=%d K=%d mpv=%s" % (mode, L, K, mpv))
    F = _transform(env, plan, X)
    ref = oracle.transform(X, ks)
    nf = 3 if mpv else 2
    zeros = int((ref["cnt"] < ref["O"][None, :]).sum())
    _assert_exact(F, ref, K, nf, "%s L=%d" % (mode, L))
    # the zero, -0 and constant rows: on the zero rows every dot product is
    # the bias, so PPV = [b > 0] with b = +-0 giving 0
    b = ks["bias"]
    for r in (1, 2):
        np.testing.assert_array_equal(F[r, 1::nf], b)
        np.testing.assert_array_equal(F[r, 0::nf], (b > 0).astype(np.float32))
    _log("  exact, %d features with some non-positive output" % zeros)


# unpadded buckets of one and two kernels at large dilations, and padded
# ones of one length per dilation (centred kernels of several lengths at one
# dilation would share longer frames instead)
TOEP_CASES = {
    # super-tiles of 1 to 4 chunks (several per block in the padded layout)
    4000: ([(ln, d, 0, 1 + i % 2) for ln in (7, 9, 11) for i, d in enumerate((60, 64, 65, 100, 129, 190, 200))]
           + [(11, 70, 1, 1), (9, 90, 1, 2), (7, 140, 1, 1), (11, 110, 1, 2), (9, 1, 1, 16), (7, 1, 0, 8)]),
    # super-tiles of 9 to 24 chunks (blocks of nearly equal size)
    16384: [(11, 600, 1, 1), (11, 560, 1, 2), (9, 700, 0, 1), (9, 1000, 1, 2), (7, 900, 0, 2), (11, 1500, 1, 1),
            (9, 1, 1, 16)],
}


@pytest.mark.parametrize("mpv", [False, True])
@pytest.mark.parametrize("mode", ["fused", "clamped"])
@pytest.mark.parametrize("L", sorted(TOEP_CASES))
def test_integer_toeplitz_exact(env, oracle, L, mode, mpv):
    """Toeplitz items (a bucket's one or two kernels at a large dilation, the
    kernel at 4 or 2 tap shifts in one MFMA group), beside MFMA items of
    8 kernels at dilation 1, on integer data: every feature exact, including
    the zero and -0 rows.  Super-tiles of 1 to 10 chunks: in the padded
    layout those of up to 4 chunks run several to a block, longer ones in
    blocks of nearly equal size; the Toeplitz kernel runs on the plan's own
    stream beside the fused kernel."""
    torch, rk = env
    rng = np.random.default_rng(4242 + L)
    ks = _int_kernels(rng, L, TOEP_CASES[L])
    v = rk.plan_tables(ks, L)["items"][:, 0]
    assert ((v >= 12) & (v % 2 == 0)).any() and ((v >= 12) & (v % 2 == 1)).any() and (v < 6).any()
    plan = _plan(rk, ks, L, mode, mpv)
    assert plan.info()["toeplitz_items"] == int((v >= 12).sum())
    assert plan.info()["clamped"] == (mode == "clamped")
    X = _int_series(rng, 7, L)
    _log("integer Toeplitz items L=%d mode=%s mpv=%s, %d kernels" % (L, mode, mpv, ks["length"].shape[0]))
    F = _transform(env, plan, X)
    nf = 3 if mpv else 2
    _assert_exact(F, oracle.transform(X, ks), ks["length"].shape[0], nf, "toeplitz " + mode)
    b = ks["bias"]
    for r in (1, 2):
        np.testing.assert_array_equal(F[r, 1::nf], b)
        np.testing.assert_array_equal(F[r, 0::nf], (b > 0).astype(np.float32))


@pytest.mark.parametrize("mpv", [False, True])
def test_integer_series_lane_by_call_size(env, oracle, mpv):
    """At least 4,096 short series: the default plan runs the series-lane
    layout (slot-ordered buffer and permutation) on its own."""
    torch, rk = env
    rng = np.random.default_rng(77)
    L = 64
    ks = _int_kernels(rng, L, BUCKETS)
    X = _int_series(rng, 4100, L)
    plan = rk.Plan(ks, L, mpv=mpv)
    assert plan.info()["series_lane"]
    _log("integer series, 4100 rows, L=64, mpv=%s" % mpv)
    F = _transform(env, plan, X)
    _assert_exact(F, oracle.transform(X, ks), ks["length"].shape[0], 3 if mpv else 2, "series by size")


ZERO_MODES = [("fused", 300), ("clamped", 300), ("direct", 300), ("tiled", 100), ("series", 100)]


@pytest.mark.parametrize("mpv", [False, True])
@pytest.mark.parametrize("mode,L", ZERO_MODES)
def test_all_outputs_signed_zero(env, mode, L, mpv):
    """Every dot product exactly +0 or -0: zero series (of either sign) with
    biases +0 and -0, and a constant 1.5 series under unpadded kernels whose
    integer weights sum to zero.  PPV and MPV must be exactly 0 and MAX a
    zero."""
    torch, rk = env
    rng = np.random.default_rng(5)
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in (2, 3, 7, 9, 11):
        for d in (1, 2, 5):
            for k in range(6):
                w = rng.integers(-3, 4, ln).astype(np.float32)
                w[-1] -= w.sum()  # integer weights summing to zero
                lengths.append(ln)
                dil.append(d)
                pad.append(0)
                bias.append(0.0 if k % 2 else -0.0)
                weights.append(w)
    ks = kernel_set(lengths, dil, pad, bias, weights)
    assert (np.signbit(ks["bias"])).any() and (~np.signbit(ks["bias"])).any()
    X = np.zeros((5, L), np.float32)
    X[1] = np.float32(-0.0)
    X[3] = 1.5
    X[4] = -1.5
    plan = _plan(rk, ks, L, mode, mpv)
    _log("all-zero outputs mode=%s L=%d mpv=%s" % (mode, L, mpv))
    F = _transform(env, plan, X)
    nf = 3 if mpv else 2
    assert np.all(F[:, 0::nf] == 0.0), "PPV of +-0 outputs must be 0"
    assert np.all(F[:, 1::nf] == 0.0), "MAX of +-0 outputs must be a zero"
    if mpv:
        assert np.all(F[:, 2::3] == 0.0), "MPV without positive outputs must be 0"


@pytest.mark.parametrize("mode,L", ZERO_MODES)
def test_denormal_biases(env, oracle, mode, L):
    """Zero series with biases +-1e-40 (denormal): every dot product is the
    bias.  The value sits inside the oracle's certified near-zero band, where
    either count is a correct fp32 result; MAX is the bias or a zero."""
    torch, rk = env
    rng = np.random.default_rng(6)
    tiny = np.float32(1e-40)
    assert 0 < tiny < np.finfo(np.float32).tiny
    n_k = 40
    ks = kernel_set([9] * n_k, [1 + (k % 4) for k in range(n_k)], [4 * (1 + k % 4) if k % 3 else 0 for k in range(n_k)],
                    [tiny if k % 2 else -tiny for k in range(n_k)],
                    [rng.integers(-2, 3, 9).astype(np.float32) for _ in range(n_k)])
    X = np.zeros((3, L), np.float32)
    plan = _plan(rk, ks, L, mode, False)
    F = _transform(env, plan, X)
    ref = oracle.transform(X, ks)
    cnt = np.rint(F[:, 0::2].astype(np.float64) * ref["O"][None, :]).astype(np.int64)
    assert np.all((cnt >= ref["cnt_lo"]) & (cnt <= ref["cnt_hi"]))
    mx = F[:, 1::2]
    assert np.all((mx == ks["bias"][None, :]) | (mx == 0.0))
    assert np.all(np.abs(mx.astype(np.float64) - ref["F"][:, 1::2]) <= ref["beta"])
    kept = bool(np.all(mx == ks["bias"][None, :]))
    _log("denormal biases mode=%s L=%d: %s" % (mode, L, "kept" if kept else "flushed"))


@pytest.mark.parametrize("mode", ["fused", "clamped", "direct"])
def test_multichannel_integer_exact(env, oracle, mode):
    """Multichannel kernels (Sec. 3.3) with integer weights on integer
    series: the channel loops of the fused kernel and of the direct kernel
    give exactly the oracle's features."""
    torch, rk = env
    rng = np.random.default_rng(12)
    C, L = 3, 150
    sets = [[0], [2], [0, 1], [1, 2], [0, 1, 2]]
    lengths, dil, pad, bias, count, index, weights = [], [], [], [], [], [], []
    for ln, d, padded in ((7, 1, 1), (9, 3, 0), (11, 2, 1), (9, 1, 1), (7, 13, 0)):
        for rep in range(3):
            for chans in sets:
                lengths.append(ln)
                dil.append(d)
                pad.append((ln - 1) * d // 2 if padded else 0)
                count.append(len(chans))
                idx = np.full(C, -1, np.int32)
                idx[:len(chans)] = chans
                index.append(idx)
                w = np.zeros((C, 11), np.float32)
                w[:len(chans), :ln] = rng.integers(-2, 3, (len(chans), ln))
                weights.append(w)
    bias = _int_bias(rng, len(lengths))
    ks = dict(length=np.array(lengths, np.int32), dilation=np.array(dil, np.int32),
              padding=np.array(pad, np.int32), bias=bias, weights=np.array(weights, np.float32),
              n_channels=C, channel_count=np.array(count, np.int32), channel_index=np.array(index, np.int32))
    X = rng.integers(-3, 4, (6, C, L)).astype(np.float32)
    X[1] = 0.0
    plan = rk.Plan(ks, L, direct=mode == "direct", clamped=mode == "clamped")
    _log("multichannel integer mode=%s, %d kernels" % (mode, len(lengths)))
    F = _transform(env, plan, X)
    _assert_exact(F, oracle.transform(X, ks), len(lengths), 2, "mc " + mode)


@pytest.mark.parametrize("clamped", [False, True])
def test_minirocket_bias_equal_to_dot_product(env, clamped):
    """MINIROCKET counts C_t > b strictly.  On integer series the dot
    products C_t (weights 2 and -1) are exact integers; biases drawn from the
    same integers (and +-0) equal many of them, and the counts must equal
    the oracle's exactly."""
    torch, rk = env
    from oracle import minirocket_oracle
    rng = np.random.default_rng(21)
    L = 70
    dil = np.array([1, 2, 4, 8], np.int32)
    feats = np.array([2, 1, 3, 1], np.int32)
    nf = 84 * int(feats.sum())
    biases = rng.integers(-8, 9, nf).astype(np.float32)
    biases[(biases == 0) & (rng.random(nf) < 0.5)] = np.float32(-0.0)
    params = dict(input_length=L, dilations=dil, features_per_dilation=feats, biases=biases)
    X = rng.integers(-2, 3, (6, L)).astype(np.float32)
    X[2] = 0.0
    X[4] = 1.0
    plan = rk.MiniRocketPlan(params, clamped=clamped)
    _log("MINIROCKET integer series, %d features, clamped=%s" % (nf, clamped))
    F = _transform(env, plan, X).astype(np.float64)
    ref = minirocket_oracle.transform(X, params)
    cnt = np.rint(F * ref["O"][None, :]).astype(np.int64)
    np.testing.assert_array_equal(cnt, ref["cnt"])
    # equality cases were reached: some bias equals a dot product
    W = minirocket_oracle.kernel_weights()
    lay = minirocket_oracle.feature_layout(params)
    hits = 0
    for f in range(0, nf, 7):
        d = int(dil[lay["dilation_index"][f]])
        k = int(lay["kernel"][f])
        p = 4 * d if lay["padded"][f] else 0
        xz = np.zeros((X.shape[0], L + 2 * p), np.float64)
        xz[:, p:p + L] = X
        O = int(lay["O"][f])
        Cv = sum(W[k, j] * xz[:, j * d:j * d + O] for j in range(9))
        hits += int((Cv == biases[f]).sum())
    assert hits > 0
    _log("  exact; %d sampled (row, output) pairs sit exactly on their bias" % hits)
