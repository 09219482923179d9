"""GPU checks of the series-lane layout (short univariate series, L <= 128):
the 64 lanes of a wavefront take 64 series and each lane reduces its own
series.  Its results equal the position-tiled layout's (same MFMA
accumulation order, the same zero-padded reads) and meet the oracle's
parity rule, for ragged series counts (not a multiple of 64), outputs that
are not a multiple of the block size, one-output kernels, hand-built
lengths and MPV."""
import sys

import numpy as np
import pytest

from _util import assert_mpv_parity, assert_parity, kernel_set

pytestmark = pytest.mark.gpu


def _log(msg):
    print("[gpu-series] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def _series(n, L, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, L)).cumsum(axis=1)
    return ((X - X.mean(1, keepdims=True)) / X.std(1, keepdims=True)).astype(np.float32)


def _run(env, ks, X_np, **flags):
    torch, rk = env
    X = torch.from_numpy(np.ascontiguousarray(X_np)).cuda()
    plan = rk.Plan(ks, X_np.shape[1], **flags)
    F = plan.transform(X)
    torch.cuda.synchronize()
    return F.cpu().numpy(), plan.info()


@pytest.mark.parametrize("n,L,K,seed", [
    (1, 12, 300, 1), (63, 16, 500, 2), (64, 33, 800, 3), (65, 64, 1000, 4),
    (130, 100, 700, 5), (200, 128, 600, 6),
])
def test_series_lane_matches_tiled_and_oracle(env, oracle, n, L, K, seed):
    torch, rk = env
    ks = rk.generate_kernels(seed, K, L)
    X = _series(n, L, seed)
    _log("n=%d L=%d K=%d" % (n, L, K))
    Fs, info = _run(env, ks, X, series=True)
    assert info["series_lane"] and info["rows_per_block"] == 64
    Ft, info_t = _run(env, ks, X, tiled=True)
    assert not info_t["series_lane"]
    # same accumulation order and zero-padded reads: equal results (+0 and
    # -0 compare equal)
    assert np.array_equal(Fs, Ft)
    assert_parity(Fs, oracle.transform(X, ks), "series L=%d" % L)


def test_series_lane_limits(env):
    torch, rk = env
    for L, want in ((128, True), (129, False)):
        ks = rk.generate_kernels(7, 50, L)
        assert rk.Plan(ks, L).info()["series_lane"] == want, L
    ks = rk.generate_kernels(7, 50, 129)
    with pytest.raises(rk.RocketError):
        rk.Plan(ks, 129, series=True)
    # multichannel sets keep the position-tiled layout
    ks = rk.generate_kernels_multi(7, 50, 64, 3)
    assert not rk.Plan(ks, 64).info()["series_lane"]
    with pytest.raises(rk.RocketError):
        rk.Plan(ks, 64, series=True)


def test_small_calls_use_tiles(env):
    """Below 4,096 series a default plan runs the position-tiled layout (too
    few workgroups for the series-lane one); the results are the same."""
    torch, rk = env
    L = 64
    ks = rk.generate_kernels(8, 300, L)
    X = _series(100, L, 8)
    Fd, info = _run(env, ks, X)
    assert info["series_lane"]
    Fs, _ = _run(env, ks, X, series=True)
    Ft, _ = _run(env, ks, X, tiled=True)
    assert np.array_equal(Fd, Ft) and np.array_equal(Fs, Ft)


def test_series_lane_hand_built(env, oracle):
    """Every length 1..11 at the largest dilation (one output when
    unpadded), padded and not, and a few small dilations."""
    rng = np.random.default_rng(9)
    L = 40
    lengths, dil, pad, ws = [], [], [], []
    for ln in range(1, 12):
        dmax = (L - 1) // max(1, ln - 1) if ln > 1 else 7
        for d in sorted({1, 2, dmax}):
            for padded in (0, 1):
                lengths.append(ln)
                dil.append(d)
                pad.append((ln - 1) * d // 2 if padded else 0)
                ws.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, rng.uniform(-1, 1, len(lengths)), ws)
    X = _series(70, L, 9)
    Fs, info = _run(env, ks, X, series=True)
    assert info["series_lane"]
    Ft, _ = _run(env, ks, X, tiled=True)
    assert np.array_equal(Fs, Ft)
    assert_parity(Fs, oracle.transform(X, ks), "series hand-built")


@pytest.mark.parametrize("seed", range(8))
def test_series_lane_random_sets(env, oracle, seed):
    """Generated kernel sets at random sizes (L from 11 to 128, K from 100 to
    1,200, 1 to 300 series, MPV on or off): the series-lane layout's PPV and
    MAX equal the tiled layout's, and every feature meets the oracle.  (MPV
    sums the positive values in a different order in the two layouts: one
    lane per series there, a wavefront tree here.)"""
    rng = np.random.default_rng(7000 + seed)
    L = int(rng.integers(11, 129))
    K = int(rng.integers(100, 1201))
    n = int(rng.integers(1, 301))
    mpv = bool(rng.integers(0, 2))
    torch, rk = env
    ks = rk.generate_kernels(7100 + seed, K, L)
    X = _series(n, L, 7200 + seed)
    _log("random set seed=%d n=%d L=%d K=%d mpv=%s" % (seed, n, L, K, mpv))
    Fs, info = _run(env, ks, X, series=True, mpv=mpv)
    assert info["series_lane"]
    Ft, info_t = _run(env, ks, X, tiled=True, mpv=mpv)
    assert not info_t["series_lane"]
    nf = 3 if mpv else 2
    for f in (0, 1):
        assert np.array_equal(Fs[:, f::nf], Ft[:, f::nf]), f
    ref = oracle.transform(X, ks)
    if mpv:
        assert_mpv_parity(Fs, ref, "series random mpv L=%d K=%d" % (L, K))
    else:
        assert_parity(Fs, ref, "series random L=%d K=%d" % (L, K))


@pytest.mark.parametrize("L", [24, 128])
def test_series_lane_mpv(env, oracle, L):
    torch, rk = env
    ks = rk.generate_kernels(11, 600, L)
    X = _series(90, L, 11)
    F, info = _run(env, ks, X, mpv=True, series=True)
    assert info["series_lane"]
    assert_mpv_parity(F, oracle.transform(X, ks), "series mpv L=%d" % L)


def test_series_lane_host_to_host(env):
    torch, rk = env
    L = 64
    ks = rk.generate_kernels(12, 400, L)
    X = _series(150, L, 12)
    Fd, _ = _run(env, ks, X, series=True)
    p = rk.Plan(ks, L, series=True)
    Xh = torch.from_numpy(X).pin_memory()
    Fh = torch.empty((150, 800), dtype=torch.float32).pin_memory()
    p.transform_host(Xh, Fh, batch_rows=40)
    assert np.array_equal(Fh.numpy(), Fd)


def test_series_lane_chunks(env):
    """More series than one chunk of the slot-ordered buffer (8,192 rows):
    equal to the position-tiled layout on every row."""
    torch, rk = env
    L, K = 20, 64
    ks = rk.generate_kernels(13, K, L)
    X = _series(8192 + 300, L, 13)
    _log("chunks n=%d" % X.shape[0])
    Fs, info = _run(env, ks, X)  # above the default threshold: series-lane
    assert info["series_lane"]
    Ft, _ = _run(env, ks, X, tiled=True)
    assert np.array_equal(Fs, Ft)


@pytest.mark.parametrize("mpv", [False, True])
def test_series_lane_chunks_many_tiles(env, oracle, mpv):
    """Two chunks whose permutations hold more 64 x 64 tiles (700 kernels,
    not a multiple of 64, x 8,192 series) than the permutation has
    workgroups, so each workgroup strides over several tiles: PPV and MAX
    equal the position-tiled layout's on every row, MPV meets the oracle's
    parity rule on rows around the chunk boundary and the ends."""
    torch, rk = env
    L, K = 20, 700
    ks = rk.generate_kernels(16, K, L)
    X = _series(8192 + 300, L, 16)
    _log("chunks many tiles n=%d K=%d mpv=%s" % (X.shape[0], K, mpv))
    Fs, info = _run(env, ks, X, mpv=mpv, series=True)
    assert info["series_lane"]
    Ft, _ = _run(env, ks, X, mpv=mpv, tiled=True)
    nf = 3 if mpv else 2
    a = Fs.reshape(len(X), K, nf)
    b = Ft.reshape(len(X), K, nf)
    assert np.array_equal(a[:, :, :2], b[:, :, :2])
    if mpv:
        rows = np.r_[0:64, 8128:8256, len(X) - 64:len(X)]
        assert_mpv_parity(Fs[rows], oracle.transform(X[rows], ks), "series mpv chunks")


def test_series_lane_two_streams(env):
    """Transforms of one plan on two streams at once take turns on the
    plan's slot-ordered buffer: each result equals its one-stream result."""
    torch, rk = env
    L = 48
    ks = rk.generate_kernels(14, 500, L)
    plan = rk.Plan(ks, L, series=True)
    Xa = torch.from_numpy(_series(3000, L, 14)).cuda()
    Xb = torch.from_numpy(_series(5000, L, 15)).cuda()
    want_a = plan.transform(Xa)
    want_b = plan.transform(Xb)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    Fa = torch.empty_like(want_a)
    Fb = torch.empty_like(want_b)
    for _ in range(3):
        Fa.zero_()
        Fb.zero_()
        torch.cuda.synchronize()
        plan.transform_into(Xa, Fa, sa)
        plan.transform_into(Xb, Fb, sb)
        torch.cuda.synchronize()
        assert torch.equal(Fa, want_a) and torch.equal(Fb, want_b)
