"""GPU parity of the MINIROCKET path (the ROCKET variant Sec. 5 names): the
library's fit equals the oracle's fit bitwise, and the HIP transform through
the C ABI matches the fp64 oracle transform on the same parameters and
series: every positive count within 2 of the oracle's and inside its
certified fp32 range."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _log(msg):
    print("[gpu-minirocket] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


@pytest.fixture(scope="module")
def rk():
    import paper_2601_17091_amd as rk
    rk.library()
    return rk


@pytest.fixture(scope="module")
def mo(oracle):
    from oracle import minirocket_oracle
    return minirocket_oracle


def _fit(rk, mo, X_train, nf, seed):
    p = rk.minirocket_fit(X_train, nf, seed)
    q = mo.fit(X_train, nf, seed)
    for key in ("dilations", "features_per_dilation", "biases"):
        assert np.array_equal(p[key], q[key]), key
    return p


def _check(F_gpu, ref, what):
    F_gpu = np.asarray(F_gpu, dtype=np.float64)
    O = ref["O"][None, :].astype(np.float64)
    cnt = np.rint(F_gpu * O).astype(np.int64)
    assert np.all(np.isfinite(F_gpu)) and np.all((F_gpu >= 0) & (F_gpu <= 1)), what
    assert np.all(np.abs(F_gpu * O - cnt) < 1e-3), what
    # PPV is the correctly rounded count / O
    np.testing.assert_array_equal(F_gpu.astype(np.float32), (cnt / O).astype(np.float32), err_msg=what)
    d = np.abs(cnt - ref["cnt"])
    assert d.max() <= 2, (what, int(d.max()))
    outside = (cnt < ref["cnt_lo"]) | (cnt > ref["cnt_hi"])
    assert not outside.any(), (what, int(outside.sum()))
    return int(d.max())


def _run(rk, torch, params, X_np, clamped=False):
    plan = rk.MiniRocketPlan(params, clamped=clamped)
    info = plan.info()
    assert info["minirocket"] and info["clamped"] == clamped
    assert info["n_features"] == params["biases"].shape[0]
    X = torch.from_numpy(np.ascontiguousarray(X_np, dtype=np.float32)).cuda()
    F = plan.transform(X)
    torch.cuda.synchronize()
    return F.cpu().numpy(), plan


@pytest.mark.parametrize("n,L,nf,seed", [
    (6, 9, 10000, 1),      # shortest series: one dilation, 119 biases per kernel
    (8, 17, 10000, 2),     # two dilations, 116 and 3 biases
    (16, 64, 10000, 3),    # short series: up to 41 biases per kernel
    (12, 130, 2000, 4),    # ragged last tile, several dilations
    (10, 500, 10000, 5),
    (4, 1000, 10000, 6),
])
@pytest.mark.parametrize("clamped", [False, True])
def test_minirocket_parity(torch_gpu, rk, mo, n, L, nf, seed, clamped):
    _log("n=%d L=%d features=%d seed=%d clamped=%s" % (n, L, nf, seed, clamped))
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, L)).cumsum(axis=1)
    X = ((X - X.mean(1, keepdims=True)) / X.std(1, keepdims=True)).astype(np.float32)
    params = _fit(rk, mo, X, nf, seed)
    F, _ = _run(rk, torch_gpu, params, X, clamped)
    ref = mo.transform(X, params)
    _check(F, ref, "L=%d" % L)


def test_minirocket_clamped_equals_padded(torch_gpu, rk, mo):
    rng = np.random.default_rng(11)
    X = rng.standard_normal((20, 300)).astype(np.float32)
    params = _fit(rk, mo, X, 10000, 7)
    Fa, _ = _run(rk, torch_gpu, params, X, False)
    Fb, _ = _run(rk, torch_gpu, params, X, True)
    np.testing.assert_array_equal(Fa, Fb)


def test_minirocket_constant_series(torch_gpu, rk, mo):
    """Constant series: unpadded pairs see c * sum(w) = 0 exactly (the
    products are exact and the sum cancels), so their features are [b < 0]."""
    rng = np.random.default_rng(12)
    X = rng.standard_normal((10, 200)).astype(np.float32)
    params = _fit(rk, mo, X, 5000, 8)
    F, _ = _run(rk, torch_gpu, params, np.full((2, 200), 0.5, np.float32), False)
    lay = mo.feature_layout(params)
    un = ~lay["padded"]
    np.testing.assert_array_equal(F[:, un], np.broadcast_to((params["biases"][un] < 0).astype(np.float32),
                                                            (2, int(un.sum()))))


def test_minirocket_host_to_host(torch_gpu, rk, mo):
    rng = np.random.default_rng(13)
    X = rng.standard_normal((37, 250)).astype(np.float32)
    params = _fit(rk, mo, X[:10], 3000, 9)
    Fd, plan = _run(rk, torch_gpu, params, X, False)
    Xh = torch_gpu.from_numpy(X).pin_memory()
    Fh = torch_gpu.empty((37, plan.n_features), dtype=torch_gpu.float32).pin_memory()
    plan.transform_host(Xh, Fh, batch_rows=8)
    np.testing.assert_array_equal(Fh.numpy(), Fd)


def test_minirocket_workload_sampled(torch_gpu, rk, mo):
    """The benchmark's MINIROCKET workload (Manufacturing-shaped AR(1) series,
    10,000 features fitted on the first 1,000 series) on the full launch,
    checked on a row sample."""
    from paper_2601_17091_amd.workloads import WORKLOADS, sample_rows, workload_series
    w = WORKLOADS["minirocket"]
    X_np = workload_series("minirocket", 20000)
    params = _fit(rk, mo, X_np[:1000], w.n_kernels, w.kernel_seed)
    _log("workload fit: %d dilations, %d features" % (len(params["dilations"]), params["biases"].shape[0]))
    F, _ = _run(rk, torch_gpu, params, X_np, False)
    rows = sample_rows(X_np.shape[0], X_np.shape[0], total=256)
    ref = mo.transform(X_np, params, rows=rows)
    _check(F[rows], ref, "workload sample")
