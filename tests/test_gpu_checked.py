"""The checked build (librocket_checked.so, ROCKET_CHECKED=1) on the GPU.

Its device code checks every LDS tile read against the bytes its workgroup
staged and every feature store against its launch's rows and columns.  Each
case below runs the same transform through the product library and through
the checked one: the checked run must report no failed check, and, since the
checks change no arithmetic, give the same features bit for bit.  The cases
reach every kernel and layout: the fused kernel (padded and clamped rows,
4- and 8-kernel items, VALU items, MPV, multichannel items), the Toeplitz
kernel, the series-lane kernel and its permutation, the direct kernel and
the MINIROCKET kernel."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _log(msg):
    print("[gpu-checked] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def _series(rng, n, L, C=1):
    X = np.cumsum(rng.standard_normal((n, C, L)), axis=2)
    X = (X - X.mean(axis=2, keepdims=True)) / X.std(axis=2, keepdims=True)
    return np.ascontiguousarray(X.reshape(n, L) if C == 1 else X).astype(np.float32)


def _run(torch, rk, make_plan, X):
    Xd = torch.from_numpy(X).cuda()
    plan = make_plan()
    try:
        F = plan.transform(Xd)
        torch.cuda.synchronize()
        return F.cpu().numpy(), plan.info()
    finally:
        plan.close()


CASES = [
    # name, L, K, n, C, plan keyword arguments
    ("padded", 1000, 800, 9, 1, {}),
    ("padded mpv", 700, 600, 5, 1, {"mpv": True}),
    ("clamped", 3000, 500, 3, 1, {"clamped": True}),
    ("toeplitz", 5000, 2000, 3, 1, {}),
    ("series-lane", 64, 700, 4200, 1, {}),
    ("series-lane mpv", 48, 300, 4100, 1, {"mpv": True}),
    ("tiled short", 100, 900, 37, 1, {"tiled": True}),
    ("direct", 300, 200, 4, 1, {"direct": True}),
    ("multichannel", 400, 500, 6, 5, {}),
]


@pytest.mark.parametrize("name,L,K,n,C,kw", CASES, ids=[c[0] for c in CASES])
def test_checked_build_matches_product(env, name, L, K, n, C, kw):
    torch, rk = env
    rng = np.random.default_rng(abs(hash(name)) % (1 << 31))
    ks = (rk.generate_kernels_multi(5000 + L, K, L, C) if C > 1 else rk.generate_kernels(5000 + L, K, L))
    X = _series(rng, n, L, C)
    _log("%s: L=%d K=%d n=%d C=%d %s" % (name, L, K, n, C, kw))
    want, info = _run(torch, rk, lambda: rk.Plan(ks, L, **kw), X)
    if name == "toeplitz":
        assert info["toeplitz_items"] > 0
    if name.startswith("series-lane"):
        assert info["series_lane"]
    with rk.library_at(rk.rocket.CHECKED_LIB_PATH):
        assert rk.checked_build()
        assert rk.check_flags() == 0
        got, _ = _run(torch, rk, lambda: rk.Plan(ks, L, **kw), X)
        flags = rk.check_flags()
    assert flags == 0, "failed device checks: %#x" % flags
    assert np.array_equal(got, want, equal_nan=False)


def test_checked_build_minirocket(env):
    torch, rk = env
    rng = np.random.default_rng(77)
    L = 500
    X = _series(rng, 300, L)
    params = rk.minirocket_fit(X[:200], 2000, 7)
    _log("MINIROCKET L=%d, %d features" % (L, int(params["n_features"]) if "n_features" in params else -1))
    want, _ = _run(torch, rk, lambda: rk.MiniRocketPlan(params), X)
    with rk.library_at(rk.rocket.CHECKED_LIB_PATH):
        got, _ = _run(torch, rk, lambda: rk.MiniRocketPlan(params), X)
        flags = rk.check_flags()
    assert flags == 0, "failed device checks: %#x" % flags
    assert np.array_equal(got, want)
