"""GPU parity of the optional third feature, MPV (mean of the positive
values), through the C ABI against the fp64 oracle: every plan layout on the
worked examples and hand-built kernels of every length, full workloads, and
the structural checks (determinism, agreement with the two-feature plan)."""
import sys

import numpy as np
import pytest

from _util import assert_mpv_parity, kernel_set, load_golden, random_kernels, split_mpv

pytestmark = pytest.mark.gpu

MODES = ["fused", "clamped", "direct"]


def _log(msg):
    print("[gpu-mpv] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def run(env, X_np, kernels, mode="fused"):
    torch, rk = env
    X = torch.from_numpy(np.ascontiguousarray(X_np, dtype=np.float32)).cuda()
    plan = rk.Plan(kernels, X.shape[1], direct=mode == "direct", clamped=mode == "clamped", mpv=True)
    info = plan.info()
    assert info["features_per_kernel"] == 3
    assert info["direct"] == (mode == "direct") and info["clamped"] == (mode == "clamped")
    F = plan.transform(X)
    torch.cuda.synchronize()
    assert F.shape == (X.shape[0], 3 * len(kernels["length"]))
    return F.cpu().numpy()


@pytest.mark.parametrize("mode", MODES)
def test_worked_examples_mpv(env, oracle, mode):
    for ex in load_golden():
        _log("worked example %s mode=%s" % (ex["name"], mode))
        X = np.asarray(ex["x"], dtype=np.float32)[None, :]
        ks = kernel_set([len(ex["w"])], [int(ex["dilation"])], [int(ex["padding"])], [ex["b"]], [ex["w"]])
        F = run(env, X, ks, mode)
        y = np.atleast_1d(np.asarray(ex["y"], dtype=np.float64))
        pos = y[y > 0]
        want = pos.mean() if pos.size else 0.0
        assert F[0, 2] == pytest.approx(want, rel=1e-6, abs=1e-7), ex["name"]
        assert_mpv_parity(F, oracle.transform(X, ks), ex["name"])


@pytest.mark.parametrize("mode", MODES)
def test_all_lengths_mpv(env, oracle, mode):
    rng = np.random.default_rng(4)
    L = 83
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in range(1, 12):
        dmax = (L - 1) // max(1, ln - 1) if ln > 1 else 30
        for d in sorted({1, 2, dmax}):
            for padded in (0, 1):
                lengths.append(ln)
                dil.append(d)
                pad.append((ln - 1) * d // 2 if padded else 0)
                bias.append(float(rng.uniform(-1, 1)))
                weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    X = rng.standard_normal((5, L)).astype(np.float32)
    _log("all lengths mode=%s" % mode)
    assert_mpv_parity(run(env, X, ks, mode), oracle.transform(X, ks), "lengths")


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_workload_every_row_mpv(env, oracle, name):
    from paper_2601_17091_amd.workloads import WORKLOADS, workload_series
    torch, rk = env
    w = WORKLOADS[name]
    ks = rk.generate_kernels(w.kernel_seed, w.n_kernels, w.L)
    X = workload_series(name)
    _log("workload %s with MPV, all rows" % name)
    r = assert_mpv_parity(run(env, X, ks), oracle.transform(X, ks), name)
    _log("  %s" % r)


@pytest.mark.parametrize("seed,mode", [(0, "fused"), (1, "clamped")])
def test_random_cases_mpv(env, oracle, seed, mode):
    rng = np.random.default_rng(700 + seed)
    L = int(rng.integers(11, 300))
    n = int(rng.integers(1, 7))
    ks = random_kernels(rng, 250, L)
    X = rng.standard_normal((n, L)).astype(np.float32)
    _log("random case seed=%d L=%d n=%d mode=%s" % (seed, L, n, mode))
    assert_mpv_parity(run(env, X, ks, mode), oracle.transform(X, ks), "random")


def test_mpv_plan_agrees_with_two_feature_plan(env):
    """Adding MPV changes nothing in PPV and MAX: same dot products, same
    reductions, bitwise."""
    torch, rk = env
    from paper_2601_17091_amd.workloads import make_series
    L = 400
    ks = rk.generate_kernels(31, 2500, L)
    X = torch.from_numpy(make_series("ar1", 23, L, 31)).cuda()
    a = rk.Plan(ks, L).transform(X)
    b = rk.Plan(ks, L, mpv=True).transform(X)
    b2 = rk.Plan(ks, L, mpv=True).transform(X)
    torch.cuda.synchronize()
    F2, mpv = split_mpv(b.cpu().numpy())
    assert np.array_equal(F2, a.cpu().numpy())
    assert torch.equal(b, b2)
    assert np.all(mpv >= 0)


def test_mpv_host_to_host(env):
    torch, rk = env
    from paper_2601_17091_amd.workloads import make_series
    L = 250
    ks = rk.generate_kernels(32, 900, L)
    X_np = make_series("sinusoids", 19, L, 32)
    p = rk.Plan(ks, L, mpv=True)
    want = p.transform(torch.from_numpy(X_np).cuda()).cpu()
    Xh = torch.from_numpy(X_np).pin_memory()
    Fh = torch.empty((19, 3 * 900), dtype=torch.float32, pin_memory=True)
    p.transform_host(Xh, Fh, batch_rows=4)
    assert torch.equal(Fh, want)
