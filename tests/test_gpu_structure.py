"""Structural GPU checks: determinism, batch and permutation invariance,
the one-shot entry point, the host-to-host entry point, empty input, and
the plain kernel against the fused one."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    from paper_2601_17091_amd.workloads import make_series
    L = 500
    ks = rk.generate_kernels(5, 3000, L)
    X = torch.from_numpy(make_series("sinusoids", 37, L, 55)).cuda()
    return torch, rk, ks, X


def test_deterministic(env):
    torch, rk, ks, X = env
    p = rk.Plan(ks, X.shape[1])
    a = p.transform(X)
    b = p.transform(X)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_rows_independent_of_batch(env):
    torch, rk, ks, X = env
    p = rk.Plan(ks, X.shape[1])
    full = p.transform(X)
    for r in (0, 17, 36):
        one = p.transform(X[r:r + 1].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(one[0], full[r])


def test_kernel_permutation(env):
    torch, rk, ks, X = env
    K = ks["length"].shape[0]
    perm = np.random.default_rng(1).permutation(K)
    pk = {k: (v[perm] if isinstance(v, np.ndarray) else v) for k, v in ks.items()}
    a = rk.Plan(ks, X.shape[1]).transform(X)
    b = rk.Plan(pk, X.shape[1]).transform(X)
    torch.cuda.synchronize()
    a = a.view(X.shape[0], K, 2)
    b = b.view(X.shape[0], K, 2)
    assert torch.equal(a[:, torch.from_numpy(perm).cuda()], b)


def test_one_shot_matches_plan(env):
    torch, rk, ks, X = env
    a = rk.Plan(ks, X.shape[1]).transform(X)
    b = rk.transform(X, ks)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_empty_input(env):
    torch, rk, ks, X = env
    p = rk.Plan(ks, X.shape[1])
    F = p.transform(X[:0])
    assert F.shape == (0, 2 * ks["length"].shape[0])


def test_direct_kernel_agrees(env):
    torch, rk, ks, X = env
    a = rk.Plan(ks, X.shape[1]).transform(X)
    b = rk.Plan(ks, X.shape[1], direct=True).transform(X)
    torch.cuda.synchronize()
    a = a.cpu().numpy()
    b = b.cpu().numpy()
    assert np.abs(a[:, 1::2] - b[:, 1::2]).max() < 1e-5
    O = 500 + 2 * ks["padding"] - (ks["length"] - 1) * ks["dilation"]
    assert np.abs(np.rint(a[:, 0::2] * O) - np.rint(b[:, 0::2] * O)).max() <= 2


@pytest.mark.parametrize("pinned,batch", [(True, 0), (True, 8), (False, 5)])
def test_host_to_host_matches_device(env, pinned, batch):
    """rocket_transform_host (overlapped copies, double-buffered batches,
    ragged last batch) gives exactly the device-resident result."""
    torch, rk, ks, X = env
    p = rk.Plan(ks, X.shape[1])
    want = p.transform(X)
    torch.cuda.synchronize()
    Xh = torch.empty(X.shape, dtype=torch.float32, pin_memory=pinned)
    Xh.copy_(X.cpu())
    Fh = torch.empty((X.shape[0], 2 * ks["length"].shape[0]), dtype=torch.float32, pin_memory=pinned)
    Fh.fill_(float("nan"))
    p.transform_host(Xh, Fh, batch_rows=batch)
    assert torch.equal(Fh, want.cpu())


def test_clamped_layout_matches_padded(env):
    """The clamped-index layout computes the same dot products in the same
    order as the zero-margin layout, so the features agree bitwise."""
    torch, rk, ks, X = env
    a = rk.Plan(ks, X.shape[1]).transform(X)
    b = rk.Plan(ks, X.shape[1], clamped=True).transform(X)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_large_lds_plan_survives_smaller_plan(env, oracle):
    """The dynamic-LDS limit is an attribute of the kernel functions shared
    by every plan of the process: creating a plan with a smaller footprint
    above 64 KB (series of 17,000 samples) must not lower it below what an
    earlier plan (20,000 samples, about 160 KB per workgroup) launches with."""
    torch, rk, _, _ = env
    from _util import assert_parity
    from paper_2601_17091_amd.workloads import make_series
    big_L, small_L = 20000, 17000
    ks_big = rk.generate_kernels(208, 300, big_L)
    ks_small = rk.generate_kernels(209, 300, small_L)
    big = rk.Plan(ks_big, big_L)
    small = rk.Plan(ks_small, small_L)
    assert big.info()["lds_bytes"] > small.info()["lds_bytes"] > 64 * 1024
    X_np = make_series("random_walk", 2, big_L, 108)
    F = big.transform(torch.from_numpy(X_np).cuda())
    torch.cuda.synchronize()
    assert_parity(F.cpu().numpy(), oracle.transform(X_np, ks_big), "big plan after small")
    Xs = make_series("random_walk", 2, small_L, 109)
    Fs = small.transform(torch.from_numpy(Xs).cuda())
    torch.cuda.synchronize()
    assert_parity(Fs.cpu().numpy(), oracle.transform(Xs, ks_small), "small plan")
