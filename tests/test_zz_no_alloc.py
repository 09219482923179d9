"""rocket_transform_plan_noalloc, the entry point that allocates no device
memory (for callers that cannot allocate), against rocket_transform_plan:
the same kernels, so bitwise the same features, on two calls in a row (the
second on fewer series), in the series-lane layout that goes through the
library's static scratch in several chunks, with and without MPV, and in a
position-tiled plan that needs no scratch; a request whose 64-series chunk
exceeds the static scratch is refused before any device work."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20


def _log(msg):
    print("[gpu-noalloc] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def _chunk_rows(rk, ks, L, nf):
    n_slots = rk.plan_tables(ks, L)["slot_kernel"].shape[0]
    return min(8192, (SCRATCH_BYTES // 2) // (n_slots * nf * 4) // 64 * 64)


@pytest.mark.parametrize("mpv", [False, True])
def test_noalloc_series_lane_matches_transform_plan(env, mpv):
    torch, rk = env
    from paper_2601_17091_amd.workloads import make_series
    L, K = 64, 3000
    ks = rk.generate_kernels(301, K, L)
    plan = rk.Plan(ks, L, mpv=mpv, series=True)
    assert plan.info()["series_lane"]
    nf = 3 if mpv else 2
    chunk = _chunk_rows(rk, ks, L, nf)
    sizes = (3 * chunk + 77, chunk + 5)  # several chunks (both halves reused), then a smaller call
    _log("series-lane K=%d mpv=%s chunk=%d sizes=%s" % (K, mpv, chunk, sizes))
    for n in sizes:
        X = torch.from_numpy(make_series("trend", n, L, 400 + n)).cuda()
        want = plan.transform(X)
        got = torch.full((n, plan.n_features), float("nan"), dtype=torch.float32, device=X.device)
        plan.transform_into_noalloc(X, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), n


def test_noalloc_tiled_plan_matches_transform_plan(env):
    torch, rk = env
    from paper_2601_17091_amd.workloads import make_series
    L, K = 500, 2000
    ks = rk.generate_kernels(302, K, L)
    plan = rk.Plan(ks, L)
    for n in (37, 11):
        X = torch.from_numpy(make_series("sinusoids", n, L, 500 + n)).cuda()
        want = plan.transform(X)
        got = torch.empty_like(want)
        plan.transform_into_noalloc(X, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), n


def test_noalloc_refuses_oversized_chunk(env):
    torch, rk = env
    L, K = 64, 70000  # features of 64 series exceed half of the static scratch
    ks = rk.generate_kernels(303, K, L)
    plan = rk.Plan(ks, L, series=True)
    assert rk.plan_tables(ks, L)["slot_kernel"].shape[0] * 2 * 4 * 64 > SCRATCH_BYTES // 2
    X = torch.zeros((64, L), dtype=torch.float32, device="cuda")
    F = torch.full((64, plan.n_features), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(rk.RocketError) as e:
        plan.transform_into_noalloc(X, F)
    from paper_2601_17091_amd import rocket as rb
    assert e.value.status == rb.ROCKET_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((F == 7.0).all())
