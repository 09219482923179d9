"""GPU parity for multivariate series (Sec. 3.3) through the C ABI: every
kernel reads its own subset of the channels; the fused kernel runs its MFMA
chains over the union of its items' channels.  Checked against the fp64
oracle in every plan layout, with and without MPV, on hand-built channel
sets (one channel, all channels, empty slots' channels) and generated ones,
plus the host-to-host path and the workload the benchmark times."""
import sys

import numpy as np
import pytest

from _util import assert_mpv_parity, assert_parity

pytestmark = pytest.mark.gpu

MODES = ["fused", "clamped", "direct"]


def _log(msg):
    print("[gpu-mc] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch

    import paper_2601_17091_amd as rk
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    rk.library()
    return torch, rk


def run(env, X_np, ks, mode="fused", mpv=False):
    torch, rk = env
    X = torch.from_numpy(np.ascontiguousarray(X_np, dtype=np.float32)).cuda()
    plan = rk.Plan(ks, X.shape[-1], direct=mode == "direct", clamped=mode == "clamped", mpv=mpv)
    info = plan.info()
    assert info["direct"] == (mode == "direct") and info["clamped"] == (mode == "clamped")
    F = plan.transform(X)
    torch.cuda.synchronize()
    return F.cpu().numpy()


def _series(seed, n, C, L):
    from paper_2601_17091_amd.workloads import make_multichannel
    return make_multichannel(n, C, L, seed)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("mpv", [False, True])
def test_generated_sets(env, oracle, mode, mpv):
    torch, rk = env
    C, L = 5, 140
    ks = rk.generate_kernels_multi(61, 700, L, C)
    X = _series(61, 6, C, L)
    _log("generated set C=%d L=%d mode=%s mpv=%s" % (C, L, mode, mpv))
    F = run(env, X, ks, mode, mpv)
    ref = oracle.transform(X, ks)
    (assert_mpv_parity if mpv else assert_parity)(F, ref, "mc")


@pytest.mark.parametrize("mode", MODES)
def test_hand_built_channel_sets(env, oracle, mode):
    """Kernels of every length reading one channel, all channels, or a few,
    several of them sharing a bucket with different channel sets (the item's
    union then holds channels some slots do not read)."""
    rng = np.random.default_rng(8)
    C, L = 4, 70
    sets = [[0], [3], [1, 2], [0, 1, 2, 3], [0, 3], [2]]
    lengths, dil, pad, bias, count, index, weights = [], [], [], [], [], [], []
    for ln in (1, 3, 7, 9, 11):
        for d in (1, 2, (L - 1) // max(1, ln - 1) if ln > 1 else 5):
            for padded in (0, 1):
                for chans in sets:
                    lengths.append(ln)
                    dil.append(d)
                    pad.append((ln - 1) * d // 2 if padded else 0)
                    bias.append(float(rng.uniform(-1, 1)))
                    count.append(len(chans))
                    idx = np.full(C, -1, np.int32)
                    idx[:len(chans)] = chans
                    index.append(idx)
                    w = np.zeros((C, 11), np.float32)
                    w[:len(chans), :ln] = rng.standard_normal((len(chans), ln))
                    weights.append(w)
    ks = dict(length=np.array(lengths, np.int32), dilation=np.array(dil, np.int32),
              padding=np.array(pad, np.int32), bias=np.array(bias, np.float32),
              weights=np.array(weights, np.float32), n_channels=C,
              channel_count=np.array(count, np.int32), channel_index=np.array(index, np.int32))
    X = rng.standard_normal((5, C, L)).astype(np.float32)
    _log("hand-built channel sets mode=%s, %d kernels" % (mode, len(lengths)))
    assert_parity(run(env, X, ks, mode), oracle.transform(X, ks), "mc-hand")


def test_multivariate_workload_sampled(env, oracle):
    from paper_2601_17091_amd.workloads import WORKLOADS, sample_rows, workload_series
    torch, rk = env
    w = WORKLOADS["multivariate"]
    ks = rk.generate_kernels_multi(w.kernel_seed, w.n_kernels, w.L, w.channels)
    X_np = workload_series("multivariate")
    _log("workload multivariate %dx%dx%d K=%d" % (w.n, w.channels, w.L, w.n_kernels))
    plan = rk.Plan(ks, w.L)
    assert not plan.info()["direct"]
    X = torch.from_numpy(X_np).cuda()
    F = plan.transform(X)
    torch.cuda.synchronize()
    rows = sample_rows(w.n, w.n, total=256)
    got = F[torch.from_numpy(rows).cuda()].cpu().numpy()
    r = assert_parity(got, oracle.transform(X_np, ks, rows=rows), "multivariate")
    _log("  rows=%d %s" % (rows.shape[0], r))


def test_multichannel_host_to_host(env):
    torch, rk = env
    C, L = 3, 200
    ks = rk.generate_kernels_multi(62, 800, L, C)
    X_np = _series(62, 11, C, L)
    p = rk.Plan(ks, L)
    want = p.transform(torch.from_numpy(X_np).cuda()).cpu()
    Xh = torch.from_numpy(X_np).pin_memory()
    Fh = torch.empty((11, 2 * 800), dtype=torch.float32, pin_memory=True)
    p.transform_host(Xh, Fh, batch_rows=4)
    assert torch.equal(Fh, want)


def test_most_channels(env, oracle):
    """The largest channel count the ABI takes (32): the item channel masks
    reach their top channel."""
    torch, rk = env
    C, L = 32, 48
    ks = rk.generate_kernels_multi(96, 400, L, C)
    assert ks["channel_index"].max() == C - 1
    X = _series(96, 3, C, L)
    _log("C=%d" % C)
    assert_parity(run(env, X, ks, "fused"), oracle.transform(X, ks), "mc-C32")
