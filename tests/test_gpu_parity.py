"""GPU parity: the HIP path through the C ABI against the fp64 oracle on the
same seeded inputs.  Full workloads run in the launch configuration the
benchmark times; the oracle checks every row where it finishes in seconds
and a row sample (first/last row, first/last of every batch, seeded random
rows) elsewhere."""
import os
import sys

import numpy as np
import pytest

from _util import assert_mpv_parity, assert_parity, kernel_set, load_golden, random_kernels

pytestmark = pytest.mark.gpu


def _log(msg):
    print("[gpu-parity] " + msg, flush=True)
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


MODES = ["fused", "clamped", "direct"]


def run(rk, torch, X_np, kernels, mode="fused"):
    """Transform through the C ABI with the plan mode: the default fused
    layout, the fused kernel with clamped indices, or the direct kernel."""
    X = torch.from_numpy(np.ascontiguousarray(X_np, dtype=np.float32)).cuda()
    plan = rk.Plan(kernels, X.shape[1], direct=mode == "direct", clamped=mode == "clamped")
    info = plan.info()
    assert info["direct"] == (mode == "direct")
    assert info["clamped"] == (mode == "clamped")
    F = plan.transform(X)
    torch.cuda.synchronize()
    return F.cpu().numpy(), plan


@pytest.mark.parametrize("mode", MODES)
def test_worked_examples(torch_gpu, rk, oracle, mode):
    for ex in load_golden():
        _log("worked example %s mode=%s" % (ex["name"], mode))
        X = np.asarray(ex["x"], dtype=np.float32)[None, :]
        ks = kernel_set([len(ex["w"])], [int(ex["dilation"])], [int(ex["padding"])], [ex["b"]], [ex["w"]])
        F, _ = run(rk, torch_gpu, X, ks, mode)
        assert F[0, 1] == np.float32(ex["max"]), ex["name"]
        y = np.atleast_1d(np.asarray(ex["y"]))
        assert round(float(F[0, 0]) * len(y)) == int((y > 0).sum()), ex["name"]


@pytest.mark.parametrize("mode", MODES)
def test_zero_and_constant_series(torch_gpu, rk, mode):
    _log("zero/constant series mode=%s" % mode)
    ks = rk.generate_kernels(77, 2000, 300)
    F, _ = run(rk, torch_gpu, np.zeros((3, 300), np.float32), ks, mode)
    # X = 0: every dot product is the bias exactly
    np.testing.assert_array_equal(F[:, 1::2], np.broadcast_to(ks["bias"], (3, 2000)))
    np.testing.assert_array_equal(F[:, 0::2], np.broadcast_to((ks["bias"] > 0).astype(np.float32), (3, 2000)))
    F, _ = run(rk, torch_gpu, np.full((1, 300), 1.5, np.float32), ks, mode)
    unp = ks["padding"] == 0
    b = ks["bias"].astype(np.float64)
    assert np.all(np.abs(F[0, 1::2][unp] - b[unp]) < 1e-5)
    clear = unp & (np.abs(b) > 1e-4)
    np.testing.assert_array_equal(F[0, 0::2][clear], (b[clear] > 0).astype(np.float32))


@pytest.mark.parametrize("name,mode", [("tiny", "fused"), ("small", "fused"), ("small", "clamped")])
def test_full_workload_every_row(torch_gpu, rk, oracle, name, mode):
    from paper_2601_17091_amd.workloads import WORKLOADS, workload_series
    w = WORKLOADS[name]
    _log("workload %s: %dx%d, K=%d, all rows, mode=%s" % (name, w.n, w.L, w.n_kernels, mode))
    ks = rk.generate_kernels(w.kernel_seed, w.n_kernels, w.L)
    X = workload_series(name)
    F, plan = run(rk, torch_gpu, X, ks, mode)
    ref = oracle.transform(X, ks)
    r = assert_parity(F, ref, name)
    _log("  %s" % r)


def _sampled(torch, rk, oracle, name, total, batch_rows=None, mpv=False):
    from paper_2601_17091_amd.workloads import WORKLOADS, sample_rows, workload_series
    w = WORKLOADS[name]
    _log("workload %s: %dx%d, K=%d, sampled rows" % (name, w.n, w.L, w.n_kernels))
    ks = rk.generate_kernels(w.kernel_seed, w.n_kernels, w.L)
    X_np = workload_series(name)
    X = torch.from_numpy(X_np).cuda()
    plan = rk.Plan(ks, w.L, mpv=mpv)
    assert not plan.info()["direct"]
    nf = 3 if mpv else 2
    rows = sample_rows(w.n, batch_rows or w.n, total=total)
    assert rows.shape[0] == total
    got = np.zeros((rows.shape[0], nf * w.n_kernels), np.float32)
    if batch_rows is None:
        F = plan.transform(X)
        torch.cuda.synchronize()
        got[:] = F[torch.from_numpy(rows).cuda()].cpu().numpy()
        del F
    else:
        Fb = torch.empty((batch_rows, nf * w.n_kernels), dtype=torch.float32, device=X.device)

        def grab(r0, Fv):
            sel = rows[(rows >= r0) & (rows < r0 + Fv.shape[0])]
            if sel.size:
                torch.cuda.synchronize()
                got[np.searchsorted(rows, sel)] = Fv[torch.from_numpy(sel - r0).cuda()].cpu().numpy()
        rk.transform_batched(plan, X, Fb, batch_rows, on_batch=grab)
        torch.cuda.synchronize()
        del Fb
    ref = oracle.transform(X_np, ks, rows=rows)
    r = assert_mpv_parity(got, ref, name) if mpv else assert_parity(got, ref, name)
    _log("  rows=%d %s" % (rows.shape[0], r))


# sampled rows per workload: the first and last row, the first and last of
# every F batch, and seeded random rows up to these counts
ROWS_MANUFACTURING = 1024
ROWS_LONG = 64
ROWS_MANY_SHORT = 16384
ROWS_PAPER_SWEEP = 64


def test_manufacturing_sampled(torch_gpu, rk, oracle):
    _sampled(torch_gpu, rk, oracle, "manufacturing", total=ROWS_MANUFACTURING)


def test_manufacturing_mpv_sampled(torch_gpu, rk, oracle):
    """Manufacturing with MPV (one launch over all 10^5 series, F of
    3 x 10,000 features per series): sampled rows against the oracle."""
    _sampled(torch_gpu, rk, oracle, "manufacturing", total=ROWS_MANUFACTURING, mpv=True)


def test_long_sampled(torch_gpu, rk, oracle):
    _sampled(torch_gpu, rk, oracle, "long", total=ROWS_LONG)


def test_many_short_batched(torch_gpu, rk, oracle):
    _sampled(torch_gpu, rk, oracle, "many_short", total=ROWS_MANY_SHORT, batch_rows=100000)


def test_many_short_mpv_batched(torch_gpu, rk, oracle):
    """Many-short with MPV: the series-lane layout's three features through
    the slot-ordered buffer, every 10^5-row batch of the full workload."""
    _sampled(torch_gpu, rk, oracle, "many_short", total=ROWS_MANY_SHORT, batch_rows=100000, mpv=True)


def test_paper_sweep_sampled(torch_gpu, rk, oracle):
    """The default point of the paper's timing sweep (Sec. 4): 1,000 series
    of length 10,000 with 10,000 kernels."""
    _sampled(torch_gpu, rk, oracle, "paper_sweep", total=ROWS_PAPER_SWEEP)


def test_largest_sweep_kernel_set(torch_gpu, rk, oracle):
    """The largest kernel set of the paper's sweep (Sec. 4): 20,000 kernels on
    series of 10,000 samples (the sweep's generator seeds), every feature of
    3 rows against the oracle."""
    from paper_2601_17091_amd.workloads import make_series
    L, K = 10000, 20000
    ks = rk.generate_kernels(206, K, L)
    X = make_series("random_walk", 3, L, 106)
    _log("sweep point K=%d L=%d, 3 rows" % (K, L))
    plan = rk.Plan(ks, L)
    F = plan.transform(torch_gpu.from_numpy(X).cuda())
    torch_gpu.cuda.synchronize()
    assert_parity(F.cpu().numpy(), oracle.transform(X, ks), "K20000")


@pytest.mark.parametrize("mode", ["fused", "clamped"])
def test_longest_sweep_length_every_row(torch_gpu, rk, oracle, mode):
    """Series of length 20,000, the longest of the paper's sweep: one staged
    row with its zero margins takes ~160 KB of LDS (one workgroup per CU);
    the clamped layout needs half of that."""
    from paper_2601_17091_amd.workloads import make_series
    L = 20000
    ks = rk.generate_kernels(207, 600, L)
    X = make_series("random_walk", 3, L, 107)
    _log("length %d, K=%d, 3 rows, mode=%s" % (L, 600, mode))
    F, plan = run(rk, torch_gpu, X, ks, mode)
    assert_parity(F, oracle.transform(X, ks), "L20000")


@pytest.mark.parametrize("L,layout", [(39000, "clamped"), (50000, "direct")])
def test_longest_rows_layouts(torch_gpu, rk, oracle, L, layout):
    """Rows near and past the LDS limit, with the default plan: at 39,000
    samples even one padded row with its margins does not fit a workgroup's
    LDS, so the plan takes the clamped layout by itself; at 50,000 not even
    the clamped row fits and the plan falls back to the direct kernel.  Both
    against the oracle on every row and kernel."""
    from paper_2601_17091_amd.workloads import make_series
    ks = rk.generate_kernels(208, 200, L)
    X = make_series("random_walk", 2, L, 108)
    plan = rk.Plan(ks, L)
    info = plan.info()
    assert info["clamped"] == (layout == "clamped") and info["direct"] == (layout == "direct"), info
    _log("length %d, K=200, 2 rows, %s layout chosen by the plan" % (L, layout))
    F = plan.transform(torch_gpu.from_numpy(X).cuda())
    torch_gpu.cuda.synchronize()
    assert_parity(F.cpu().numpy(), oracle.transform(X, ks), "L%d" % L)


def test_largest_output_count(torch_gpu, rk, oracle):
    """The largest number of dot products a kernel may have: O just below
    2^24 (the bound that keeps counts exact in fp32), in a 16,777,215-sample
    series that only the direct kernel can take.  PPV = count / O then needs
    all 24 bits of the fp32 quotient."""
    rng = np.random.default_rng(5)
    L = (1 << 24) - 1
    lengths = [9, 7, 11, 9]
    dil = [1, 3, 2, 1]
    pad = [0, 0, 0, 4]  # the last one centred: O = L
    ks = kernel_set(lengths, dil, pad, [0.1, -0.2, 0.0, 0.05], [rng.standard_normal(n) for n in lengths])
    X = np.cumsum(rng.standard_normal((1, L)), axis=1).astype(np.float32)
    X = ((X - X.mean()) / X.std()).astype(np.float32)
    plan = rk.Plan(ks, L)
    assert plan.info()["direct"]
    _log("one series of %d samples, O up to %d, direct kernel" % (L, L))
    F = plan.transform(torch_gpu.from_numpy(X).cuda())
    torch_gpu.cuda.synchronize()
    ref = oracle.transform(X, ks)
    assert int(ref["O"].max()) == L
    assert_parity(F.cpu().numpy(), ref, "O = 2^24 - 1")


@pytest.mark.parametrize("mode", MODES)
def test_all_lengths_and_extremes(torch_gpu, rk, oracle, mode):
    """Hand-built kernels of every length 1..11, with dilation 1, 2 and the
    largest admissible one (O = 1 for unpadded kernels), padded or not, on a
    length that is not a multiple of 64 and a ragged row count."""
    _log("all lengths mode=%s" % mode)
    rng = np.random.default_rng(3)
    L = 97
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in range(1, 12):
        dmax = (L - 1) // max(1, ln - 1) if ln > 1 else 40
        for d in sorted({1, 2, 3, dmax, max(1, dmax // 2)}):
            for padded in (0, 1):
                lengths.append(ln)
                dil.append(d)
                pad.append((ln - 1) * d // 2 if padded else 0)
                bias.append(float(rng.uniform(-1, 1)))
                weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    X = rng.standard_normal((7, L)).astype(np.float32)
    F, _ = run(rk, torch_gpu, X, ks, mode)
    assert_parity(F, oracle.transform(X, ks), "lengths")


@pytest.mark.parametrize("seed,mode", [(0, "fused"), (1, "fused"), (2, "fused"), (3, "clamped"),
                                       (4, "clamped")])
def test_random_small_cases(torch_gpu, rk, oracle, seed, mode):
    rng = np.random.default_rng(900 + seed)
    L = int(rng.integers(11, 400))
    n = int(rng.integers(1, 9))
    _log("random case seed=%d L=%d n=%d mode=%s" % (seed, L, n, mode))
    ks = random_kernels(rng, 300, L)
    X = rng.standard_normal((n, L)).astype(np.float32)
    F, _ = run(rk, torch_gpu, X, ks, mode)
    assert_parity(F, oracle.transform(X, ks), "random")


@pytest.mark.parametrize("seed,mode", [(20, "fused"), (21, "fused"), (22, "clamped"), (23, "fused"),
                                       (24, "clamped"), (25, "fused")])
def test_random_generated_sets(torch_gpu, rk, oracle, seed, mode):
    """Generated kernel sets at random sizes (L log-uniform from 500 to
    8,000, K from 200 to 1,500, 2 to 5 series): MFMA, VALU and Toeplitz items
    in whatever mix the planner makes, against the oracle."""
    from paper_2601_17091_amd.workloads import make_series
    rng = np.random.default_rng(seed)
    L = int(np.exp(rng.uniform(np.log(500), np.log(8000))))
    K = int(rng.integers(200, 1500))
    n = int(rng.integers(2, 6))
    ks = rk.generate_kernels(1000 + seed, K, L)
    X = make_series("random_walk", n, L, 2000 + seed)
    _log("random generated set seed=%d L=%d K=%d n=%d mode=%s" % (seed, L, K, n, mode))
    F, plan = run(rk, torch_gpu, X, ks, mode)
    assert_parity(F, oracle.transform(X, ks), "random L=%d K=%d" % (L, K))


@pytest.mark.parametrize("mode", ["fused", "clamped"])
@pytest.mark.parametrize("mpv", [False, True])
def test_valu_items(torch_gpu, rk, oracle, mode, mpv):
    """Buckets of 1, 2, 5, 9 and 10 kernels at L = 200 (above the short-series
    limit): the one or two kernels left over in a bucket, and the fifth of a
    five, run as VALU items beside 4- and 8-kernel MFMA items; lengths 3, 7,
    9 and 11, padded and not, last tiles ragged."""
    from _util import assert_mpv_parity
    rng = np.random.default_rng(31)
    L = 200
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for size, (ln, d, padded) in zip((1, 2, 5, 10, 9, 1, 2, 2),
                                     ((9, 3, 0), (7, 5, 1), (11, 2, 0), (9, 1, 1), (3, 17, 0), (11, 19, 1), (7, 33, 0),
                                      (11, 7, 0))):
        for _ in range(size):
            lengths.append(ln)
            dil.append(d)
            pad.append((ln - 1) * d // 2 if padded else 0)
            bias.append(float(rng.uniform(-1, 1)))
            weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    t = rk.plan_tables(ks, L)
    assert set(range(6, 12)) <= set(t["items"][:, 0].tolist())  # every VALU variant
    X = rng.standard_normal((11, L)).astype(np.float32)
    _log("VALU items mode=%s mpv=%s" % (mode, mpv))
    Xd = torch_gpu.from_numpy(X).cuda()
    plan = rk.Plan(ks, L, clamped=mode == "clamped", mpv=mpv)
    F = plan.transform(Xd)
    torch_gpu.cuda.synchronize()
    ref = oracle.transform(X, ks)
    (assert_mpv_parity if mpv else assert_parity)(F.cpu().numpy(), ref, "valu items")


@pytest.mark.parametrize("mode", ["fused", "clamped"])
@pytest.mark.parametrize("mpv", [False, True])
def test_toeplitz_items(torch_gpu, rk, oracle, mode, mpv):
    """The one or two kernels left over in a bucket at a large dilation run
    as Toeplitz items (one MFMA group holding the kernel at 4 or 2 tap
    shifts): single and paired kernels at dilations around multiples of 64,
    padded and not, beside MFMA and VALU items, against the oracle."""
    from _util import assert_mpv_parity
    rng = np.random.default_rng(41)
    L = 1300
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for ln in (7, 9, 11):
        for d in (20, 60, 64, 65, 100, 127, 128, 129):
            if (ln - 1) * d >= L:
                continue
            for padded in (0, 1):
                for _ in range(1 + (d % 2) + 8 * (d == 20)):
                    lengths.append(ln)
                    dil.append(d)
                    pad.append((ln - 1) * d // 2 if padded else 0)
                    bias.append(float(rng.uniform(-1, 1)))
                    weights.append(rng.standard_normal(ln))
    ks = kernel_set(lengths, dil, pad, bias, weights)
    v = rk.plan_tables(ks, L)["items"][:, 0]
    assert ((v >= 12) & (v % 2 == 0)).any() and ((v >= 12) & (v % 2 == 1)).any() and (v < 12).any()
    X = np.cumsum(rng.standard_normal((5, L)), axis=1).astype(np.float32)
    _log("Toeplitz items mode=%s mpv=%s, %d kernels" % (mode, mpv, len(lengths)))
    Xd = torch_gpu.from_numpy(X).cuda()
    plan = rk.Plan(ks, L, clamped=mode == "clamped", mpv=mpv)
    assert plan.info()["toeplitz_items"] == int((v >= 12).sum())
    F = plan.transform(Xd)
    torch_gpu.cuda.synchronize()
    (assert_mpv_parity if mpv else assert_parity)(F.cpu().numpy(), oracle.transform(X, ks), "toeplitz")


def test_toeplitz_plan_two_streams(torch_gpu, rk):
    """A plan with Toeplitz items runs their kernel on a stream of its own,
    beside the fused kernel on the caller's stream.  Transforms of one such
    plan issued on two streams at once (and a third waiting on neither) each
    equal the one-stream result, bit for bit; the features of every call are
    complete when its own stream is synchronised."""
    torch = torch_gpu
    L = 5000
    ks = rk.generate_kernels(31, 2000, L)
    plan = rk.Plan(ks, L)
    assert plan.info()["toeplitz_items"] > 0
    rng = np.random.default_rng(31)
    Xa = torch.from_numpy(np.cumsum(rng.standard_normal((40, L)), axis=1).astype(np.float32)).cuda()
    Xb = torch.from_numpy(np.cumsum(rng.standard_normal((70, L)), axis=1).astype(np.float32)).cuda()
    want_a = plan.transform(Xa)
    want_b = plan.transform(Xb)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    Fa = torch.empty_like(want_a)
    Fb = torch.empty_like(want_b)
    for _ in range(3):
        Fa.fill_(float("nan"))
        Fb.fill_(float("nan"))
        torch.cuda.synchronize()
        plan.transform_into(Xa, Fa, sa)
        plan.transform_into(Xb, Fb, sb)
        sa.synchronize()
        assert torch.equal(Fa, want_a)
        sb.synchronize()
        assert torch.equal(Fb, want_b)
