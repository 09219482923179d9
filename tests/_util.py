"""Shared helpers for the tests (fixture parsing, brute force, kernel sets)."""
import glob
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
MAX_LEN = 11


def load_golden():
    """Parse every worked-example fixture under tests/golden/."""
    out = []
    for path in sorted(glob.glob(os.path.join(GOLDEN, "w*.txt"))):
        rec = {"name": os.path.basename(path)}
        with open(path) as f:
            for line in f:
                line = line.split("#", 1)[0].strip()
                if not line:
                    continue
                key, val = line.split(":", 1)
                vals = [float(v) for v in val.split()]
                rec[key.strip()] = vals if len(vals) > 1 or key.strip() in ("x", "w", "y") else vals[0]
        out.append(rec)
    return out


def kernel_set(lengths, dilations, paddings, biases, weights):
    """Kernel arrays in the shared SoA layout (weights row stride 11, zero tail)."""
    K = len(lengths)
    W = np.zeros((K, MAX_LEN), dtype=np.float32)
    for k, w in enumerate(weights):
        W[k, :len(w)] = np.asarray(w, dtype=np.float32)
    return dict(length=np.asarray(lengths, dtype=np.int32),
                dilation=np.asarray(dilations, dtype=np.int32),
                padding=np.asarray(paddings, dtype=np.int32),
                bias=np.asarray(biases, dtype=np.float32), weights=W)


def brute_force(X, kernels):
    """Literal transcription of the definitions with Python floats (fp64).

    For every row and kernel: the dot products y_t, t < O, then PPV (strictly
    positive share) and MAX.  Independent of the C oracle; small inputs only.
    """
    n, L = X.shape
    K = len(kernels["length"])
    F = np.zeros((n, 2 * K))
    for i in range(n):
        x = [float(v) for v in X[i]]
        for k in range(K):
            ln = int(kernels["length"][k])
            d = int(kernels["dilation"][k])
            p = int(kernels["padding"][k])
            b = float(kernels["bias"][k])
            w = [float(v) for v in kernels["weights"][k][:ln]]
            O = L + 2 * p - (ln - 1) * d
            ys = []
            for t in range(O):
                acc = b
                for j in range(ln):
                    m = t - p + j * d
                    if 0 <= m < L:
                        acc += w[j] * x[m]
                ys.append(acc)
            F[i, 2 * k] = sum(1 for y in ys if y > 0) / O
            F[i, 2 * k + 1] = max(ys)
    return F


def brute_force_mpv(X, kernels):
    """Mean of the strictly positive dot products per (row, kernel), 0 when
    none is positive; literal Python loops in fp64, small inputs only."""
    n, L = X.shape
    K = len(kernels["length"])
    out = np.zeros((n, K))
    for i in range(n):
        x = [float(v) for v in X[i]]
        for k in range(K):
            ln = int(kernels["length"][k])
            d = int(kernels["dilation"][k])
            p = int(kernels["padding"][k])
            b = float(kernels["bias"][k])
            w = [float(v) for v in kernels["weights"][k][:ln]]
            pos = []
            for t in range(L + 2 * p - (ln - 1) * d):
                acc = b
                for j in range(ln):
                    m = t - p + j * d
                    if 0 <= m < L:
                        acc += w[j] * x[m]
                if acc > 0:
                    pos.append(acc)
            out[i, k] = sum(pos) / len(pos) if pos else 0.0
    return out


def random_kernels(rng, K, L, max_len=MAX_LEN):
    """Random valid kernels (any length 1..11, any admissible dilation, either
    padding choice) for brute-force cross-checks."""
    lengths, dil, pad, bias, weights = [], [], [], [], []
    for _ in range(K):
        ln = int(rng.choice([1, 2, 3, 5, 7, 9, 11])) if max_len >= 11 else int(rng.integers(1, max_len + 1))
        ln = min(ln, L)
        dmax = max(1, (L - 1) // max(1, ln - 1)) if ln > 1 else int(rng.integers(1, 5))
        d = int(rng.integers(1, dmax + 1))
        p = ((ln - 1) * d) // 2 if rng.integers(2) else 0
        if L + 2 * p - (ln - 1) * d < 1:
            p = ((ln - 1) * d) // 2
        lengths.append(ln)
        dil.append(d)
        pad.append(p)
        bias.append(float(rng.uniform(-1, 1)))
        weights.append(rng.standard_normal(ln).astype(np.float32))
    return kernel_set(lengths, dil, pad, bias, weights)


def fp32_features(X, kernels, order="ascending", with_mpv=False):
    """fp32 evaluation in numpy with a chosen summation order, used to check
    that the oracle's certified intervals contain real fp32 results."""
    n, L = X.shape
    K = len(kernels["length"])
    cnt = np.zeros((n, K), dtype=np.int64)
    mx = np.zeros((n, K), dtype=np.float64)
    mpv = np.zeros((n, K), dtype=np.float64)
    for k in range(K):
        ln = int(kernels["length"][k])
        d = int(kernels["dilation"][k])
        p = int(kernels["padding"][k])
        b = np.float32(kernels["bias"][k])
        w = kernels["weights"][k][:ln].astype(np.float32)
        O = L + 2 * p - (ln - 1) * d
        xz = np.zeros((n, L + 2 * p + 1), dtype=np.float32)
        xz[:, p:p + L] = X
        taps = range(ln) if order == "ascending" else range(ln - 1, -1, -1)
        y = np.full((n, O), b, dtype=np.float32) if order == "ascending" else np.zeros((n, O), np.float32)
        for j in taps:
            y = (y + w[j] * xz[:, j * d:j * d + O]).astype(np.float32)
        if order != "ascending":
            y = (y + b).astype(np.float32)
        cnt[:, k] = (y > 0).sum(axis=1)
        mx[:, k] = y.max(axis=1)
        if with_mpv:
            # positive values summed in fp32 in output order, then one fp32 division
            s32 = np.zeros(n, dtype=np.float32)
            for t in range(O):
                s32 = np.where(y[:, t] > 0, (s32 + y[:, t]).astype(np.float32), s32)
            c = cnt[:, k].astype(np.float32)
            mpv[:, k] = np.where(cnt[:, k] > 0, (s32 / np.maximum(c, 1)).astype(np.float32), 0.0)
    return (cnt, mx, mpv) if with_mpv else (cnt, mx)


def ceil_div(a, b):
    return -(-a // b)


def z_norm(x):
    x = np.asarray(x, dtype=np.float64)
    sd = x.std(axis=1, keepdims=True)
    sd[sd == 0] = 1
    return ((x - x.mean(axis=1, keepdims=True)) / sd).astype(np.float32)


__all__ = ["load_golden", "kernel_set", "brute_force", "brute_force_mpv", "random_kernels", "fp32_features",
           "ceil_div", "z_norm", "math"]


# ---------------------------------------------------------------------------
# parity rule shared by the GPU tests
# ---------------------------------------------------------------------------
MAX_ABS_TOL = 1e-4   # MAX within 1e-4 absolute on z-normalised input
COUNT_TOL = 2        # PPV within 2/O, i.e. the positive count within 2


def parity_report(F_gpu, ref):
    """Compare GPU features (fp32 [m, 2K]) with an oracle result on the same
    rows.  Returns a dict of the worst deviations and violation counts."""
    F_gpu = np.asarray(F_gpu, dtype=np.float64)
    O = ref["O"][None, :].astype(np.float64)
    ppv = F_gpu[:, 0::2]
    cnt = np.rint(ppv * O).astype(np.int64)
    mx = F_gpu[:, 1::2]
    dmax = np.abs(mx - ref["F"][:, 1::2])
    dcnt = np.abs(cnt - ref["cnt"])
    return dict(
        max_abs_err=float(dmax.max()) if dmax.size else 0.0,
        max_count_err=int(dcnt.max()) if dcnt.size else 0,
        # PPV must be the fp32 quotient (float)count / (float)O, correctly
        # rounded (exact at any O; a fixed tolerance on PPV * O - count
        # would not be: half an ulp of PPV times O reaches 1e-3 at O ~ 33,500)
        ppv_not_integral=int((F_gpu[:, 0::2].astype(np.float32)
                              != cnt.astype(np.float32) / O.astype(np.float32)).sum()),
        outside_count_interval=int(((cnt < ref["cnt_lo"]) | (cnt > ref["cnt_hi"])).sum()),
        max_beyond_bound=int((dmax > ref["beta"]).sum()),
        nonfinite=int((~np.isfinite(F_gpu)).sum()),
        ppv_out_of_range=int(((ppv < 0) | (ppv > 1)).sum()),
        n_features=int(cnt.size),
    )


def assert_parity(F_gpu, ref, what=""):
    r = parity_report(F_gpu, ref)
    assert r["nonfinite"] == 0, (what, r)
    assert r["ppv_out_of_range"] == 0, (what, r)
    assert r["ppv_not_integral"] == 0, (what, r)
    assert r["max_abs_err"] <= MAX_ABS_TOL, (what, r)
    assert r["max_count_err"] <= COUNT_TOL, (what, r)
    # stricter: inside the certified fp32 envelope of the exact result
    assert r["outside_count_interval"] == 0, (what, r)
    assert r["max_beyond_bound"] == 0, (what, r)
    return r


# ---------------------------------------------------------------------------
# MPV parity (the optional third feature)
# ---------------------------------------------------------------------------
MPV_REL_TOL = 1e-4   # |MPV_gpu - MPV_oracle| <= MPV_REL_TOL * MPV_oracle + beta
                     # where the GPU's count equals the oracle's


def split_mpv(F3):
    """[m, 3K] (PPV, MAX, MPV per kernel) -> ([m, 2K] (PPV, MAX), [m, K] MPV)."""
    F3 = np.asarray(F3)
    m, K3 = F3.shape
    K = K3 // 3
    F2 = np.empty((m, 2 * K), dtype=F3.dtype)
    F2[:, 0::2] = F3[:, 0::3]
    F2[:, 1::2] = F3[:, 1::3]
    return F2, F3[:, 2::3]


def assert_mpv_parity(F3, ref, what=""):
    """PPV and MAX under the usual rule; MPV inside the oracle's certified
    fp32 range and, where the GPU counted the same positives as the oracle,
    within MPV_REL_TOL * MPV + beta of it.  beta (the oracle's bound on any
    one dot product's fp32 error) covers the error the averaged values carry;
    the relative part covers the kernel's own summation: in the
    position-tiled layout each lane adds at most ceil(O/64) values in
    sequence and a 64-lane tree adds 6 more roundings, (O/64 + 6) * 2^-24 <
    1e-4 for every O below 2^24 / 100; in the series-lane layout (L <= 128)
    a lane adds the O <= 128 values of its series in sequence, 128 * 2^-24 <
    1e-4."""
    F2, mpv = split_mpv(F3)
    r = assert_parity(F2, ref, what)
    mpv = np.asarray(mpv, dtype=np.float64)
    assert np.all(np.isfinite(mpv)), what
    inside = (mpv >= ref["mpv_lo"]) & (mpv <= ref["mpv_hi"])
    assert inside.all(), (what, int((~inside).sum()))
    cnt = np.rint(F2[:, 0::2].astype(np.float64) * ref["O"][None, :]).astype(np.int64)
    same = cnt == ref["cnt"]
    err = np.abs(mpv - ref["mpv"])[same]
    lim = (MPV_REL_TOL * np.abs(ref["mpv"]) + ref["beta"])[same]
    assert np.all(err <= lim), (what, float((err - lim).max()))
    r["mpv_max_rel_err"] = float((err / np.maximum(np.abs(ref["mpv"][same]), 1e-30)).max()) if err.size else 0.0
    return r
