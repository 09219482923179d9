"""MINIROCKET oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check in ``__graft_entry__`` and the CPU-baseline
leg of ``bench.py`` may import this module.  It shares no code with the HIP
library or its Python binding, and imports neither.

The CUROCKET paper (Sec. 5) names MINIROCKET (Dempster, Schmidt and Webb,
KDD 2021) as a ROCKET variant its principle carries over to, but does not
restate it; this module follows the published definition, in plain Python
(the fit) and plain C (``minirocket_oracle.c``, the fp64 transform):

* kernels: the 84 choices of 3 of 9 taps (lexicographic), weight 2 on the
  chosen taps and -1 on the others;
* dilations: ``fit_dilations`` -- the features per kernel (num_features // 84)
  are spread over at most 32 exponentially spaced dilations
  floor(2^e), e on an even grid over [0, log2((L-1)/8)], duplicates merged
  and their counts scaled, the remainder dealt one by one from the smallest
  dilation;
* biases: ``fit`` -- for each (dilation, kernel) pair one training series is
  drawn, its padded ("same") dilated convolution C_t, t = 0..L-1, computed,
  and the pair's biases are the quantiles of C at the low-discrepancy
  positions q_m = frac(m * golden ratio), m = 1, 2, ... (linear
  interpolation between order statistics);
* features: PPV of C_t - b over the pair's outputs; pairs with i + k even
  (dilation index i, kernel k) are padded (O = L), the others unpadded
  (O = L - 8d).

Random draws: the training series of pair (i, k) is
e = (n_train * (v >> 11)) >> 53 with v element i*84 + k of the SplitMix64
sequence started at ``seed`` (the same counter-based generator as the
ROCKET kernel generator; Steele, Lea and Flood, OOPSLA 2014).

Readings where MINIROCKET leaves a choice open (the design notes list them):
the convolution of the fit is summed in fp64, tap by tap in order; the
quantile positions are rounded to fp32 before use; the biases are the fp64
quantiles rounded to fp32.
"""
from __future__ import annotations

import ctypes
import math

import numpy as np

from oracle import rocket_oracle as _ro

N_KERNELS = 84
N_TAPS = 9
MAX_DILATIONS_PER_KERNEL = 32
_PHI = (math.sqrt(5.0) + 1.0) / 2.0


def kernel_choices() -> list:
    """The 3-of-9 tap choices, lexicographic."""
    out = []
    for a in range(N_TAPS):
        for b in range(a + 1, N_TAPS):
            for c in range(b + 1, N_TAPS):
                out.append((a, b, c))
    return out


def kernel_weights() -> np.ndarray:
    """[84, 9] weights: 2 on the chosen taps, -1 elsewhere."""
    w = -np.ones((N_KERNELS, N_TAPS), dtype=np.float64)
    for k, ch in enumerate(kernel_choices()):
        w[k, list(ch)] = 2.0
    return w


def fit_dilations(L: int, num_features: int = 10000,
                  max_dilations_per_kernel: int = MAX_DILATIONS_PER_KERNEL):
    """Dilations and features per kernel at each dilation."""
    if L < N_TAPS:
        raise ValueError("series must have at least 9 samples")
    per_kernel = num_features // N_KERNELS
    if per_kernel < 1:
        raise ValueError("need at least 84 features")
    T = min(per_kernel, max_dilations_per_kernel)
    multiplier = per_kernel / T
    max_exponent = math.log2((L - 1) / (N_TAPS - 1))
    raw = []
    for i in range(T):
        e = max_exponent if (T > 1 and i == T - 1) else (i * (max_exponent / (T - 1)) if T > 1 else 0.0)
        raw.append(int(math.pow(2.0, e)))
    dil = sorted(set(raw))
    counts = [raw.count(d) for d in dil]
    feats = [int(c * multiplier) for c in counts]
    rem = per_kernel - sum(feats)
    i = 0
    while rem > 0:
        feats[i] += 1
        rem -= 1
        i = (i + 1) % len(feats)
    return np.array(dil, dtype=np.int32), np.array(feats, dtype=np.int32)


def quantile_positions(n: int) -> np.ndarray:
    """q_m = frac(m * golden ratio), m = 1..n, rounded to fp32."""
    out = np.empty(n, dtype=np.float32)
    for m in range(1, n + 1):
        v = m * _PHI
        out[m - 1] = np.float32(v - math.floor(v))
    return out


def quantile_linear(sorted_vals: np.ndarray, q: float) -> float:
    """Quantile with linear interpolation between order statistics: position
    h = q (n - 1), value s[lo] + (h - lo) (s[lo+1] - s[lo])."""
    n = sorted_vals.shape[0]
    h = (n - 1) * float(q)
    lo = int(math.floor(h))
    if lo >= n - 1:
        return float(sorted_vals[n - 1])
    frac = h - lo
    a = float(sorted_vals[lo])
    b = float(sorted_vals[lo + 1])
    return a + frac * (b - a)


def same_convolution(x: np.ndarray, k: int, d: int) -> np.ndarray:
    """Padded dilated dot products of kernel k at dilation d over a series x
    (fp32): C_t = sum_j w[j] xz[t - 4d + j d], t = 0..L-1, summed in fp64 tap
    by tap."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    L = x.shape[0]
    w = kernel_weights()[k]
    xz = np.zeros(L + 8 * d, dtype=np.float64)
    xz[4 * d:4 * d + L] = x
    C = np.zeros(L, dtype=np.float64)
    for j in range(N_TAPS):
        C = C + w[j] * xz[j * d:j * d + L]
    return C


def example_index(seed: int, i: int, k: int, n_train: int) -> int:
    v = _ro.splitmix64_at(seed & ((1 << 64) - 1), i * N_KERNELS + k)
    return (n_train * (v >> 11)) >> 53


def fit(X_train, num_features: int = 10000, seed: int = 0,
        max_dilations_per_kernel: int = MAX_DILATIONS_PER_KERNEL) -> dict:
    """MINIROCKET parameters for series of the training set's length."""
    X_train = np.ascontiguousarray(X_train, dtype=np.float32)
    if X_train.ndim != 2 or X_train.shape[0] < 1:
        raise ValueError("X_train must be [n, L] with n >= 1")
    n, L = X_train.shape
    dil, feats = fit_dilations(L, num_features, max_dilations_per_kernel)
    total = N_KERNELS * int(feats.sum())
    qpos = quantile_positions(total)
    biases = np.empty(total, dtype=np.float32)
    examples = np.empty((dil.shape[0], N_KERNELS), dtype=np.int64)
    f = 0
    for i, d in enumerate(dil):
        for k in range(N_KERNELS):
            e = example_index(seed, i, k, n)
            examples[i, k] = e
            s = np.sort(same_convolution(X_train[e], k, int(d)))
            for q in range(int(feats[i])):
                biases[f] = np.float32(quantile_linear(s, qpos[f]))
                f += 1
    return dict(input_length=L, dilations=dil, features_per_dilation=feats, biases=biases,
                examples=examples)


def feature_layout(params: dict) -> dict:
    """Per feature: dilation index, kernel, padded flag and outputs O."""
    L = int(params["input_length"])
    dil, feats = params["dilations"], params["features_per_dilation"]
    di, kk, pad, O = [], [], [], []
    for i, d in enumerate(dil):
        for k in range(N_KERNELS):
            padded = (i + k) % 2 == 0
            for _ in range(int(feats[i])):
                di.append(i)
                kk.append(k)
                pad.append(padded)
                O.append(L if padded else L - 8 * int(d))
    return dict(dilation_index=np.array(di, np.int64), kernel=np.array(kk, np.int64),
                padded=np.array(pad, bool), O=np.array(O, np.int64))


def _load():
    lib = _ro._load()
    if not getattr(lib, "_mr_ready", False):
        p = ctypes.c_void_p
        lib.oracle_minirocket_transform.restype = ctypes.c_int
        lib.oracle_minirocket_transform.argtypes = [p, ctypes.c_int64, p, ctypes.c_int64, ctypes.c_int32,
                                                    ctypes.c_int32, p, p, p, p, p, p, p, ctypes.c_int]
        lib._mr_ready = True
    return lib


def transform(X, params: dict, rows=None, threads: int = 0) -> dict:
    """Plain fp64 MINIROCKET transform of the fp32 series X [n, L] with
    fitted ``params``.  Returns F fp64 [m, n_features] (PPV), cnt and the
    certified count range cnt_lo, cnt_hi (int64 [m, n_features]), and O
    (int64 [n_features])."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    if X.ndim != 2:
        raise ValueError("X must be [n, L]")
    n, L = X.shape
    dil = np.ascontiguousarray(params["dilations"], dtype=np.int32)
    feats = np.ascontiguousarray(params["features_per_dilation"], dtype=np.int32)
    biases = np.ascontiguousarray(params["biases"], dtype=np.float32)
    nf = N_KERNELS * int(feats.sum())
    if biases.shape != (nf,):
        raise ValueError("biases must have 84 * sum(features_per_dilation) entries")
    if rows is None:
        rows_arr, m = None, n
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        m = rows_arr.shape[0]
    F = np.empty((m, nf), dtype=np.float64)
    cnt = np.empty((m, nf), dtype=np.int64)
    lo = np.empty((m, nf), dtype=np.int64)
    hi = np.empty((m, nf), dtype=np.int64)
    ptr = _ro._ptr
    rc = _load().oracle_minirocket_transform(ptr(X), n, None if rows_arr is None else ptr(rows_arr), m, L,
                                             dil.shape[0], ptr(dil), ptr(feats), ptr(biases), ptr(F),
                                             ptr(cnt), ptr(lo), ptr(hi), int(threads))
    if rc == -2:
        raise ValueError("a dilation leaves no outputs on series of length %d" % L)
    if rc != 0:
        raise ValueError("oracle_minirocket_transform rejected its arguments (code %d)" % rc)
    lay = feature_layout(dict(params, input_length=L))
    return dict(F=F, cnt=cnt, cnt_lo=lo, cnt_hi=hi, O=lay["O"])
