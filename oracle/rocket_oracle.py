"""ROCKET oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check in ``__graft_entry__`` and the CPU-baseline
leg of ``bench.py`` may import this module.  It shares no code with the HIP
library or its Python binding, and imports neither.

Two parts:

* ``transform`` -- ctypes wrapper around ``rocket_oracle.c``: the plain fp64
  evaluation of the ROCKET transform (paper Sec. 2.1 for the kernels and the
  two features, Sec. 3.2 for dividing the positive count by the number of dot
  products), plus certified fp32 error bounds for the parity tests.
* ``generate_kernels`` -- the kernel generator written from Sec. 2.1 in plain
  Python: length uniform on {7, 9, 11}, weights standard normal then
  mean-centred, bias uniform on [-1, 1), dilation floor(2^x) with x uniform on
  [0, A), A = log2((L-1)/(l-1)), zero padding (l-1)d/2 with probability 1/2.
  The random numbers come from SplitMix64 (Steele, Lea and Flood, OOPSLA 2014)
  used as a counter-based generator, and normals from the Box-Muller transform
  (Box and Muller, 1958).  The draw layout is fixed so that an independent
  implementation of the same published generator yields the same kernels:
  kernel k, draw slot s (0..15) reads stream element k*16 + s of the SplitMix64
  sequence started at ``seed``:
      slot 0        length   : (3 * (v >> 11)) >> 53 indexes (7, 9, 11)
      slots 1..12   weights  : six Box-Muller pairs (u1 from the odd slot, in
                               (0, 1]; u2 from the even slot, in [0, 1))
      slot 13       bias     : 2u - 1
      slot 14       dilation : floor(2 ** (u * A)), capped at (L-1) // (l-1)
      slot 15       padding  : applied when the top bit of v is set
  with u = (v >> 11) * 2^-53.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rocket_oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "minirocket_oracle.c")]
_LIB_PATH = os.path.join(_HERE, "librocket_oracle.so")

MAX_LEN = 11  # weights row stride used by the kernel arrays (longest kernel)

ORACLE_OK = 0
ORACLE_ERR_ARG = -1
ORACLE_ERR_LENGTH = -2


def build(force: bool = False) -> str:
    """Compile rocket_oracle.c and minirocket_oracle.c with gcc (fp64, no
    fast-math, no FMA contraction) into one library."""
    stale = not os.path.exists(_LIB_PATH) or any(
        os.path.getmtime(_LIB_PATH) < os.path.getmtime(src) for src in _SRCS)
    if force or stale:
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-o", tmp] + _SRCS + ["-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        p = ctypes.c_void_p
        lib.oracle_transform.restype = ctypes.c_int
        lib.oracle_transform.argtypes = [p, ctypes.c_int64, p, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, p, p, p, p, p, ctypes.c_int32,
                                         p, p, p, p, p, p, p, p, ctypes.c_int]
        lib.oracle_transform_mc.restype = ctypes.c_int
        lib.oracle_transform_mc.argtypes = [p, ctypes.c_int64, p, ctypes.c_int64, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_int32, p, p, p, p, p,
                                            ctypes.c_int32, p, p, p, p, p, p, p, p, p, p,
                                            ctypes.c_int]
        lib.oracle_output_length.restype = ctypes.c_int64
        lib.oracle_output_length.argtypes = [ctypes.c_int32] * 4
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_max_threads.argtypes = []
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def output_lengths(kernels: dict, L: int) -> np.ndarray:
    """O_k = L + 2 p_k - (l_k - 1) d_k for every kernel (Sec. 2.1)."""
    ln = np.asarray(kernels["length"], dtype=np.int64)
    d = np.asarray(kernels["dilation"], dtype=np.int64)
    p = np.asarray(kernels["padding"], dtype=np.int64)
    return L + 2 * p - (ln - 1) * d


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def transform(X, kernels: dict, rows=None, threads: int = 0) -> dict:
    """Plain fp64 ROCKET transform of the fp32 series X: [n, L] (univariate)
    or [n, C, L] (multivariate, Sec. 3.3: the kernel set then carries
    ``channel_count`` [K], ``channel_index`` [K, C] and ``weights``
    [K, C, stride], one weight row per channel slot).

    Returns a dict with
      F        fp64 [m, 2K]: PPV and MAX per kernel, interleaved;
      cnt      int64 [m, K]: positive counts;
      cnt_lo, cnt_hi int64 [m, K]: certified range of counts any fp32
               evaluation can give;
      beta     fp64 [m, K]: certified bound on |MAX_fp32 - MAX_exact|;
      mpv      fp64 [m, K]: mean of the positive dot products (0 if none);
      mpv_lo, mpv_hi fp64 [m, K]: certified range of MPV for any fp32
               evaluation (see rocket_oracle.c);
      O        int64 [K]: number of dot products per kernel.
    ``rows`` selects a subset of rows (m = len(rows)); default all rows.
    """
    X = np.ascontiguousarray(X, dtype=np.float32)
    if X.ndim == 2:
        n, L = X.shape
        C = 1
    elif X.ndim == 3:
        n, C, L = X.shape
    else:
        raise ValueError("X must be [n, L] or [n, C, L]")
    ln = np.ascontiguousarray(kernels["length"], dtype=np.int32)
    dl = np.ascontiguousarray(kernels["dilation"], dtype=np.int32)
    pd = np.ascontiguousarray(kernels["padding"], dtype=np.int32)
    bs = np.ascontiguousarray(kernels["bias"], dtype=np.float32)
    wt = np.ascontiguousarray(kernels["weights"], dtype=np.float32)
    K = ln.shape[0]
    if X.ndim == 3:
        if wt.ndim != 3 or wt.shape[:2] != (K, C):
            raise ValueError("multivariate weights must be [K, C, stride]")
        cc = np.ascontiguousarray(kernels["channel_count"], dtype=np.int32)
        ci = np.ascontiguousarray(kernels["channel_index"], dtype=np.int32)
        if cc.shape != (K,) or ci.shape != (K, C):
            raise ValueError("channel_count must be [K] and channel_index [K, C]")
        stride = wt.shape[2]
    else:
        if wt.ndim != 2 or wt.shape[0] != K:
            raise ValueError("weights must be [K, stride]")
        cc = ci = None
        stride = wt.shape[1]
    if rows is None:
        rows_arr = None
        m = n
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        m = rows_arr.shape[0]
    F = np.empty((m, 2 * K), dtype=np.float64)
    cnt = np.empty((m, K), dtype=np.int64)
    lo = np.empty((m, K), dtype=np.int64)
    hi = np.empty((m, K), dtype=np.int64)
    beta = np.empty((m, K), dtype=np.float64)
    mpv = np.empty((m, K), dtype=np.float64)
    mpv_lo = np.empty((m, K), dtype=np.float64)
    mpv_hi = np.empty((m, K), dtype=np.float64)
    rc = _load().oracle_transform_mc(_ptr(X), n, None if rows_arr is None else _ptr(rows_arr), m, C, L,
                                     K, _ptr(ln), _ptr(dl), _ptr(pd), _ptr(bs), _ptr(wt), stride,
                                     None if cc is None else _ptr(cc), None if ci is None else _ptr(ci),
                                     _ptr(F), _ptr(cnt), _ptr(lo), _ptr(hi), _ptr(beta), _ptr(mpv),
                                     _ptr(mpv_lo), _ptr(mpv_hi), int(threads))
    if rc == ORACLE_ERR_LENGTH:
        raise ValueError("a kernel has no dot products on series of length %d" % L)
    if rc != ORACLE_OK:
        raise ValueError("oracle_transform rejected its arguments (code %d)" % rc)
    return dict(F=F, cnt=cnt, cnt_lo=lo, cnt_hi=hi, beta=beta, mpv=mpv, mpv_lo=mpv_lo, mpv_hi=mpv_hi,
                O=output_lengths(kernels, L))


# ---------------------------------------------------------------------------
# Kernel generator (Sec. 2.1), pure Python.
# ---------------------------------------------------------------------------
_MASK64 = (1 << 64) - 1
_GOLDEN_GAMMA = 0x9E3779B97F4A7C15
_SLOTS = 16
_TWO_PI = 2.0 * math.pi


def splitmix64_mix(z: int) -> int:
    """The SplitMix64 output function (Steele, Lea, Flood 2014)."""
    z &= _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def splitmix64_at(seed: int, index: int) -> int:
    """Element ``index`` (0-based) of the SplitMix64 sequence started at ``seed``."""
    return splitmix64_mix((seed + (index + 1) * _GOLDEN_GAMMA) & _MASK64)


def _u01(v: int) -> float:
    return (v >> 11) * 2.0 ** -53


def _u01_open(v: int) -> float:
    return ((v >> 11) + 1) * 2.0 ** -53


def generate_kernels(seed: int, n_kernels: int, input_length: int) -> dict:
    """ROCKET kernels for series of length ``input_length`` (Sec. 2.1)."""
    if n_kernels < 1 or input_length < MAX_LEN:
        raise ValueError("need n_kernels >= 1 and input_length >= 11")
    seed &= _MASK64
    L = input_length
    length = np.zeros(n_kernels, dtype=np.int32)
    dilation = np.zeros(n_kernels, dtype=np.int32)
    padding = np.zeros(n_kernels, dtype=np.int32)
    bias = np.zeros(n_kernels, dtype=np.float32)
    weights = np.zeros((n_kernels, MAX_LEN), dtype=np.float32)
    for k in range(n_kernels):
        draw = [splitmix64_at(seed, k * _SLOTS + s) for s in range(_SLOTS)]
        ln = (7, 9, 11)[(3 * (draw[0] >> 11)) >> 53]
        z = []
        for i in range(6):
            u1 = _u01_open(draw[1 + 2 * i])
            u2 = _u01(draw[2 + 2 * i])
            r = math.sqrt(-2.0 * math.log(u1))
            theta = _TWO_PI * u2
            z.append(r * math.cos(theta))
            z.append(r * math.sin(theta))
        s = 0.0
        for j in range(ln):
            s += z[j]
        mean = s / ln
        for j in range(ln):
            weights[k, j] = np.float32(z[j] - mean)
        bias[k] = np.float32(2.0 * _u01(draw[13]) - 1.0)
        A = math.log2((L - 1) / (ln - 1))
        d = int(math.floor(math.pow(2.0, _u01(draw[14]) * A)))
        d = max(1, min(d, (L - 1) // (ln - 1)))
        p = (ln - 1) * d // 2 if (draw[15] >> 63) else 0
        length[k], dilation[k], padding[k] = ln, d, p
    return dict(length=length, dilation=dilation, padding=padding, bias=bias, weights=weights,
                input_length=L)


# ---------------------------------------------------------------------------
# Multivariate kernel generator (Sec. 3.3), pure Python.
# ---------------------------------------------------------------------------
MC_SLOTS = 512          # stream elements reserved per kernel
MC_MAX_CHANNELS = 32
_MC_SUBSET = 2          # first slot of the channel shuffle
_MC_NORMALS = 64        # first slot of the weight normals
_MC_BIAS, _MC_DIL, _MC_PAD = 509, 510, 511


def generate_kernels_multi(seed: int, n_kernels: int, input_length: int, n_channels: int) -> dict:
    """Multivariate ROCKET kernels (Sec. 3.3): each kernel also picks how many
    channels it reads and which.  Lengths, bias, dilation and padding follow
    Sec. 2.1 as in ``generate_kernels``; the channel count is floor(2^x), x
    uniform on [0, log2(C + 1)), clamped to [1, C]; the channels are a uniform
    random subset; each channel has its own weight row, standard normal and
    mean-centred over the kernel's taps.

    Stream layout: kernel k, slot s reads element k*512 + s of the SplitMix64
    sequence started at ``seed``; u = (v >> 11) * 2^-53.
      slot 0          length: (3 * (v >> 11)) >> 53 indexes (7, 9, 11)
      slot 1          channel count
      slots 2 .. C+1  partial Fisher-Yates shuffle of 0..C-1: step i swaps
                      position i with i + (((C - i) * (v >> 11)) >> 53)
                      (slot 2 + i); the first `count` entries, ascending
      slots 64 ..     normals from Box-Muller pairs, pair m from slots 64+2m
                      (u1 in (0, 1]) and 65+2m (u2 in [0, 1)); normal q is
                      weight (channel slot q // 11, tap q % 11)
      slot 509 bias 2u - 1; slot 510 dilation; slot 511 padding (top bit)
    Returns weights [K, C, 11] (rows past the kernel's count are zero),
    channel_count [K], channel_index [K, C] (-1 past the count)."""
    C = int(n_channels)
    if n_kernels < 1 or input_length < MAX_LEN or not (1 <= C <= MC_MAX_CHANNELS):
        raise ValueError("need n_kernels >= 1, input_length >= 11 and 1 <= n_channels <= 32")
    seed &= _MASK64
    L = input_length
    length = np.zeros(n_kernels, dtype=np.int32)
    dilation = np.zeros(n_kernels, dtype=np.int32)
    padding = np.zeros(n_kernels, dtype=np.int32)
    bias = np.zeros(n_kernels, dtype=np.float32)
    weights = np.zeros((n_kernels, C, MAX_LEN), dtype=np.float32)
    count = np.zeros(n_kernels, dtype=np.int32)
    index = np.full((n_kernels, C), -1, dtype=np.int32)
    for k in range(n_kernels):
        def draw(s):
            return splitmix64_at(seed, k * MC_SLOTS + s)
        ln = (7, 9, 11)[(3 * (draw(0) >> 11)) >> 53]
        cnt = int(math.floor(math.pow(2.0, _u01(draw(1)) * math.log2(C + 1))))
        cnt = max(1, min(cnt, C))
        perm = list(range(C))
        for i in range(cnt):
            j = i + (((C - i) * (draw(_MC_SUBSET + i) >> 11)) >> 53)
            perm[i], perm[j] = perm[j], perm[i]
        chans = sorted(perm[:cnt])
        z = []
        for m in range((cnt * MAX_LEN + 1) // 2):
            u1 = _u01_open(draw(_MC_NORMALS + 2 * m))
            u2 = _u01(draw(_MC_NORMALS + 2 * m + 1))
            r = math.sqrt(-2.0 * math.log(u1))
            theta = _TWO_PI * u2
            z.append(r * math.cos(theta))
            z.append(r * math.sin(theta))
        for sidx in range(cnt):
            row = z[sidx * MAX_LEN:sidx * MAX_LEN + ln]
            tot = 0.0
            for v in row:
                tot += v
            mean = tot / ln
            for j in range(ln):
                weights[k, sidx, j] = np.float32(row[j] - mean)
        bias[k] = np.float32(2.0 * _u01(draw(_MC_BIAS)) - 1.0)
        A = math.log2((L - 1) / (ln - 1))
        d = int(math.floor(math.pow(2.0, _u01(draw(_MC_DIL)) * A)))
        d = max(1, min(d, (L - 1) // (ln - 1)))
        p = (ln - 1) * d // 2 if (draw(_MC_PAD) >> 63) else 0
        length[k], dilation[k], padding[k] = ln, d, p
        count[k] = cnt
        index[k, :cnt] = chans
    return dict(length=length, dilation=dilation, padding=padding, bias=bias, weights=weights,
                channel_count=count, channel_index=index, n_channels=C, input_length=L)
