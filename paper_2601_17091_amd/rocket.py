"""ctypes binding of librocket.so (the C ABI declared in include/rocket.h).

Argument marshalling only: kernel arrays are passed as host pointers, X and F
as device pointers of torch tensors, the stream as torch's current HIP
stream.  Every step of the transform runs in the HIP library; if the library
is missing, calls raise instead of computing anything elsewhere.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
PRODUCT_LIB_PATH = os.path.join(HERE, "librocket.so")
# the checked build (device-side bounds checks, for debugging): used when the
# environment sets ROCKET_DEBUG=1
CHECKED_LIB_PATH = os.path.join(HERE, "librocket_checked.so")
LIB_PATH = CHECKED_LIB_PATH if os.environ.get("ROCKET_DEBUG") == "1" else PRODUCT_LIB_PATH

ROCKET_OK = 0
ROCKET_ERR_INVALID_ARG = -1
ROCKET_ERR_LENGTH = -2
ROCKET_ERR_OOM = -3
ROCKET_ERR_HIP = -4
ROCKET_ERR_INTERNAL = -5
ROCKET_ERR_SCRATCH = -6
ROCKET_PLAN_DEFAULT = 0
ROCKET_PLAN_DIRECT = 1
ROCKET_PLAN_CLAMPED = 2
ROCKET_PLAN_MPV = 4
ROCKET_PLAN_TILED = 8
ROCKET_PLAN_SERIES = 16
MAX_KERNEL_LENGTH = 11

# every symbol include/rocket.h declares
EXPORTED = (
    "rocket_generate_kernels",
    "rocket_generate_kernels_multi",
    "rocket_free_kernels",
    "rocket_plan_create",
    "rocket_plan_create_ex",
    "rocket_plan_destroy",
    "rocket_transform_plan",
    "rocket_transform_plan_noalloc",
    "rocket_transform",
    "rocket_transform_host",
    "rocket_plan_info",
    "rocket_plan_tables_build",
    "rocket_plan_tables_free",
    "rocket_status_string",
    "rocket_minirocket_fit",
    "rocket_minirocket_free",
    "rocket_minirocket_plan_create",
    "rocket_checked_build",
    "rocket_check_flags",
)


class RocketError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (what, status_string(status), status))


class CKernels(ctypes.Structure):
    _fields_ = [
        ("n_kernels", ctypes.c_int32),
        ("input_length", ctypes.c_int32),
        ("max_len", ctypes.c_int32),
        ("length", ctypes.POINTER(ctypes.c_int32)),
        ("dilation", ctypes.POINTER(ctypes.c_int32)),
        ("padding", ctypes.POINTER(ctypes.c_int32)),
        ("bias", ctypes.POINTER(ctypes.c_float)),
        ("weights", ctypes.POINTER(ctypes.c_float)),
        ("n_channels", ctypes.c_int32),
        ("channel_count", ctypes.POINTER(ctypes.c_int32)),
        ("channel_index", ctypes.POINTER(ctypes.c_int32)),
    ]


class CPlanFacts(ctypes.Structure):
    _fields_ = [
        ("n_items", ctypes.c_int64), ("n_buckets", ctypes.c_int64),
        ("mfma_per_row", ctypes.c_int64), ("lds_bytes", ctypes.c_int64),
        ("direct", ctypes.c_int32), ("clamped", ctypes.c_int32),
        ("features_per_kernel", ctypes.c_int32), ("rows_per_block", ctypes.c_int32),
        ("n_features", ctypes.c_int64), ("minirocket", ctypes.c_int32), ("series_lane", ctypes.c_int32),
        ("valu_fma_per_row", ctypes.c_int64), ("toeplitz_items", ctypes.c_int64),
    ]


class CMiniRocketParams(ctypes.Structure):
    _fields_ = [
        ("input_length", ctypes.c_int32), ("n_dilations", ctypes.c_int32),
        ("n_features", ctypes.c_int32),
        ("dilations", ctypes.POINTER(ctypes.c_int32)),
        ("features_per_dilation", ctypes.POINTER(ctypes.c_int32)),
        ("biases", ctypes.POINTER(ctypes.c_float)),
    ]


class CPlanTables(ctypes.Structure):
    _fields_ = [
        ("n_items", ctypes.c_int64), ("item_words", ctypes.c_int32), ("n_channels", ctypes.c_int32),
        ("items", ctypes.POINTER(ctypes.c_int32)),
        ("n_chan", ctypes.c_int64), ("chan", ctypes.POINTER(ctypes.c_int32)),
        ("n_wpk", ctypes.c_int64), ("wpk", ctypes.POINTER(ctypes.c_float)),
        ("n_slots", ctypes.c_int64), ("slot_bias", ctypes.POINTER(ctypes.c_float)),
        ("slot_kernel", ctypes.POINTER(ctypes.c_int32)),
        ("n_order", ctypes.c_int64), ("order", ctypes.POINTER(ctypes.c_int32)),
        ("n_split_begin", ctypes.c_int64), ("split_begin", ctypes.POINTER(ctypes.c_int32)),
        ("n_layouts", ctypes.c_int32), ("layout_off", ctypes.POINTER(ctypes.c_int32)),
        ("split_counts", ctypes.POINTER(ctypes.c_int32)),
        ("halo_lo", ctypes.c_int32), ("halo_hi", ctypes.c_int32), ("row_stride", ctypes.c_int32),
        ("tail_pad", ctypes.c_int32), ("internal", ctypes.c_void_p),
    ]


_lib = None


def _signatures() -> dict:
    """argtypes and restype of every entry point include/rocket.h declares."""
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    kp = ctypes.POINTER(CKernels)
    mp = ctypes.POINTER(CMiniRocketParams)
    st = ctypes.c_int
    return {
        "rocket_generate_kernels": ([ctypes.c_uint64, i32, i32, kp], st),
        "rocket_generate_kernels_multi": ([ctypes.c_uint64, i32, i32, i32, kp], st),
        "rocket_free_kernels": ([kp], None),
        "rocket_plan_create": ([kp, i32, ctypes.POINTER(vp)], st),
        "rocket_plan_create_ex": ([kp, i32, ctypes.c_uint32, ctypes.POINTER(vp)], st),
        "rocket_plan_destroy": ([vp], None),
        "rocket_transform_plan": ([vp, vp, i64, vp, vp], st),
        "rocket_transform_plan_noalloc": ([vp, vp, i64, vp, vp], st),
        "rocket_transform": ([vp, i64, i32, kp, vp, vp], st),
        "rocket_transform_host": ([vp, vp, i64, vp, i64, vp], st),
        "rocket_plan_info": ([vp, ctypes.POINTER(CPlanFacts)], st),
        "rocket_plan_tables_build": ([kp, i32, ctypes.POINTER(CPlanTables)], st),
        "rocket_plan_tables_free": ([ctypes.POINTER(CPlanTables)], None),
        "rocket_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "rocket_checked_build": ([], ctypes.c_int32),
        "rocket_check_flags": ([ctypes.POINTER(ctypes.c_uint32)], ctypes.c_int),
        "rocket_minirocket_fit": ([vp, i64, i32, i32, ctypes.c_uint64, mp], st),
        "rocket_minirocket_free": ([mp], None),
        "rocket_minirocket_plan_create": ([mp, ctypes.c_uint32, ctypes.POINTER(vp)], st),
    }


# the entry points that run on the host only (generator, planner tables,
# MINIROCKET fit, status strings): plain C++ with no HIP code
HOST_SYMBOLS = (
    "rocket_generate_kernels",
    "rocket_generate_kernels_multi",
    "rocket_free_kernels",
    "rocket_plan_tables_build",
    "rocket_plan_tables_free",
    "rocket_status_string",
    "rocket_minirocket_fit",
    "rocket_minirocket_free",
)


def bind(lib: ctypes.CDLL, names=EXPORTED) -> ctypes.CDLL:
    """Set the ctypes signatures of `names` on a loaded library (a missing
    symbol raises AttributeError)."""
    sig = _signatures()
    for name in names:
        fn = getattr(lib, name)
        fn.argtypes, fn.restype = sig[name]
    return lib


def library() -> ctypes.CDLL:
    """Load librocket.so (built by ``build_lib.build``); raise if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("librocket.so is not built (run paper_2601_17091_amd.build_lib.build())")
    _lib = bind(ctypes.CDLL(LIB_PATH))
    return _lib


@contextlib.contextmanager
def library_at(path: str):
    """Route the binding's calls to the library at `path` inside the block
    (for example the checked build, CHECKED_LIB_PATH).  A plan keeps the
    library that made it, so a plan made inside stays valid after the block."""
    global _lib
    if not os.path.exists(path):
        raise RuntimeError("%s is not built (run paper_2601_17091_amd.build_lib.build())" % path)
    prev = _lib
    _lib = bind(ctypes.CDLL(path))
    try:
        yield _lib
    finally:
        _lib = prev


def checked_build() -> bool:
    """Whether the loaded library is the checked build."""
    return bool(library().rocket_checked_build())


def check_flags() -> int:
    """The device-side checks that failed since the last call (checked
    builds; waits for the device): bit 0 an LDS read, bit 1 a feature store,
    bit 2 a slot column read of the series-lane permutation."""
    v = ctypes.c_uint32(0)
    _check(library().rocket_check_flags(ctypes.byref(v)), "rocket_check_flags")
    return int(v.value)


def status_string(status: int) -> str:
    return library().rocket_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != ROCKET_OK:
        raise RocketError(status, what)


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def as_c_kernels(kernels: dict):
    """A CKernels view of numpy kernel arrays (kept alive by the returned
    tuple).  Univariate sets: weights [K, max_len].  Multivariate sets carry
    n_channels C > 1, channel_count [K], channel_index [K, C] and weights
    [K, C, max_len]."""
    length = np.ascontiguousarray(kernels["length"], dtype=np.int32)
    dilation = np.ascontiguousarray(kernels["dilation"], dtype=np.int32)
    padding = np.ascontiguousarray(kernels["padding"], dtype=np.int32)
    bias = np.ascontiguousarray(kernels["bias"], dtype=np.float32)
    weights = np.ascontiguousarray(kernels["weights"], dtype=np.float32)
    K = length.shape[0]
    C = int(kernels.get("n_channels", 1))
    if C > 1:
        if weights.ndim != 3 or weights.shape[:2] != (K, C):
            raise ValueError("multivariate weights must be [n_kernels, n_channels, max_len]")
        count = np.ascontiguousarray(kernels["channel_count"], dtype=np.int32)
        index = np.ascontiguousarray(kernels["channel_index"], dtype=np.int32)
        if count.shape != (K,) or index.shape != (K, C):
            raise ValueError("channel_count must be [n_kernels], channel_index [n_kernels, n_channels]")
        count_p, index_p = _ptr(count, ctypes.c_int32), _ptr(index, ctypes.c_int32)
        max_len = weights.shape[2]
    else:
        if weights.ndim != 2 or weights.shape[0] != K:
            raise ValueError("weights must be [n_kernels, max_len]")
        count = index = None
        count_p = index_p = ctypes.POINTER(ctypes.c_int32)()
        max_len = weights.shape[1]
    c = CKernels(int(K), int(kernels.get("input_length", 0)), int(max_len),
                 _ptr(length, ctypes.c_int32), _ptr(dilation, ctypes.c_int32),
                 _ptr(padding, ctypes.c_int32), _ptr(bias, ctypes.c_float),
                 _ptr(weights, ctypes.c_float), C, count_p, index_p)
    return c, (length, dilation, padding, bias, weights, count, index)


def _kernels_to_numpy(ck) -> dict:
    K, M, C = ck.n_kernels, ck.max_len, max(1, ck.n_channels)
    out = dict(
        length=np.ctypeslib.as_array(ck.length, (K,)).copy(),
        dilation=np.ctypeslib.as_array(ck.dilation, (K,)).copy(),
        padding=np.ctypeslib.as_array(ck.padding, (K,)).copy(),
        bias=np.ctypeslib.as_array(ck.bias, (K,)).copy(),
        input_length=ck.input_length,
    )
    if C > 1:
        out["weights"] = np.ctypeslib.as_array(ck.weights, (K * C * M,)).copy().reshape(K, C, M)
        out["n_channels"] = C
        out["channel_count"] = np.ctypeslib.as_array(ck.channel_count, (K,)).copy()
        out["channel_index"] = np.ctypeslib.as_array(ck.channel_index, (K * C,)).copy().reshape(K, C)
    else:
        out["weights"] = np.ctypeslib.as_array(ck.weights, (K * M,)).copy().reshape(K, M)
    return out


def generate_kernels(seed: int, n_kernels: int, input_length: int) -> dict:
    """rocket_generate_kernels, copied into numpy arrays (library copy freed)."""
    lib = library()
    ck = CKernels()
    _check(lib.rocket_generate_kernels(ctypes.c_uint64(seed & (2 ** 64 - 1)), n_kernels, input_length,
                                       ctypes.byref(ck)), "rocket_generate_kernels")
    try:
        return _kernels_to_numpy(ck)
    finally:
        lib.rocket_free_kernels(ctypes.byref(ck))


def generate_kernels_multi(seed: int, n_kernels: int, input_length: int, n_channels: int) -> dict:
    """rocket_generate_kernels_multi (multivariate kernels, Sec. 3.3), copied
    into numpy arrays: weights [K, C, 11], channel_count [K], channel_index
    [K, C] (-1 past each kernel's count); for C = 1 the univariate form."""
    lib = library()
    ck = CKernels()
    _check(lib.rocket_generate_kernels_multi(ctypes.c_uint64(seed & (2 ** 64 - 1)), n_kernels,
                                             input_length, n_channels, ctypes.byref(ck)),
           "rocket_generate_kernels_multi")
    try:
        # a one-channel set comes back in the univariate form (weights [K, 11])
        return _kernels_to_numpy(ck)
    finally:
        lib.rocket_free_kernels(ctypes.byref(ck))


def plan_tables(kernels: dict, L: int) -> dict:
    """rocket_plan_tables_build copied into numpy arrays (host only)."""
    lib = library()
    c, keep = as_c_kernels(kernels)
    t = CPlanTables()
    _check(lib.rocket_plan_tables_build(ctypes.byref(c), int(L), ctypes.byref(t)),
           "rocket_plan_tables_build")
    try:
        def arr(ptr, n, shape=None):
            a = np.ctypeslib.as_array(ptr, (int(n),)).copy() if n > 0 else np.zeros(0)
            return a.reshape(shape) if shape is not None else a
        out = dict(
            items=arr(t.items, t.n_items * t.item_words, (int(t.n_items), int(t.item_words))),
            chan=arr(t.chan, t.n_chan),
            n_channels=t.n_channels,
            wpk=arr(t.wpk, t.n_wpk),
            slot_bias=arr(t.slot_bias, t.n_slots),
            slot_kernel=arr(t.slot_kernel, t.n_slots),
            order=arr(t.order, t.n_order),
            split_begin=arr(t.split_begin, t.n_split_begin),
            layout_off=arr(t.layout_off, t.n_layouts),
            split_counts=arr(t.split_counts, t.n_layouts),
            halo_lo=t.halo_lo, halo_hi=t.halo_hi, row_stride=t.row_stride,
            tail_pad=t.tail_pad,
        )
    finally:
        lib.rocket_plan_tables_free(ctypes.byref(t))
    del keep
    return out


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _series_shape_ok(X, L: int, C: int) -> bool:
    if C > 1:
        return X.dim() == 3 and X.shape[1] == C and X.shape[2] == L
    return X.dim() == 2 and X.shape[1] == L


def _check_series(X, L: int, C: int = 1):
    import torch
    if not isinstance(X, torch.Tensor) or not X.is_cuda:
        raise TypeError("X must be a torch tensor on the GPU")
    if X.dtype != torch.float32 or not _series_shape_ok(X, L, C) or not X.is_contiguous():
        raise ValueError("X must be contiguous float32 %s" % ("[n, %d, %d]" % (C, L) if C > 1 else "[n, %d]" % L))


class Plan:
    """rocket_plan: a kernel set planned for series of length L on the current device."""

    def __init__(self, kernels: dict, L: int, direct: bool = False, clamped: bool = False,
                 mpv: bool = False, tiled: bool = False, series: bool = False):
        lib = library()
        self._lib = lib  # every call on this plan goes to the library that made it
        self._c, self._keep = as_c_kernels(kernels)
        self.n_kernels = int(self._c.n_kernels)
        self.L = int(L)
        h = ctypes.c_void_p()
        flags = ((ROCKET_PLAN_DIRECT if direct else ROCKET_PLAN_DEFAULT)
                 | (ROCKET_PLAN_CLAMPED if clamped else 0) | (ROCKET_PLAN_MPV if mpv else 0)
                 | (ROCKET_PLAN_TILED if tiled else 0) | (ROCKET_PLAN_SERIES if series else 0))
        _check(lib.rocket_plan_create_ex(ctypes.byref(self._c), self.L, flags, ctypes.byref(h)),
               "rocket_plan_create")
        self._h = h
        self.features_per_kernel = 3 if mpv else 2
        self.n_channels = max(1, int(self._c.n_channels))

    def info(self) -> dict:
        f = CPlanFacts()
        _check(self._lib.rocket_plan_info(self._h, ctypes.byref(f)), "rocket_plan_info")
        return dict(n_items=f.n_items, n_buckets=f.n_buckets, mfma_per_row=f.mfma_per_row,
                    lds_bytes=f.lds_bytes, direct=bool(f.direct), clamped=bool(f.clamped),
                    features_per_kernel=f.features_per_kernel, rows_per_block=f.rows_per_block,
                    n_features=f.n_features, minirocket=bool(f.minirocket),
                    series_lane=bool(f.series_lane), valu_fma_per_row=f.valu_fma_per_row,
                    toeplitz_items=f.toeplitz_items)

    @property
    def n_features(self) -> int:
        """Columns of F: features_per_kernel * n_kernels (MINIROCKET: its
        feature count)."""
        return self.features_per_kernel * self.n_kernels

    def transform_into(self, X, F, stream=None):
        """F[n, fK] <- features of X[n, L] (f = 2, or 3 with MPV);
        asynchronous on `stream`."""
        self._check_io(X, F)
        _check(self._lib.rocket_transform_plan(self._h, ctypes.c_void_p(X.data_ptr()), X.shape[0],
                                               ctypes.c_void_p(F.data_ptr()), _stream_handle(stream)),
               "rocket_transform_plan")
        return F

    def _check_io(self, X, F):
        import torch
        _check_series(X, self.L, self.n_channels)
        n = X.shape[0]
        if (not isinstance(F, torch.Tensor) or not F.is_cuda or F.dtype != torch.float32
                or tuple(F.shape) != (n, self.n_features) or not F.is_contiguous()):
            raise ValueError("F must be contiguous float32 [n, %d] on the GPU" % self.n_features)
        if X.device != F.device:
            raise ValueError("X and F must be on the same device")

    def transform(self, X, stream=None):
        import torch
        F = torch.empty((X.shape[0], self.n_features), dtype=torch.float32, device=X.device)
        return self.transform_into(X, F, stream)

    def transform_into_noalloc(self, X, F, stream=None):
        """transform_into through rocket_transform_plan_noalloc: no device
        allocation in the library (the series-lane layout uses its static
        scratch); the caller allocates F."""
        self._check_io(X, F)
        _check(self._lib.rocket_transform_plan_noalloc(self._h, ctypes.c_void_p(X.data_ptr()), X.shape[0],
                                                       ctypes.c_void_p(F.data_ptr()), _stream_handle(stream)),
               "rocket_transform_plan_noalloc")
        return F

    def transform_host(self, X_host, F_host, batch_rows: int = 0, stream=None):
        """F_host[n, fK] <- features of X_host[n, L], both in host memory
        (CPU torch tensors, pinned for overlap, or numpy arrays); copies and
        transforms of successive row batches overlap.  Blocks until done."""
        import torch
        X_t = X_host if isinstance(X_host, torch.Tensor) else torch.from_numpy(X_host)
        F_t = F_host if isinstance(F_host, torch.Tensor) else torch.from_numpy(F_host)
        if X_t.is_cuda or F_t.is_cuda:
            raise ValueError("transform_host takes host tensors")
        if X_t.dtype != torch.float32 or not X_t.is_contiguous() or not _series_shape_ok(X_t, self.L, self.n_channels):
            raise ValueError("X_host must be a contiguous float32 series array for this plan")
        n = X_t.shape[0]
        if (F_t.dtype != torch.float32 or not F_t.is_contiguous()
                or tuple(F_t.shape) != (n, self.n_features)):
            raise ValueError("F_host must be a contiguous float32 [%d, %d] array" % (n, self.n_features))
        if stream is None:
            stream = torch.cuda.current_stream()
        _check(self._lib.rocket_transform_host(self._h, ctypes.c_void_p(X_t.data_ptr()), n,
                                               ctypes.c_void_p(F_t.data_ptr()), int(batch_rows),
                                               ctypes.c_void_p(stream.cuda_stream)),
               "rocket_transform_host")
        return F_host

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.rocket_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def minirocket_fit(X_train, num_features: int = 10000, seed: int = 0) -> dict:
    """rocket_minirocket_fit on a host training set X_train [n, L] (fp32),
    copied into numpy arrays (library copy freed)."""
    lib = library()
    X = np.ascontiguousarray(X_train, dtype=np.float32)
    if X.ndim != 2:
        raise ValueError("X_train must be [n, L]")
    cp = CMiniRocketParams()
    _check(lib.rocket_minirocket_fit(_ptr(X, ctypes.c_float), X.shape[0], X.shape[1], int(num_features),
                                     ctypes.c_uint64(seed & (2 ** 64 - 1)), ctypes.byref(cp)),
           "rocket_minirocket_fit")
    try:
        nd, nf = cp.n_dilations, cp.n_features
        return dict(input_length=cp.input_length,
                    dilations=np.ctypeslib.as_array(cp.dilations, (nd,)).copy(),
                    features_per_dilation=np.ctypeslib.as_array(cp.features_per_dilation, (nd,)).copy(),
                    biases=np.ctypeslib.as_array(cp.biases, (nf,)).copy())
    finally:
        lib.rocket_minirocket_free(ctypes.byref(cp))


def as_c_minirocket(params: dict):
    """A rocket_minirocket_params view of numpy MINIROCKET parameters; returns
    (struct, keepalive)."""
    dil = np.ascontiguousarray(params["dilations"], dtype=np.int32)
    feats = np.ascontiguousarray(params["features_per_dilation"], dtype=np.int32)
    biases = np.ascontiguousarray(params["biases"], dtype=np.float32)
    c = CMiniRocketParams(int(params["input_length"]), dil.shape[0], biases.shape[0],
                          _ptr(dil, ctypes.c_int32), _ptr(feats, ctypes.c_int32), _ptr(biases, ctypes.c_float))
    return c, (dil, feats, biases)


class MiniRocketPlan(Plan):
    """rocket_minirocket_plan_create: MINIROCKET parameters planned for series
    of their input length; transform_into writes F [n, n_features] (PPV)."""

    def __init__(self, params: dict, clamped: bool = False):
        lib = library()
        self._lib = lib
        self._c, self._keep = as_c_minirocket(params)
        self.L = int(params["input_length"])
        h = ctypes.c_void_p()
        _check(lib.rocket_minirocket_plan_create(ctypes.byref(self._c),
                                                 ROCKET_PLAN_CLAMPED if clamped else ROCKET_PLAN_DEFAULT,
                                                 ctypes.byref(h)), "rocket_minirocket_plan_create")
        self._h = h
        self.n_kernels = 84
        self.features_per_kernel = 0
        self.n_channels = 1
        self._n_features = int(self._c.n_features)

    @property
    def n_features(self) -> int:
        return self._n_features


def transform(X, kernels: dict, stream=None):
    """One-shot rocket_transform: returns F[n, 2K] (blocks until done)."""
    import torch
    c, keep = as_c_kernels(kernels)
    C = max(1, int(c.n_channels))
    L = int(X.shape[-1]) if C > 1 else int(X.shape[1])
    _check_series(X, L, C)
    F = torch.empty((X.shape[0], 2 * c.n_kernels), dtype=torch.float32, device=X.device)
    _check(library().rocket_transform(ctypes.c_void_p(X.data_ptr()), X.shape[0], L, ctypes.byref(c),
                                      ctypes.c_void_p(F.data_ptr()), _stream_handle(stream)),
           "rocket_transform")
    del keep
    return F


def transform_batched(plan: Plan, X, F_batch, batch_rows: int, stream=None, on_batch=None):
    """Stream X through a reused F buffer of ``batch_rows`` rows (row batching
    for feature matrices larger than the caller wants resident).  ``on_batch``
    (optional) is called with (row0, F_view) after each batch is enqueued."""
    n = X.shape[0]
    for r0 in range(0, n, batch_rows):
        nb = min(batch_rows, n - r0)
        Fv = F_batch[:nb]
        plan.transform_into(X[r0:r0 + nb], Fv, stream)
        if on_batch is not None:
            on_batch(r0, Fv)
