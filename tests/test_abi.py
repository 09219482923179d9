"""The C ABI without a GPU: the library loads, exports every declared symbol,
generates the same kernels as the oracle's independent generator, and
rejects invalid arguments before touching a device."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2601_17091_amd as rk
from paper_2601_17091_amd import rocket as rb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rocket.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rb.LIB_PATH):
        from paper_2601_17091_amd import build_lib
        build_lib.build()
    return rb.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rocket_[a-z_]+)\s*\(", text)))


def test_header_declares_exported_set(lib):
    assert declared_functions() == sorted(rb.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", rb.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_product_build_is_unchecked(lib):
    v = ctypes.c_uint32(7)
    assert lib.rocket_checked_build() == 0
    assert lib.rocket_check_flags(ctypes.byref(v)) == rb.ROCKET_OK
    assert v.value == 0
    assert lib.rocket_check_flags(None) == rb.ROCKET_ERR_INVALID_ARG


def test_checked_build_exports_the_same_symbols(lib):
    if not os.path.exists(rb.CHECKED_LIB_PATH):
        from paper_2601_17091_amd import build_lib
        build_lib.build()
    out = subprocess.run(["nm", "-D", "--defined-only", rb.CHECKED_LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in declared_functions():
        assert name in exported, name
    with rb.library_at(rb.CHECKED_LIB_PATH) as clib:
        assert clib.rocket_checked_build() == 1
        assert clib.rocket_check_flags(None) == rb.ROCKET_ERR_INVALID_ARG
        assert rk.checked_build()
    assert not rk.checked_build()


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert rk.status_string(code) not in ("", "unknown status")
    assert rk.status_string(7) == "unknown status"


@pytest.mark.parametrize("seed,K,L", [(0, 500, 11), (1, 2000, 64), (203, 3000, 1000),
                                      (2 ** 64 - 1, 1000, 16384), (42, 700, 500)])
def test_generator_matches_oracle_bitwise(lib, oracle, seed, K, L):
    a = rk.generate_kernels(seed, K, L)
    b = oracle.generate_kernels(seed, K, L)
    for key in ("length", "dilation", "padding", "bias", "weights"):
        assert a[key].dtype == b[key].dtype, key
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    assert a["input_length"] == L


def test_generator_errors_and_free(lib):
    ck = rb.CKernels()
    assert lib.rocket_generate_kernels(1, 0, 100, ctypes.byref(ck)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_generate_kernels(1, 10, 10, ctypes.byref(ck)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_generate_kernels(1, 10, 100, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_generate_kernels(1, 10, 100, ctypes.byref(ck)) == rb.ROCKET_OK
    assert ck.n_kernels == 10 and ck.max_len == 11
    lib.rocket_free_kernels(ctypes.byref(ck))
    assert ck.n_kernels == 0 and not ck.length
    lib.rocket_free_kernels(ctypes.byref(ck))  # idempotent
    lib.rocket_free_kernels(None)  # NULL-safe


def _kernels(**over):
    k = dict(length=np.array([7, 9]), dilation=np.array([1, 2]), padding=np.array([0, 8]),
             bias=np.array([0.1, -0.2], np.float32), weights=np.ones((2, 11), np.float32))
    k.update(over)
    return k


def _plan_status(lib, k, L, flags=0):
    c, keep = rb.as_c_kernels(k)
    h = ctypes.c_void_p()
    st = lib.rocket_plan_create_ex(ctypes.byref(c), L, flags, ctypes.byref(h))
    assert not h.value  # every case below fails before a plan exists
    return st


@pytest.mark.parametrize("over,L,expect", [
    (dict(), 0, rb.ROCKET_ERR_INVALID_ARG),
    (dict(length=np.array([0, 9])), 100, rb.ROCKET_ERR_INVALID_ARG),
    (dict(length=np.array([12, 9])), 100, rb.ROCKET_ERR_INVALID_ARG),
    (dict(dilation=np.array([0, 2])), 100, rb.ROCKET_ERR_INVALID_ARG),
    (dict(padding=np.array([-1, 8])), 100, rb.ROCKET_ERR_INVALID_ARG),
    (dict(dilation=np.array([20, 2])), 100, rb.ROCKET_ERR_LENGTH),   # O = 100 - 120 < 1
    (dict(dilation=np.array([2, 2])), 10, rb.ROCKET_ERR_LENGTH),     # length 7, d 2: O = 10 - 12
    (dict(padding=np.array([0, 2 ** 24])), 100, rb.ROCKET_ERR_LENGTH),  # O above 2^24 - 1
])
def test_plan_validation(lib, over, L, expect):
    assert _plan_status(lib, _kernels(**over), L) == expect


def test_plan_validation_null_and_flags(lib):
    h = ctypes.c_void_p()
    assert lib.rocket_plan_create(None, 100, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    k = _kernels()
    c, keep = rb.as_c_kernels(k)
    assert lib.rocket_plan_create(ctypes.byref(c), 100, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_plan_create_ex(ctypes.byref(c), 100, 32, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    for a, b in ((rb.ROCKET_PLAN_DIRECT, rb.ROCKET_PLAN_CLAMPED), (rb.ROCKET_PLAN_DIRECT, rb.ROCKET_PLAN_TILED),
                 (rb.ROCKET_PLAN_SERIES, rb.ROCKET_PLAN_DIRECT), (rb.ROCKET_PLAN_SERIES, rb.ROCKET_PLAN_CLAMPED),
                 (rb.ROCKET_PLAN_SERIES, rb.ROCKET_PLAN_TILED)):
        assert lib.rocket_plan_create_ex(ctypes.byref(c), 100, a | b, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    bad = rb.CKernels(2, 0, 11, c.length, c.dilation, c.padding, c.bias, None)
    assert lib.rocket_plan_create(ctypes.byref(bad), 100, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    bad = rb.CKernels(2, 0, 12, c.length, c.dilation, c.padding, c.bias, c.weights)
    assert lib.rocket_plan_create(ctypes.byref(bad), 100, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    bad = rb.CKernels(0, 0, 11, c.length, c.dilation, c.padding, c.bias, c.weights)
    assert lib.rocket_plan_create(ctypes.byref(bad), 100, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG
    lib.rocket_plan_destroy(None)


def test_transform_validation(lib):
    k = _kernels()
    c, keep = rb.as_c_kernels(k)
    dummy = ctypes.c_void_p(0x1000)
    assert lib.rocket_transform(dummy, -1, 100, ctypes.byref(c), dummy, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_transform(None, 4, 100, ctypes.byref(c), dummy, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_transform(dummy, 4, 100, ctypes.byref(c), None, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_transform(dummy, 4, 100, None, dummy, None) == rb.ROCKET_ERR_INVALID_ARG
    bad = _kernels(dilation=np.array([30, 2]))
    cb, keep2 = rb.as_c_kernels(bad)
    assert lib.rocket_transform(dummy, 4, 100, ctypes.byref(cb), dummy, None) == rb.ROCKET_ERR_LENGTH
    # n == 0 is a no-op that never touches memory
    assert lib.rocket_transform(None, 0, 100, ctypes.byref(c), None, None) == rb.ROCKET_OK
    assert lib.rocket_transform_plan(None, dummy, 1, dummy, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_transform_plan_noalloc(None, dummy, 1, dummy, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_plan_info(None, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_transform_host(None, dummy, 1, dummy, 0, None) == rb.ROCKET_ERR_INVALID_ARG


def test_plan_tables_errors(lib):
    t = rb.CPlanTables()
    assert lib.rocket_plan_tables_build(None, 100, ctypes.byref(t)) == rb.ROCKET_ERR_INVALID_ARG
    c, keep = rb.as_c_kernels(_kernels())
    assert lib.rocket_plan_tables_build(ctypes.byref(c), 100, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_plan_tables_build(ctypes.byref(c), 5, ctypes.byref(t)) == rb.ROCKET_ERR_LENGTH
    assert lib.rocket_plan_tables_build(ctypes.byref(c), 100, ctypes.byref(t)) == rb.ROCKET_OK
    assert t.n_items == 2
    lib.rocket_plan_tables_free(ctypes.byref(t))
    lib.rocket_plan_tables_free(ctypes.byref(t))
    lib.rocket_plan_tables_free(None)


@pytest.mark.parametrize("n,L,nf,seed", [(5, 9, 10000, 0), (7, 17, 10000, 1), (40, 300, 5000, 2),
                                         (30, 1000, 10000, 3), (3, 64, 10000, 2 ** 64 - 1)])
def test_minirocket_fit_matches_oracle_bitwise(lib, oracle, n, L, nf, seed):
    from oracle import minirocket_oracle as mo
    rng = np.random.default_rng(seed % 1000)
    X = rng.standard_normal((n, L)).cumsum(axis=1).astype(np.float32)
    a = rk.minirocket_fit(X, nf, seed)
    b = mo.fit(X, nf, seed)
    assert a["input_length"] == L
    for key in ("dilations", "features_per_dilation", "biases"):
        assert a[key].dtype == b[key].dtype, key
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)


def test_minirocket_fit_errors_and_free(lib):
    cp = rb.CMiniRocketParams()
    X = np.zeros((2, 20), np.float32)
    xp = X.ctypes.data_as(ctypes.c_void_p)
    assert lib.rocket_minirocket_fit(None, 2, 20, 100, 0, ctypes.byref(cp)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_minirocket_fit(xp, 0, 20, 100, 0, ctypes.byref(cp)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_minirocket_fit(xp, 2, 8, 100, 0, ctypes.byref(cp)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_minirocket_fit(xp, 2, 20, 83, 0, ctypes.byref(cp)) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_minirocket_fit(xp, 2, 20, 100, 0, None) == rb.ROCKET_ERR_INVALID_ARG
    assert lib.rocket_minirocket_fit(xp, 2, 20, 100, 0, ctypes.byref(cp)) == rb.ROCKET_OK
    assert cp.n_features == 84 and cp.n_dilations == 1 and cp.input_length == 20
    lib.rocket_minirocket_free(ctypes.byref(cp))
    assert cp.n_features == 0 and not cp.biases
    lib.rocket_minirocket_free(ctypes.byref(cp))  # idempotent
    lib.rocket_minirocket_free(None)              # NULL-safe


def test_minirocket_plan_rejects_bad_params_before_the_device(lib):
    """Validation happens before any device call, so these run without a GPU."""
    good = dict(input_length=100, dilations=np.array([1, 3], np.int32),
                features_per_dilation=np.array([1, 2], np.int32), biases=np.zeros(84 * 3, np.float32))

    def status(params, flags=0):
        c, keep = rb.as_c_minirocket(params)
        h = ctypes.c_void_p()
        r = lib.rocket_minirocket_plan_create(ctypes.byref(c), flags, ctypes.byref(h))
        del keep
        return r

    bad = [
        (dict(good, biases=np.zeros(84 * 3 - 1, np.float32)), rb.ROCKET_ERR_INVALID_ARG),  # count mismatch
        (dict(good, dilations=np.array([3, 1], np.int32)), rb.ROCKET_ERR_INVALID_ARG),     # not ascending
        (dict(good, dilations=np.array([0, 3], np.int32)), rb.ROCKET_ERR_INVALID_ARG),
        (dict(good, features_per_dilation=np.array([-1, 4], np.int32)), rb.ROCKET_ERR_INVALID_ARG),
        (dict(good, input_length=8), rb.ROCKET_ERR_INVALID_ARG),
        (dict(good, dilations=np.array([1, 13], np.int32)), rb.ROCKET_ERR_LENGTH),         # 100 - 8*13 < 1
    ]
    for params, want in bad:
        assert status(params) == want, (params, want)
    assert status(good, rb.ROCKET_PLAN_MPV) == rb.ROCKET_ERR_INVALID_ARG
    assert status(good, rb.ROCKET_PLAN_DIRECT) == rb.ROCKET_ERR_INVALID_ARG
    h = ctypes.c_void_p()
    assert lib.rocket_minirocket_plan_create(None, 0, ctypes.byref(h)) == rb.ROCKET_ERR_INVALID_ARG


def _overcommit_mode():
    try:
        return int(open("/proc/sys/vm/overcommit_memory").read().strip())
    except (OSError, ValueError):
        return None


def test_generator_reports_oom(lib):
    """An absurd kernel set (2^31 - 1 multivariate kernels of 32 channels:
    2.75 TiB of weights) cannot be allocated: the generator returns
    ROCKET_ERR_OOM and leaves the output zeroed.  Nothing is touched before
    the allocation fails, so no memory is used."""
    if _overcommit_mode() == 1:
        pytest.skip("the kernel always overcommits memory here: an absurd request would not fail")
    k = rb.CKernels()
    rc = lib.rocket_generate_kernels_multi(ctypes.c_uint64(1), 2 ** 31 - 1, 1000, 32, ctypes.byref(k))
    assert rc == rb.ROCKET_ERR_OOM
    assert k.n_kernels == 0 and not k.weights and not k.length
    lib.rocket_free_kernels(ctypes.byref(k))
