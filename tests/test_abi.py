"""The C ABI without a GPU: the library loads, exports every function that
include/ccdpp.h declares, and rejects bad arguments on the host, before any
HIP call, with the documented status codes."""
import ctypes

import numpy as np
import pytest

import paper_1511_02433_amd.ccdpp as C


def _lib_or_skip():
    try:
        return C.lib()
    except RuntimeError as e:  # not built in this checkout
        pytest.skip(str(e))


def test_every_declared_function_is_exported():
    L = _lib_or_skip()
    names = C.declared_symbols()
    assert len(names) >= 15
    assert "ccdpp_get_factors_f64" in names and "ccdpp_debug_inject" in names
    for name in names:
        assert hasattr(L, name), name
    # and the binding knows a signature for each of them
    for name in names:
        assert getattr(L, name).argtypes is not None or name == "ccdpp_destroy", name


def _create(m=10, n=8, k=2, lam=0.1, row=(0, 1), col=(0, 1), val=(1.0, 2.0), opts=None):
    return C.ccdpp_create_ex(m, n, k, lam, np.array(row, np.int32), np.array(col, np.int32),
                             np.array(val, np.float32), 0, opts)


@pytest.mark.parametrize("kw, msg", [
    (dict(m=0), "m and n"),
    (dict(n=0), "m and n"),
    (dict(m=1 << 30), "m and n"),
    (dict(m=1 << 28), "m and n"),
    (dict(n=1 << 28), "m and n"),
    (dict(k=0), "k must be"),
    (dict(lam=-1.0), "lambda"),
    (dict(lam=float("nan")), "lambda"),
    (dict(row=(0, 10)), "out of range"),
    (dict(col=(0, -1)), "out of range"),
    (dict(val=(1.0, float("inf"))), "not finite"),
])
def test_create_rejects_bad_arguments_on_the_host(kw, msg):
    _lib_or_skip()
    with pytest.raises(C.CCDPPError) as ei:
        _create(**kw)
    assert ei.value.code == C.CCDPP_EINVAL
    assert msg in str(ei.value)


@pytest.mark.parametrize("kw, msg", [
    (dict(gather_mode=(7, 0)), "gather_mode"),
    (dict(gather_mode=(0, 4)), "gather_mode"),
    (dict(gather_mode=(3, 0), tile_width=(100, 0)), "multiple of 32"),
    (dict(tile_width=(0, -1)), "tile_width"),
    (dict(precision=2), "precision"),
    (dict(cache=(4, 0)), "cache"),
    (dict(cache=(0, -1)), "cache"),
    (dict(index_coding=(2, 0)), "index_coding"),
    (dict(split_rows=-2), "split_rows"),
    (dict(split_rows=8), "split_rows"),  # n = 8 in _create
    (dict(split_rows=3, gather_mode=(0, 2)), "split_rows"),
])
def test_create_rejects_bad_options(kw, msg):
    _lib_or_skip()
    with pytest.raises(C.CCDPPError) as ei:
        _create(opts=C.make_options(**kw))
    assert ei.value.code == C.CCDPP_EINVAL
    assert msg in str(ei.value)


def test_null_pointers_and_handles():
    L = _lib_or_skip()
    out = ctypes.c_void_p()
    # NULL out-parameter
    rc = L.ccdpp_create(4, 4, 1, 0.1, 0, None, None, None, 0, None)
    assert rc == C.CCDPP_EINVAL
    assert L.ccdpp_last_error(None)  # the failed create left a message
    # nnz > 0 with NULL arrays
    rc = L.ccdpp_create(4, 4, 1, 0.1, 3, None, None, None, 0, ctypes.byref(out))
    assert rc == C.CCDPP_EINVAL
    # every call on a NULL handle answers ESTATE; destroy accepts NULL
    assert L.ccdpp_run(None, 1, 1) == C.CCDPP_ESTATE
    assert L.ccdpp_ccd_run(None, 1) == C.CCDPP_ESTATE
    done = ctypes.c_int32()
    assert L.ccdpp_run_until(None, 1, 1, 0.0, 0, None, None, None, None,
                             ctypes.byref(done)) == C.CCDPP_ESTATE
    assert L.ccdpp_get_factors(None, None, None) == C.CCDPP_ESTATE
    assert L.ccdpp_set_factors(None, None, None) == C.CCDPP_ESTATE
    assert L.ccdpp_train_rmse(None, None) == C.CCDPP_ESTATE
    assert L.ccdpp_check_consistency(None, None) == C.CCDPP_ESTATE
    assert L.ccdpp_profile(None, 1) == C.CCDPP_ESTATE
    assert L.ccdpp_profile_only(None, 0, 0) == C.CCDPP_ESTATE
    assert L.ccdpp_profile_every(None, 4) == C.CCDPP_ESTATE
    buf = (ctypes.c_int64 * 4)()
    assert L.ccdpp_info(None, buf, 4) == C.CCDPP_ESTATE
    L.ccdpp_destroy(None)


def test_debug_inject_arguments():
    L = _lib_or_skip()
    assert L.ccdpp_debug_inject(2, 0) == C.CCDPP_EINVAL
    for what in (0, 1):
        assert L.ccdpp_debug_inject(what, 5) == C.CCDPP_OK
        assert L.ccdpp_debug_inject(what, -1) == C.CCDPP_OK  # disarmed again


def test_without_a_device_create_reports_edevice():
    """On a machine without a GPU, a valid problem fails with EDEVICE (no fallback)."""
    _lib_or_skip()
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(C.CCDPPError) as ei:
        _create()
    assert ei.value.code == C.CCDPP_EDEVICE


def test_create_reports_the_first_bad_triplet():
    """Triplets are checked by several host threads over contiguous ranges; the error
    still names the first bad one in input order."""
    _lib_or_skip()
    nnz = 200_003
    row = np.arange(nnz, dtype=np.int32) % 97
    col = np.arange(nnz, dtype=np.int32) % 89
    val = np.ones(nnz, np.float32)
    val[190_000] = np.nan
    col[150_001] = 89
    row[120_000] = -3
    with pytest.raises(C.CCDPPError) as ei:
        C.ccdpp_create_ex(97, 89, 2, 0.1, row, col, val, 0, None)
    assert ei.value.code == C.CCDPP_EINVAL
    assert "row[120000] = -3 out of range" in str(ei.value)
    row[120_000] = 0
    with pytest.raises(C.CCDPPError) as ei:
        C.ccdpp_create_ex(97, 89, 2, 0.1, row, col, val, 0, None)
    assert "col[150001] = 89 out of range" in str(ei.value)
    col[150_001] = 0
    with pytest.raises(C.CCDPPError) as ei:
        C.ccdpp_create_ex(97, 89, 2, 0.1, row, col, val, 0, None)
    assert "val[190000] is not finite" in str(ei.value)


def test_every_handle_call_answers_estate_on_a_null_handle():
    """Every exported call that takes a handle refuses a NULL one with ESTATE before
    touching any other argument (destroy accepts NULL)."""
    L = _lib_or_skip()
    skip = {"ccdpp_create", "ccdpp_create_ex", "ccdpp_destroy", "ccdpp_last_error",
            "ccdpp_debug_inject"}
    checked = 0
    for name in C.declared_symbols():
        if name in skip:
            continue
        fn = getattr(L, name)
        args = []
        for t in fn.argtypes:
            args.append(None if t in (ctypes.c_void_p,) or hasattr(t, "contents") or
                        t is ctypes.c_char_p else t(0))
        assert fn(*args) == C.CCDPP_ESTATE, name
        checked += 1
    assert checked >= 18
