"""Python binding of the C ABI in include/ccdpp.h (argument marshalling only).

Every computation happens in libccdpp.so on the GPU.  The module-level
functions carry the C names; the ``CCDPP`` class wraps a handle.  If the
library has not been built, importing works but every call raises.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libccdpp.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "ccdpp.h")

CCDPP_OK, CCDPP_EINVAL, CCDPP_EDUP, CCDPP_ENOMEM, CCDPP_EDEVICE, CCDPP_ESTATE = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "OK", -1: "EINVAL", -2: "EDUP", -3: "ENOMEM", -4: "EDEVICE", -5: "ESTATE"}
K_PASS_FUSED, K_PASS, K_COMBINE, K_COMMIT, K_FLUSH = range(5)
KERNEL_KINDS = {K_PASS_FUSED: "ccd_pass_fused*", K_PASS: "ccd_pass", K_COMBINE: "ccd_combine",
                K_COMMIT: "ccd_copy", K_FLUSH: "ccd_flush"}


class Options(ctypes.Structure):
    """ccdpp_options_t: layout knobs (0 = automatic).  Index 0 is the user-major copy,
    1 the item-major copy.  gather_mode: 1 global memory, 2 LDS-staged, 3 hot.
    cache: 1 streaming, 2 write-back residual stores, 3 cached loads and stores.
    index_coding: 0 delta-coded windows where they fit, 1 plain 16-bit indices."""
    _fields_ = [("gather_mode", ctypes.c_int32 * 2), ("tile_width", ctypes.c_int32 * 2),
                ("workgroups", ctypes.c_int32), ("seg_weight", ctypes.c_int32),
                ("precision", ctypes.c_int32), ("cache", ctypes.c_int32 * 2),
                ("index_coding", ctypes.c_int32 * 2), ("split_rows", ctypes.c_int32)]


def make_options(gather_mode=(0, 0), tile_width=(0, 0), workgroups=0, seg_weight=0,
                 precision=0, cache=(0, 0), index_coding=(0, 0), split_rows=0) -> Options:
    """precision: 0 float32 residual and factors, 1 float64.  split_rows: item-major
    copy split into tiled leading items and hot others (0 automatic, -1 never, n1 > 0
    that many tiled items)."""
    o = Options()
    o.gather_mode[0], o.gather_mode[1] = gather_mode
    o.tile_width[0], o.tile_width[1] = tile_width
    o.workgroups = workgroups
    o.seg_weight = seg_weight
    o.precision = precision
    o.cache[0], o.cache[1] = cache
    o.index_coding[0], o.index_coding[1] = index_coding
    o.split_rows = split_rows
    return o


class CCDPPError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {message}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libccdpp.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_1511_02433_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, i64, i32, u64, dbl = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                 ctypes.c_double)
        sig = {
            "ccdpp_create": ([i64, i64, i32, dbl, i64, P, P, P, u64, ctypes.POINTER(P)], ctypes.c_int),
            "ccdpp_create_ex": ([i64, i64, i32, dbl, i64, P, P, P, u64, ctypes.POINTER(Options),
                                 ctypes.POINTER(P)], ctypes.c_int),
            "ccdpp_run": ([P, i32, i32], ctypes.c_int),
            "ccdpp_ccd_run": ([P, i32], ctypes.c_int),
            "ccdpp_run_until": ([P, i32, i32, dbl, i64, P, P, P, P, ctypes.POINTER(i32)],
                                ctypes.c_int),
            "ccdpp_get_factors": ([P, P, P], ctypes.c_int),
            "ccdpp_get_factors_f64": ([P, P, P], ctypes.c_int),
            "ccdpp_set_factors": ([P, P, P], ctypes.c_int),
            "ccdpp_set_factors_f64": ([P, P, P], ctypes.c_int),
            "ccdpp_rmse": ([P, i64, P, P, P, ctypes.POINTER(dbl)], ctypes.c_int),
            "ccdpp_rmse_noalloc": ([P, i64, P, P, P, ctypes.POINTER(dbl)], ctypes.c_int),
            "ccdpp_train_rmse": ([P, ctypes.POINTER(dbl)], ctypes.c_int),
            "ccdpp_get_residual": ([P, P], ctypes.c_int),
            "ccdpp_get_residual_f64": ([P, P], ctypes.c_int),
            "ccdpp_check_consistency": ([P, ctypes.POINTER(i64)], ctypes.c_int),
            "ccdpp_set_stream": ([P, P], ctypes.c_int),
            "ccdpp_profile": ([P, i32], ctypes.c_int),
            "ccdpp_profile_only": ([P, i32, i32], ctypes.c_int),
            "ccdpp_profile_every": ([P, i32], ctypes.c_int),
            "ccdpp_profile_read": ([P, i32, i32, ctypes.POINTER(i64), ctypes.POINTER(dbl),
                                    ctypes.POINTER(dbl)], ctypes.c_int),
            "ccdpp_info": ([P, ctypes.POINTER(i64), i32], ctypes.c_int),
            "ccdpp_debug_inject": ([i32, i64], ctypes.c_int),
            "ccdpp_last_error": ([P], ctypes.c_char_p),
            "ccdpp_destroy": ([P], None),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def declared_symbols() -> list[str]:
    """Function names declared in include/ccdpp.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(ccdpp_[a-z0-9_]+)\s*\(", text)))


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(h, rc):
    if rc < 0:
        msg = lib().ccdpp_last_error(h)
        raise CCDPPError(rc, msg.decode() if msg else "")
    return rc


# ---- C-named functions ---------------------------------------------------------------
def ccdpp_create(m, n, k, lam, row, col, val, seed=0):
    return ccdpp_create_ex(m, n, k, lam, row, col, val, seed, None)


def ccdpp_create_ex(m, n, k, lam, row, col, val, seed=0, opts=None):
    row = np.ascontiguousarray(row, dtype=np.int32)
    col = np.ascontiguousarray(col, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    if not (row.size == col.size == val.size):
        raise ValueError("row, col and val must have the same length")
    h = ctypes.c_void_p()
    args = (int(m), int(n), int(k), float(lam), int(row.size), _p(row), _p(col), _p(val),
            int(seed) & (2**64 - 1))
    if opts is None:
        rc = lib().ccdpp_create(*args, ctypes.byref(h))
    else:
        rc = lib().ccdpp_create_ex(*args, ctypes.byref(opts), ctypes.byref(h))
    _check(None, rc)
    return h


def ccdpp_run(h, outer_iters, inner_iters):
    _check(h, lib().ccdpp_run(h, int(outer_iters), int(inner_iters)))


def ccdpp_ccd_run(h, outer_iters):
    _check(h, lib().ccdpp_ccd_run(h, int(outer_iters)))


def ccdpp_run_until(h, max_outer, inner_iters, rel_tol, test=None):
    """Returns (outer iterations run, history (that many x 3): objective of eq. 1,
    training RMSE, held-out RMSE or NaN)."""
    if test is None:
        r = c = v = None
        tn = 0
    else:
        r = np.ascontiguousarray(test[0], dtype=np.int32)
        c = np.ascontiguousarray(test[1], dtype=np.int32)
        v = np.ascontiguousarray(test[2], dtype=np.float32)
        if not (r.size == c.size == v.size):
            raise ValueError("test row, col and val must have the same length")
        tn = r.size
    hist = np.zeros((max(int(max_outer), 1), 3))
    done = ctypes.c_int32(0)
    _check(h, lib().ccdpp_run_until(h, int(max_outer), int(inner_iters), float(rel_tol), tn, _p(r),
                                    _p(c), _p(v), _p(hist), ctypes.byref(done)))
    return done.value, hist[:done.value]


def ccdpp_get_factors(h, m, n, k):
    W = np.empty((m, k), dtype=np.float32)
    H = np.empty((n, k), dtype=np.float32)
    _check(h, lib().ccdpp_get_factors(h, _p(W), _p(H)))
    return W, H


def ccdpp_get_factors_f64(h, m, n, k):
    W = np.empty((m, k), dtype=np.float64)
    H = np.empty((n, k), dtype=np.float64)
    _check(h, lib().ccdpp_get_factors_f64(h, _p(W), _p(H)))
    return W, H


def ccdpp_set_factors(h, W=None, H=None):
    W = None if W is None else np.ascontiguousarray(W, dtype=np.float32)
    H = None if H is None else np.ascontiguousarray(H, dtype=np.float32)
    _check(h, lib().ccdpp_set_factors(h, _p(W), _p(H)))


def ccdpp_set_factors_f64(h, W=None, H=None):
    W = None if W is None else np.ascontiguousarray(W, dtype=np.float64)
    H = None if H is None else np.ascontiguousarray(H, dtype=np.float64)
    _check(h, lib().ccdpp_set_factors_f64(h, _p(W), _p(H)))


def ccdpp_rmse(h, row, col, val):
    row = np.ascontiguousarray(row, dtype=np.int32)
    col = np.ascontiguousarray(col, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    out = ctypes.c_double()
    _check(h, lib().ccdpp_rmse(h, int(row.size), _p(row), _p(col), _p(val), ctypes.byref(out)))
    return out.value


def ccdpp_rmse_noalloc(h, nnz, row_ptr, col_ptr, val_ptr):
    """Held-out RMSE from triplets in device memory (device addresses, e.g. torch's
    data_ptr() of int32, int32 and float32 tensors); allocates no device memory."""
    out = ctypes.c_double()
    _check(h, lib().ccdpp_rmse_noalloc(h, int(nnz), ctypes.c_void_p(row_ptr),
                                       ctypes.c_void_p(col_ptr), ctypes.c_void_p(val_ptr),
                                       ctypes.byref(out)))
    return out.value


def ccdpp_train_rmse(h):
    out = ctypes.c_double()
    _check(h, lib().ccdpp_train_rmse(h, ctypes.byref(out)))
    return out.value


def ccdpp_get_residual(h, nnz):
    R = np.empty(nnz, dtype=np.float32)
    _check(h, lib().ccdpp_get_residual(h, _p(R)))
    return R


def ccdpp_get_residual_f64(h, nnz):
    R = np.empty(nnz, dtype=np.float64)
    _check(h, lib().ccdpp_get_residual_f64(h, _p(R)))
    return R


def ccdpp_check_consistency(h):
    out = ctypes.c_int64()
    _check(h, lib().ccdpp_check_consistency(h, ctypes.byref(out)))
    return out.value


def ccdpp_set_stream(h, stream_ptr):
    _check(h, lib().ccdpp_set_stream(h, ctypes.c_void_p(stream_ptr) if stream_ptr else None))


def ccdpp_profile(h, enable):
    _check(h, lib().ccdpp_profile(h, 1 if enable else 0))


def ccdpp_profile_only(h, kind=-1, layout=-1):
    _check(h, lib().ccdpp_profile_only(h, int(kind), int(layout)))


def ccdpp_profile_every(h, every):
    _check(h, lib().ccdpp_profile_every(h, int(every)))


def ccdpp_profile_read(h, kind, layout=-1):
    n, ms, b = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double()
    _check(h, lib().ccdpp_profile_read(h, int(kind), int(layout), ctypes.byref(n),
                                       ctypes.byref(ms), ctypes.byref(b)))
    return n.value, ms.value, b.value


INFO_FIELDS = ("m", "n", "nnz", "k", "build_us", "u_gather", "u_tiles", "u_tile_width",
               "u_workgroups", "u_segments", "v_gather", "v_tiles", "v_tile_width", "v_workgroups",
               "v_segments", "device_bytes", "value_bytes", "u_rows_finished_in_pass",
               "u_rows_combined", "v_rows_finished_in_pass", "v_rows_combined", "u_cache",
               "v_cache", "u_delta_windows", "u_windows", "v_delta_windows", "v_windows",
               "v_split_rows", "v2_gather", "v2_tile_width", "v2_workgroups", "v2_segments",
               "v2_rows_finished_in_pass", "v2_rows_combined", "v2_cache", "build_inputs_us",
               "build_relabel_us", "build_user_major_us", "build_item_major_us", "build_setup_us",
               "build_factors_us", "build_device_setup_us")


def ccdpp_info(h):
    buf = (ctypes.c_int64 * len(INFO_FIELDS))()
    w = _check(h, lib().ccdpp_info(h, buf, len(INFO_FIELDS)))
    return {INFO_FIELDS[i]: int(buf[i]) for i in range(w)}


def ccdpp_debug_inject(what, after):
    """Testing hook of the error paths: what 0 fails the device allocation after
    `after` more, what 1 the sweep launch after `after` more; after < 0 disarms."""
    _check(None, lib().ccdpp_debug_inject(int(what), int(after)))


def ccdpp_last_error(h=None):
    msg = lib().ccdpp_last_error(h)
    return msg.decode() if msg else ""


def ccdpp_destroy(h):
    lib().ccdpp_destroy(h)


# ---- convenience wrapper ---------------------------------------------------------------
class CCDPP:
    """A CCD++ problem held on the current HIP device."""

    def __init__(self, m, n, k, lam, row, col, val, seed=0, opts=None):
        self.m, self.n, self.k, self.lam = int(m), int(n), int(k), float(lam)
        self.nnz = int(np.asarray(row).size)
        self._h = ccdpp_create_ex(m, n, k, lam, row, col, val, seed, opts)

    def close(self):
        if getattr(self, "_h", None):
            ccdpp_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def run(self, outer_iters, inner_iters):
        ccdpp_run(self._h, outer_iters, inner_iters)

    def ccd_run(self, outer_iters):
        """Algorithm 2 (element-wise CCD)."""
        ccdpp_ccd_run(self._h, outer_iters)

    def run_until(self, max_outer, inner_iters, rel_tol, test=None):
        return ccdpp_run_until(self._h, max_outer, inner_iters, rel_tol, test)

    def factors(self):
        return ccdpp_get_factors(self._h, self.m, self.n, self.k)

    def set_factors(self, W=None, H=None):
        ccdpp_set_factors(self._h, W, H)

    def factors_f64(self):
        return ccdpp_get_factors_f64(self._h, self.m, self.n, self.k)

    def set_factors_f64(self, W=None, H=None):
        ccdpp_set_factors_f64(self._h, W, H)

    def residual_f64(self):
        return ccdpp_get_residual_f64(self._h, self.nnz)

    def rmse(self, row, col, val):
        return ccdpp_rmse(self._h, row, col, val)

    def rmse_noalloc(self, nnz, row_ptr, col_ptr, val_ptr):
        return ccdpp_rmse_noalloc(self._h, nnz, row_ptr, col_ptr, val_ptr)

    def train_rmse(self):
        return ccdpp_train_rmse(self._h)

    def residual(self):
        return ccdpp_get_residual(self._h, self.nnz)

    def check_consistency(self):
        return ccdpp_check_consistency(self._h)

    def set_stream(self, stream_ptr):
        ccdpp_set_stream(self._h, stream_ptr)

    def use_torch_stream(self):
        """Run on PyTorch's current HIP stream (PyTorch is used for streams only)."""
        import torch
        self.set_stream(torch.cuda.current_stream().cuda_stream)

    def profile(self, enable=True):
        ccdpp_profile(self._h, enable)

    def profile_only(self, kind=-1, layout=-1):
        ccdpp_profile_only(self._h, kind, layout)

    def profile_every(self, every):
        ccdpp_profile_every(self._h, every)

    def profile_read(self, kind, layout=-1):
        return ccdpp_profile_read(self._h, kind, layout)

    def info(self):
        return ccdpp_info(self._h)
