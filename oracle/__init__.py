"""ctypes binding of the CPU CCD++ oracle (plain fp64 C, Algorithm 3 of the paper).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only users.  The GPU library never imports this
package and this package imports nothing from the GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ccdpp_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle_ccdpp.so")


def build(quiet: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", LIB_PATH + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True, capture_output=quiet)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i64, i32, dbl = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        L.oracle_create.restype = P
        L.oracle_create.argtypes = [i64, i64, i32, dbl, i64, P, P, P, P, P]
        L.oracle_destroy.argtypes = [P]
        L.oracle_set_threads.argtypes = [P, i32]
        L.oracle_set_from_scratch.argtypes = [P, i32]
        L.oracle_run.argtypes = [P, i32, i32, P]
        L.oracle_rank.argtypes = [P, i32, i32, P, P, P, P]
        L.oracle_ccd_run.argtypes = [P, i32]
        L.oracle_get_factors.argtypes = [P, P, P]
        L.oracle_get_residual.argtypes = [P, P]
        L.oracle_objective.restype = dbl
        L.oracle_objective.argtypes = [P]
        L.oracle_train_rmse.restype = dbl
        L.oracle_train_rmse.argtypes = [P]
        L.oracle_test_rmse.restype = dbl
        L.oracle_test_rmse.argtypes = [P, i64, P, P, P]
        L.oracle_run_until.restype = ctypes.c_int32
        L.oracle_run_until.argtypes = [P, i32, i32, ctypes.c_double, i64, P, P, P, P]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """Double-precision CCD++ on the CPU.  W and H are row-major (m x k, n x k)."""

    def __init__(self, m, n, k, lam, row, col, val, H0, W0=None, threads=0):
        self.m, self.n, self.k, self.lam = int(m), int(n), int(k), float(lam)
        self._row = np.ascontiguousarray(row, dtype=np.int32)
        self._col = np.ascontiguousarray(col, dtype=np.int32)
        a = np.ascontiguousarray(val, dtype=np.float64)
        H0 = np.ascontiguousarray(H0, dtype=np.float64).reshape(self.n, self.k)
        W0 = None if W0 is None else np.ascontiguousarray(W0, dtype=np.float64).reshape(self.m, self.k)
        self.nnz = self._row.size
        self._h = lib().oracle_create(self.m, self.n, self.k, self.lam, self.nnz, _ptr(self._row),
                                      _ptr(self._col), _ptr(a), _ptr(W0), _ptr(H0))
        if not self._h:
            raise ValueError("oracle_create rejected the input (range, duplicates or sizes)")
        lib().oracle_set_threads(self._h, int(threads))

    def close(self):
        if getattr(self, "_h", None):
            lib().oracle_destroy(self._h)
            self._h = None

    __del__ = close

    def set_threads(self, threads: int):
        lib().oracle_set_threads(self._h, int(threads))

    def set_from_scratch(self, on: bool):
        lib().oracle_set_from_scratch(self._h, 1 if on else 0)

    def run(self, outer: int, inner: int, trace: bool = False):
        tr = np.zeros(outer * self.k * (1 + 2 * inner)) if trace else None
        rc = lib().oracle_run(self._h, int(outer), int(inner), _ptr(tr))
        if rc:
            raise ValueError("oracle_run: bad arguments")
        return tr

    def rank(self, t: int, inner: int, debug: bool = True):
        """One rank update; returns (trace, rhat in input order, u history, v history),
        or None when debug is False (no side outputs are produced)."""
        if not debug:
            if lib().oracle_rank(self._h, int(t), int(inner), None, None, None, None):
                raise ValueError("oracle_rank: bad arguments")
            return None
        tr = np.zeros(1 + 2 * inner)
        rh = np.zeros(self.nnz)
        uh = np.zeros((inner, self.m))
        vh = np.zeros((inner, self.n))
        rc = lib().oracle_rank(self._h, int(t), int(inner), _ptr(tr), _ptr(rh), _ptr(uh), _ptr(vh))
        if rc:
            raise ValueError("oracle_rank: bad arguments")
        return tr, rh, uh, vh

    def run_until(self, max_outer: int, inner: int, rel_tol: float, test=None):
        """Algorithm 3 with its outer loop open (see oracle_run_until).  Returns (number
        of outer iterations run, history array of shape (that number, 3): objective,
        train RMSE, test RMSE (NaN without a test set))."""
        if test is None:
            r = c = a = None
            tn = 0
        else:
            r = np.ascontiguousarray(test[0], dtype=np.int32)
            c = np.ascontiguousarray(test[1], dtype=np.int32)
            a = np.ascontiguousarray(test[2], dtype=np.float64)
            tn = r.size
        hist = np.zeros((max(int(max_outer), 1), 3))
        done = lib().oracle_run_until(self._h, int(max_outer), int(inner), float(rel_tol), tn,
                                      _ptr(r), _ptr(c), _ptr(a), _ptr(hist))
        if done < 0:
            raise ValueError("oracle_run_until: bad arguments")
        return done, hist[:done]

    def ccd_run(self, outer: int):
        if lib().oracle_ccd_run(self._h, int(outer)):
            raise ValueError("oracle_ccd_run: bad arguments")

    def factors(self):
        W = np.zeros((self.m, self.k))
        H = np.zeros((self.n, self.k))
        lib().oracle_get_factors(self._h, _ptr(W), _ptr(H))
        return W, H

    def residual(self):
        R = np.zeros(self.nnz)
        lib().oracle_get_residual(self._h, _ptr(R))
        return R

    def objective(self) -> float:
        return lib().oracle_objective(self._h)

    def train_rmse(self) -> float:
        return lib().oracle_train_rmse(self._h)

    def test_rmse(self, row, col, val) -> float:
        r = np.ascontiguousarray(row, dtype=np.int32)
        c = np.ascontiguousarray(col, dtype=np.int32)
        a = np.ascontiguousarray(val, dtype=np.float64)
        return lib().oracle_test_rmse(self._h, r.size, _ptr(r), _ptr(c), _ptr(a))
