"""GPU path against the fp64 oracle at the benchmark workloads' full sizes.

Every matrix here is the full synthetic workload, created with the default
layout options, which is the configuration bench.py times.  The oracle runs the
same iterations on the host (OpenMP), so W, H and the RMSEs are compared in
full rather than on samples.  For every workload one GPU handle and one oracle
run side by side:

* after the first outer iteration, W and H within 1e-3 (per-feature scaled max
  relative error);
* both then continue, without starting over, to the workload's full schedule,
  after which train and test RMSE agree within 1e-4;
* the two residual copies agree bit for bit.

Workloads: medium (10 x 3), large (10 x 3), the rank sweep on the large matrix
(k = 10 and k = 100, 5 x 3; k = 40 is the large workload's own k) and the very
large matrix (5 x 3, lambda = 1), whose item-major copy is split (its leading
items tiled, the others a hot layout) and whose user-major copy is tiled, so
that its combine covers every row.  Each
test prints what it runs before it starts, and keeps to about two minutes: the
very large workload is split into drawing the matrix, the first outer
iteration and the rest of the schedule.
"""
import os
import time

import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

W_TOL = 1e-3
RMSE_TOL = 1e-4
THREADS = min(16, os.cpu_count() or 1)


def _say(msg):
    print(f"[fullsize] {msg}", flush=True)


# The automatic cache policy of the two copies (1 streaming, 2 write-back residual
# stores, 3 cached): medium's residual streams fit in the memory-side cache; large
# takes write-back stores on its one-tile user-major copy; the very large matrix has
# no one-tile copy.  The gather mode of each copy (2 tiled, 3 hot), and whether the
# item-major copy is split into tiled leading items and a hot rest: the very large
# matrix's is (its hot part streams too).
EXPECT_CACHE = {"medium": (3, 3), "large": (1, 2), "vlarge": (1, 1)}
EXPECT_GATHER = {"medium": (2, 2), "large": (2, 2), "vlarge": (2, 2)}
EXPECT_SPLIT = {"medium": False, "large": False, "vlarge": True}


class Side:
    """One GPU handle and one oracle on the same workload, the same k and H0."""

    def __init__(self, ds, k):
        w = ds.workload
        self.ds, self.k, self.w = ds, k, w
        self.g = CCDPP(w.m, w.n, k, w.lam, ds.row, ds.col, ds.val)
        info = self.g.info()
        _say(f"{w.name} k={k}: layout "
             f"{({key: v for key, v in info.items() if key.startswith(('u_', 'v_'))})}")
        if w.name in EXPECT_CACHE:
            assert (info["u_cache"], info["v_cache"]) == EXPECT_CACHE[w.name]
            assert (info["u_gather"], info["v_gather"]) == EXPECT_GATHER[w.name]
            assert (info["v_split_rows"] > 0) == EXPECT_SPLIT[w.name]
            if EXPECT_SPLIT[w.name]:
                assert info["v2_gather"] == 3 and info["v2_cache"] == 1
        h0 = ds.h0(k)
        self.g.set_factors(np.zeros((w.m, k), np.float32), h0)
        t0 = time.perf_counter()
        self.o = Oracle(w.m, w.n, k, w.lam, ds.row, ds.col, ds.val, h0, threads=THREADS)
        _say(f"{w.name} k={k}: oracle built in {time.perf_counter() - t0:.1f} s")
        self.outer = 0

    def first_outer(self):
        w = self.w
        t0 = time.perf_counter()
        self.g.run(1, w.inner)
        Wg, Hg = self.g.factors()
        t1 = time.perf_counter()
        self.o.run(1, w.inner)
        Wo, Ho = self.o.factors()
        self.outer = 1
        ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
        _say(f"{w.name} k={self.k}: one outer iteration x {w.inner} inner; gpu {t1 - t0:.1f} s, "
             f"oracle {time.perf_counter() - t1:.1f} s; W err {ew:.2e}, H err {eh:.2e}")
        assert ew <= W_TOL and eh <= W_TOL

    def rest(self, outer):
        w, ds = self.w, self.ds
        more = outer - self.outer
        t0 = time.perf_counter()
        self.g.run(more, w.inner)
        tr_g = self.g.train_rmse()
        te_g = self.g.rmse(ds.test_row, ds.test_col, ds.test_val) if ds.test_row.size else None
        assert self.g.check_consistency() == 0
        t1 = time.perf_counter()
        self.o.run(more, w.inner)
        tr_o = self.o.train_rmse()
        te_o = self.o.test_rmse(ds.test_row, ds.test_col, ds.test_val) if ds.test_row.size else None
        self.outer = outer
        _say(f"{w.name} k={self.k}: {outer} x {w.inner} in all; gpu {t1 - t0:.1f} s, oracle "
             f"{time.perf_counter() - t1:.1f} s; train RMSE gpu {tr_g:.8f} oracle {tr_o:.8f} "
             f"(|d| {abs(tr_g - tr_o):.2e}); test RMSE gpu {te_g} oracle {te_o}")
        assert abs(tr_g - tr_o) <= RMSE_TOL
        if te_g is not None:
            assert abs(te_g - te_o) <= RMSE_TOL

    def close(self):
        self.g.close()
        self.o.close()


def _whole(name, k=None, outer=None):
    ds = synth.load(name)
    w = ds.workload
    k = k or w.k
    outer = outer or w.outer
    _say(f"{name}: {w.m} x {w.n}, nnz {w.nnz}, k {k}, {outer} x {w.inner}")
    s = Side(ds, k)
    try:
        s.first_outer()
        s.rest(outer)
    finally:
        s.close()


@pytest.mark.timeout(600)
def test_medium():
    _whole("medium")


@pytest.mark.timeout(900)
def test_large():
    _whole("large")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("k", [10, 100])
def test_rank_sweep(k):
    # The rank sweep's schedule: 5 outer x 3 inner on the large matrix.
    _whole("large", k=k, outer=5)


# The very large matrix, in three steps that share one drawn matrix, one handle and
# one oracle.
_VL = {}


@pytest.mark.timeout(900)
def test_vlarge_draw():
    t0 = time.perf_counter()
    ds = synth.load("vlarge", verbose=True)
    _say(f"vlarge: matrix ready in {time.perf_counter() - t0:.1f} s")
    assert ds.row.size == ds.workload.nnz
    _VL["ds"] = ds


@pytest.mark.timeout(900)
def test_vlarge_one_outer():
    if "ds" not in _VL:
        pytest.skip("the very large matrix was not drawn")
    _VL["side"] = s = Side(_VL.pop("ds"), synth.WORKLOADS["vlarge"].k)
    s.first_outer()


@pytest.mark.timeout(900)
def test_vlarge_full_run():
    s = _VL.pop("side", None)
    if s is None:
        pytest.skip("the first outer iteration did not run")
    try:
        s.rest(s.w.outer)
    finally:
        s.close()
