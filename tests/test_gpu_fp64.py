"""The float64 variant of the sweep (options.precision = 1: residual, factors and
all arithmetic in double, the paper's double version) against the fp64 oracle.

Both sides compute in double and differ only in summation order, so the
tolerances are far tighter than for the float32 path: W and H within 1e-9
(per-feature scaled max relative error) after one outer iteration, RMSE within
1e-9 after a full run, the residual within 1e-9 of the oracle's.
"""
import os

import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP, make_options
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

W_TOL = 1e-9
RMSE_TOL = 1e-9


def _opts(**kw):
    return make_options(precision=1, **kw)


def _pair(m, n, k, lam, row, col, val, H0, opts=None, threads=16):
    g = CCDPP(m, n, k, lam, row, col, val, opts=opts or _opts())
    assert g.info()["value_bytes"] == 8
    g.set_factors_f64(np.zeros((m, k)), np.asarray(H0, np.float64))
    o = Oracle(m, n, k, lam, row, col, val, H0, threads=threads)
    return g, o


def _errs(g, o):
    Wg, Hg = g.factors_f64()
    Wo, Ho = o.factors()
    return colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)


def test_tiny_one_outer_full_run_and_residual():
    ds = synth.load("tiny")
    w = ds.workload
    print(f"case: fp64 tiny {w.describe()}", flush=True)
    g, o = _pair(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, ds.H0)
    g.run(1, w.inner)
    o.run(1, w.inner)
    ew, eh = _errs(g, o)
    print(f"fp64 tiny after 1 outer: W err {ew:.3e}  H err {eh:.3e}")
    assert ew <= W_TOL and eh <= W_TOL
    g.run(w.outer - 1, w.inner)
    o.run(w.outer - 1, w.inner)
    tr_g, tr_o = g.train_rmse(), o.train_rmse()
    te_g = g.rmse(ds.test_row, ds.test_col, ds.test_val)
    te_o = o.test_rmse(ds.test_row, ds.test_col, ds.test_val)
    print(f"fp64 tiny full run: train {tr_g:.12f} vs {tr_o:.12f}; test {te_g:.12f} vs {te_o:.12f}")
    assert abs(tr_g - tr_o) <= RMSE_TOL and abs(te_g - te_o) <= RMSE_TOL
    R = g.residual_f64()
    Ro = o.residual()
    assert np.max(np.abs(R - Ro)) <= 1e-9 * np.abs(ds.val).max()
    assert g.check_consistency() == 0
    # Far closer to the oracle than the float32 path.
    g32 = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val)
    g32.set_factors(np.zeros((w.m, w.k), np.float32), ds.H0)
    g32.run(w.outer, w.inner)
    assert abs(g32.train_rmse() - tr_o) > 10 * abs(tr_g - tr_o)


def test_factors_roundtrip_and_rebuild():
    ds = synth.load("tiny")
    w = ds.workload
    g = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, opts=_opts())
    rng = np.random.default_rng(7)
    W = rng.standard_normal((w.m, w.k)) * 0.3
    H = rng.standard_normal((w.n, w.k)) * 0.3
    g.set_factors_f64(W, H)
    Wg, Hg = g.factors_f64()
    assert np.array_equal(Wg, W) and np.array_equal(Hg, H)
    pred = np.einsum("ij,ij->i", W[ds.row], H[ds.col])
    np.testing.assert_allclose(g.residual_f64(), ds.val.astype(np.float64) - pred, rtol=0,
                               atol=1e-12)
    assert g.check_consistency() == 0


LAYOUTS = {
    "global": dict(gather_mode=(1, 1)),
    "tiled": dict(gather_mode=(2, 2), tile_width=(192, 128)),
    "tiled_odd": dict(gather_mode=(2, 2), tile_width=(100, 333), workgroups=3),
    "hot": dict(gather_mode=(3, 3), tile_width=(64, 96)),
}


@pytest.mark.parametrize("name", list(LAYOUTS))
def test_layout_strategies(name):
    lens = [850, 700, 300, 40] + list(np.random.default_rng(31).integers(0, 80, 1496))
    row, col, val, H0 = synth.lengths_problem(lens, 900, 4, seed=32)
    print(f"case: fp64 layout {name} nnz={row.size}", flush=True)
    g, o = _pair(1500, 900, 4, 0.1, row, col, val, H0, opts=_opts(**LAYOUTS[name]))
    g.run(1, 2)
    o.run(1, 2)
    ew, eh = _errs(g, o)
    print(f"W err {ew:.3e}  H err {eh:.3e}")
    assert ew <= W_TOL and eh <= W_TOL
    assert g.check_consistency() == 0


@pytest.mark.parametrize("transpose", [False, True])
def test_short_segments_and_32bit_indices(transpose):
    lens = list(np.random.default_rng(51).integers(1, 9, 6000))
    row, col, val, H0 = synth.lengths_problem(lens, 40_000, 3, seed=52)
    m, n = len(lens), 40_000
    if transpose:
        row, col = col, row
        m, n = n, m
        H0 = (np.random.default_rng(53).standard_normal((n, 3)) * 0.1).astype(np.float32)
    for opts in (_opts(), _opts(gather_mode=(1, 1)), _opts(gather_mode=(3, 3), tile_width=(4096, 4096))):
        g, o = _pair(m, n, 3, 0.1, row, col, val, H0, opts=opts)
        g.run(1, 2)
        o.run(1, 2)
        ew, eh = _errs(g, o)
        print(f"fp64 short segments transpose={transpose}: W err {ew:.3e}  H err {eh:.3e}")
        assert ew <= W_TOL and eh <= W_TOL
        assert g.check_consistency() == 0


def test_determinism():
    ds = synth.load("tiny")
    w = ds.workload
    res = []
    for split in (False, True):
        g = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, opts=_opts())
        g.set_factors_f64(np.zeros((w.m, w.k)), ds.H0.astype(np.float64))
        if split:
            g.run(1, 3)
            g.run(1, 3)
        else:
            g.run(2, 3)
        res.append(g.factors_f64())
    assert all(np.array_equal(a, b) for a, b in zip(*res))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["medium", "large"])
def test_full_size_one_outer(name):
    ds = synth.load(name)
    w = ds.workload
    print(f"case: fp64 {name} {w.m} x {w.n}, nnz {w.nnz}, one outer iteration", flush=True)
    g, o = _pair(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, ds.h0(w.k))
    g.run(1, w.inner)
    o.run(1, w.inner)
    ew, eh = _errs(g, o)
    print(f"fp64 {name}: W err {ew:.3e}  H err {eh:.3e}; train RMSE {g.train_rmse():.12f} vs "
          f"{o.train_rmse():.12f}")
    assert ew <= W_TOL and eh <= W_TOL
    assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    assert g.check_consistency() == 0
    if name == "medium":  # on to the full schedule
        g.run(w.outer - 1, w.inner)
        o.run(w.outer - 1, w.inner)
        print(f"fp64 {name} after {w.outer} x {w.inner}: train RMSE {g.train_rmse():.12f} vs "
              f"{o.train_rmse():.12f}")
        assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
        assert g.check_consistency() == 0
