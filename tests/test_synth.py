"""The seeded generators: exact sizes, distinct positions, disjoint holdout, determinism."""
import numpy as np

from paper_1511_02433_amd import synth


def _check(ds):
    w = ds.workload
    assert ds.row.size == w.nnz == ds.col.size == ds.val.size
    assert ds.test_row.size == w.holdout
    assert ds.row.dtype == np.int32 and ds.col.dtype == np.int32 and ds.val.dtype == np.float32
    assert ds.row.min() >= 0 and ds.row.max() < w.m and ds.col.min() >= 0 and ds.col.max() < w.n
    keys = ds.row.astype(np.int64) * w.n + ds.col
    assert np.unique(keys).size == keys.size
    if w.holdout:
        tkeys = ds.test_row.astype(np.int64) * w.n + ds.test_col
        assert np.unique(tkeys).size == tkeys.size
        assert np.intersect1d(keys, tkeys).size == 0
    assert ds.H0.shape == (w.n, w.k) and ds.H0.dtype == np.float32
    assert np.all(np.isfinite(ds.val))


def test_tiny_shape_and_determinism():
    a = synth.generate("tiny")
    b = synth.generate("tiny")
    _check(a)
    for f in ("row", "col", "val", "test_row", "H0"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    # N(0, 0.01) initial H: standard deviation 0.1.
    assert abs(a.H0.std() - 0.1) < 0.005


def test_medium_powerlaw_shape():
    ds = synth.generate("medium")
    _check(ds)
    w = ds.workload
    rd = np.bincount(ds.row, minlength=w.m)
    assert rd.min() >= 20                       # users clamped to at least 20 ratings
    assert rd.max() > 50 * np.median(rd)        # heavy tail
    assert set(np.unique(ds.val * 2).astype(int)) <= set(range(1, 11))  # half stars 0.5..5


def test_rank_curve_exact_total():
    d = synth.rank_curve(1000, 123_457, 1.1, 3, 5000)
    assert d.sum() == 123_457 and d.min() >= 3 and d.max() <= 5000
    assert np.all(np.diff(d) <= 0)


def test_lengths_problem():
    lens = [0, 1, 5, 64, 65, 300]
    row, col, val, H0 = synth.lengths_problem(lens, 400, 2, seed=1)
    assert np.array_equal(np.bincount(row, minlength=len(lens)), lens)
