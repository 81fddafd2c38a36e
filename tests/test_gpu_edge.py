"""Degenerate and boundary shapes on the GPU against the fp64 oracle: an empty
matrix, one entry, one dense row or column, rows that end exactly at window and
chunk boundaries, one feature with one inner iteration, and the 16/32-bit index
boundary of layouts that gather from global memory."""
import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP, CCDPPError, make_options, CCDPP_EINVAL
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

W_TOL = 1e-3
RMSE_TOL = 1e-4


def _compare(m, n, k, lam, row, col, val, H0, outer, inner, opts=None):
    g = CCDPP(m, n, k, lam, row, col, val, opts=opts)
    g.set_factors(np.zeros((m, k), np.float32), H0)
    o = Oracle(m, n, k, lam, row, col, val, H0)
    g.run(1, inner)
    o.run(1, inner)
    Wg, Hg = g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
    print(f"W err {ew:.3e}  H err {eh:.3e}", flush=True)
    assert ew <= W_TOL and eh <= W_TOL
    if outer > 1:
        g.run(outer - 1, inner)
        o.run(outer - 1, inner)
        assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    assert g.check_consistency() == 0
    return g


@pytest.mark.parametrize("lam", [0.1, 0.0])
def test_empty_matrix(lam):
    # No observed entries: every coordinate is 0/lambda = 0 (reading A-6 for lambda = 0),
    # the training RMSE is undefined, and a held-out RMSE measures the zero prediction.
    print(f"case: empty matrix lambda={lam}", flush=True)
    e = np.zeros(0, np.int32)
    g = CCDPP(50, 40, 3, lam, e, e, np.zeros(0, np.float32))
    H0 = (np.random.default_rng(1).standard_normal((40, 3)) * 0.1).astype(np.float32)
    g.set_factors(np.zeros((50, 3), np.float32), H0)
    g.run(2, 3)
    W, H = g.factors()
    assert not W.any() and not H.any()
    with pytest.raises(CCDPPError) as ei:
        g.train_rmse()
    assert ei.value.code == CCDPP_EINVAL
    tr = np.array([0, 7, 49], np.int32)
    tc = np.array([0, 3, 39], np.int32)
    tv = np.array([1.0, -2.0, 3.0], np.float32)
    assert g.rmse(tr, tc, tv) == pytest.approx(np.sqrt(np.mean(tv.astype(np.float64) ** 2)),
                                               rel=1e-12)
    assert g.check_consistency() == 0


def test_single_entry():
    print("case: one entry", flush=True)
    row, col = np.array([0], np.int32), np.array([0], np.int32)
    val = np.array([2.5], np.float32)
    H0 = np.array([[0.3, -0.2]], np.float32)
    _compare(1, 1, 2, 0.05, row, col, val, H0, outer=3, inner=2)


@pytest.mark.parametrize("transpose", [False, True])
def test_one_dense_row_or_column(transpose):
    # One row of 5000 entries: it spans windows, chunks and (one workgroup) every wave.
    # k = 1: a single row or column is rank one, so a first feature leaves a residual
    # near the fp32 rounding of A and any further feature would fit rounding noise.
    print(f"case: one dense row transpose={transpose}", flush=True)
    row, col, val, H0 = synth.lengths_problem([5000], 5000, 1, seed=61)
    m, n = 1, 5000
    if transpose:
        row, col, m, n = col, row, n, m
        H0 = (np.random.default_rng(62).standard_normal((n, 1)) * 0.1).astype(np.float32)
    _compare(m, n, 1, 0.1, row, col, val, H0, outer=2, inner=3)


def test_row_across_every_wave_of_a_workgroup():
    # One row of 20,000 entries with a few short rows after it, in one workgroup: the long row
    # is cut between all 16 waves, more partials than a workgroup finishes itself, so the
    # combine kernel finishes it (any short row cut between waves the workgroup finishes).
    lens = [20_000] + list(np.random.default_rng(66).integers(1, 30, 20))
    row, col, val, H0 = synth.lengths_problem(lens, 20_000, 1, seed=67)
    print(f"case: one row across all waves nnz={row.size}", flush=True)
    g = _compare(len(lens), 20_000, 1, 0.1, row, col, val, H0, outer=2, inner=2,
                 opts=make_options(workgroups=1))
    info = g.info()
    print({k: v for k, v in info.items() if k.startswith("u_")})
    assert info["u_rows_combined"] == 1


def test_rows_at_window_and_chunk_boundaries():
    # Lengths around multiples of the 8-entry lane group and the 512-entry window.
    lens = [511, 512, 513, 1023, 1024, 1025, 7, 8, 9, 63, 64, 65, 255, 256, 257] * 4
    row, col, val, H0 = synth.lengths_problem(lens, 3000, 2, seed=63)
    print(f"case: boundary lengths nnz={row.size}", flush=True)
    for opts in (None, make_options(workgroups=2), make_options(gather_mode=(2, 2), tile_width=(256, 64))):
        _compare(len(lens), 3000, 2, 0.05, row, col, val, H0, outer=2, inner=2, opts=opts)


def test_one_feature_one_inner_iteration():
    # k = 1, inner 1: the commit copies the coordinates instead of finishing in place.
    ds = synth.load("tiny")
    w = ds.workload
    print("case: k=1 inner=1", flush=True)
    _compare(w.m, w.n, 1, w.lam, ds.row, ds.col, ds.val, ds.h0(1), outer=4, inner=1)


@pytest.mark.parametrize("n", [32_767, 32_768])
def test_index_width_boundary_of_global_layouts(n):
    # Global gathers keep 16-bit indices while the padding index (the column count)
    # stays below the start bit; one more column needs 32-bit indices.
    lens = list(np.random.default_rng(64).integers(1, 40, 800))
    row, col, val, H0 = synth.lengths_problem(lens, n, 2, seed=65)
    print(f"case: global layout with {n} columns", flush=True)
    g = _compare(len(lens), n, 2, 0.1, row, col, val, H0, outer=2, inner=2,
                 opts=make_options(gather_mode=(1, 1)))
    assert g.info()["u_tile_width"] == n


@pytest.mark.parametrize("m, n", [(32_768, 32_769), (32_769, 32_768)])
@pytest.mark.parametrize("shuffle", [False, True])
def test_degree_counts_at_the_lds_bin_limit(m, n, shuffle):
    # Degrees are counted in LDS for up to 32,768 rows or columns and in global memory
    # above; triplets grouped by row (runs of one key) or shuffled (no runs).
    lens = list(np.random.default_rng(68).integers(1, 16, m))
    row, col, val, H0 = synth.lengths_problem(lens, n, 2, seed=69)
    if shuffle:
        p = np.random.default_rng(70).permutation(row.size)
        row, col, val = row[p], col[p], val[p]
    print(f"case: degree counts m={m} n={n} shuffle={shuffle} nnz={row.size}", flush=True)
    _compare(m, n, 2, 0.1, row, col, val, H0, outer=2, inner=2)


def _splitmix64(x):
    """splitmix64 (Steele, Lea and Flood, OOPSLA 2014) on uint64 arrays."""
    with np.errstate(over="ignore"):
        x = x + np.uint64(0x9E3779B97F4A7C15)
        x = (x ^ (x >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        x = (x ^ (x >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return x ^ (x >> np.uint64(31))


def test_seeded_initial_state():
    """ccdpp_create's initial state: W = 0 (Algorithm 3), and H entry (j, t) is 0.1 z
    with z from the Box-Muller transform of counter draws 2e and 2e + 1 (e = j k + t)
    of splitmix64 keyed by the seed, rounded to float: checked against that
    definition evaluated here, to within one float rounding, and for the spread of
    N(0, 0.01)."""
    m, n, k = 700, 5000, 6
    row, col, val, _ = synth.small_random(m, n, 20_000, k, seed=71)
    g = CCDPP(m, n, k, 0.1, row, col, val, seed=12345)
    W, H = g.factors()
    assert np.all(W == 0)
    e = np.arange(n * k, dtype=np.uint64)
    key = _splitmix64(np.array([12345], dtype=np.uint64))[0]
    with np.errstate(over="ignore"):
        u1 = (_splitmix64(key + np.uint64(2) * e) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
        u2 = (_splitmix64(key + np.uint64(2) * e + np.uint64(1)) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    z = np.sqrt(-2.0 * np.log1p(-u1)) * np.cos(6.283185307179586 * u2)
    ref = (0.1 * z).astype(np.float32).reshape(n, k)
    ulp = np.spacing(np.abs(ref))
    assert np.all(np.abs(H - ref) <= ulp)
    assert abs(float(H.std()) - 0.1) < 0.003 and abs(float(H.mean())) < 0.003
    # the same seed gives the same H, another seed another one; float64 handles start
    # from the same float values
    W2, H2 = CCDPP(m, n, k, 0.1, row, col, val, seed=12345).factors()
    assert np.array_equal(H, H2)
    _, H3 = CCDPP(m, n, k, 0.1, row, col, val, seed=54321).factors()
    assert not np.array_equal(H, H3)
    from paper_1511_02433_amd.ccdpp import make_options
    _, H4 = CCDPP(m, n, k, 0.1, row, col, val, seed=12345, opts=make_options(precision=1)).factors_f64()
    assert np.array_equal(H4, H.astype(np.float64))
