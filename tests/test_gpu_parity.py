"""GPU path against the fp64 CPU oracle on identical seeded inputs.

Tolerances: W and H within 1e-3 (per-feature scaled max relative error) after
one outer iteration, and |delta RMSE| <= 1e-4 after the full run.  The GPU keeps
the residual in fp32 (as the paper's float version does) and sums in fp64, so it
is not bitwise equal to the oracle.
"""
import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

W_TOL = 1e-3
RMSE_TOL = 1e-4


def _pair(m, n, k, lam, row, col, val, H0, threads=0):
    g = CCDPP(m, n, k, lam, row, col, val)
    g.set_factors(np.zeros((m, k), np.float32), H0)
    o = Oracle(m, n, k, lam, row, col, val, H0, threads=threads)
    return g, o


def test_tiny_parity_one_outer_and_full_run():
    ds = synth.load("tiny")
    w = ds.workload
    print(f"case: tiny {w.describe()}", flush=True)
    g, o = _pair(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, ds.H0)
    g.run(1, w.inner)
    o.run(1, w.inner)
    Wg, Hg = g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
    print(f"tiny after 1 outer: W err {ew:.3e}  H err {eh:.3e}")
    assert ew <= W_TOL and eh <= W_TOL
    g.run(w.outer - 1, w.inner)
    o.run(w.outer - 1, w.inner)
    tr_g, tr_o = g.train_rmse(), o.train_rmse()
    te_g = g.rmse(ds.test_row, ds.test_col, ds.test_val)
    te_o = o.test_rmse(ds.test_row, ds.test_col, ds.test_val)
    print(f"tiny full run: train {tr_g:.6f} vs {tr_o:.6f}; test {te_g:.6f} vs {te_o:.6f}")
    assert abs(tr_g - tr_o) <= RMSE_TOL
    assert abs(te_g - te_o) <= RMSE_TOL
    assert g.check_consistency() == 0


# Row lengths at every edge of the scheduling classes: lane groups of 1..64 lanes
# (up to 8 or 16 entries per lane), one workgroup per row up to 32768 entries, and
# rows split over several workgroups beyond that.
EDGE_LENGTHS = [0, 1, 2, 7, 8, 9, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256,
                257, 511, 512, 513, 1023, 1024, 1025, 4095, 4096, 4097, 32767, 32768, 32769,
                70001]


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("inner", [1, 2])
def test_every_schedule_class(transpose, inner):
    n_other = 70_001 + 5
    row, col, val, H0 = synth.lengths_problem(EDGE_LENGTHS * 2, n_other, 3, seed=17)
    m, n = len(EDGE_LENGTHS) * 2, n_other
    if transpose:
        row, col = col, row
        m, n = n, m
        H0 = (np.random.default_rng(5).standard_normal((n, 3)) * 0.1).astype(np.float32)
    print(f"case: edge lengths transpose={transpose} inner={inner} m={m} n={n} nnz={row.size}",
          flush=True)
    g, o = _pair(m, n, 3, 0.1, row, col, val, H0)
    g.run(1, inner)
    o.run(1, inner)
    Wg, Hg = g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
    print(f"W err {ew:.3e}  H err {eh:.3e}")
    assert ew <= W_TOL and eh <= W_TOL
    # Empty rows / columns get a zero coordinate.
    assert np.all(Wg[np.bincount(row, minlength=m) == 0] == 0)
    assert np.all(Hg[np.bincount(col, minlength=n) == 0] == 0)
    assert g.check_consistency() == 0
    R = g.residual().astype(np.float64)
    np.testing.assert_allclose(R, o.residual(), rtol=0, atol=1e-4 * np.abs(val).max())


def test_determinism_and_split_runs_bitwise():
    ds = synth.load("tiny")
    w = ds.workload
    print("case: tiny determinism", flush=True)
    a = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val)
    b = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val)
    for h in (a, b):
        h.set_factors(np.zeros((w.m, w.k), np.float32), ds.H0)
    a.run(2, 3)
    b.run(1, 3)
    b.run(1, 3)
    Wa, Ha = a.factors()
    Wb, Hb = b.factors()
    assert np.array_equal(Wa, Wb) and np.array_equal(Ha, Hb)
    assert np.array_equal(a.residual(), b.residual())
    c = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val)
    c.set_factors(np.zeros((w.m, w.k), np.float32), ds.H0)
    c.run(2, 3)
    Wc, Hc = c.factors()
    assert np.array_equal(Wa, Wc) and np.array_equal(Ha, Hc)


def test_residual_is_a_minus_wht_and_factors_roundtrip():
    row, col, val, H0 = synth.small_random(300, 200, 9000, 5, seed=23)
    print("case: residual definition 300x200", flush=True)
    g = CCDPP(300, 200, 5, 0.05, row, col, val)
    g.run(2, 2)
    W, H = g.factors()
    R = g.residual().astype(np.float64)
    ref = val.astype(np.float64) - np.einsum("ek,ek->e", W[row].astype(np.float64),
                                             H[col].astype(np.float64))
    assert np.abs(R - ref).max() <= 1e-5 * np.abs(val).max()
    # set_factors / get_factors round trip is exact, and the rebuilt residual agrees.
    g.set_factors(W, H)
    W2, H2 = g.factors()
    assert np.array_equal(W, W2) and np.array_equal(H, H2)
    R2 = g.residual().astype(np.float64)
    assert np.abs(R2 - ref).max() <= 1e-6 * np.abs(val).max()
    assert g.check_consistency() == 0


def test_rmse_kernels_match_their_definition():
    row, col, val, H0 = synth.small_random(500, 400, 20000, 6, seed=29)
    print("case: rmse 500x400", flush=True)
    g = CCDPP(500, 400, 6, 0.1, row[:18000], col[:18000], val[:18000])
    g.run(1, 2)
    W, H = g.factors()
    pred = np.einsum("ek,ek->e", W[row].astype(np.float64), H[col].astype(np.float64))
    err = val.astype(np.float64) - pred
    te = np.sqrt(np.mean(err[18000:] ** 2))
    tr = np.sqrt(np.mean(err[:18000] ** 2))
    assert abs(g.rmse(row[18000:], col[18000:], val[18000:]) - te) <= 1e-9 * te
    assert abs(g.train_rmse() - tr) <= 1e-5 * tr


def test_zero_lambda_and_empty_rows():
    row = np.array([0, 0, 1, 1, 3, 4], dtype=np.int32)
    col = np.array([0, 1, 1, 2, 0, 4], dtype=np.int32)
    val = np.array([1.0, -2.0, 0.5, 3.0, 1.5, 2.0], dtype=np.float32)
    H0 = np.full((6, 2), 0.1, dtype=np.float32)
    print("case: lambda 0 and 0.1 with empty rows", flush=True)
    # lambda = 0: rows 2, 5 and columns 3, 5 are empty, their coordinates are 0, nothing is NaN.
    # (With lambda = 0 the second feature of a single-entry row is a ratio of two rounding
    # residues, so values are compared with the oracle only for lambda > 0.)
    for lam in (0.0, 0.1):
        g, o = _pair(6, 6, 2, lam, row, col, val, H0)
        g.run(2, 2)
        o.run(2, 2)
        Wg, Hg = g.factors()
        assert np.all(np.isfinite(Wg)) and np.all(np.isfinite(Hg))
        assert np.all(Wg[[2, 5]] == 0) and np.all(Hg[[3, 5]] == 0)
        if lam > 0:
            Wo, Ho = o.factors()
            assert colscaled_max_rel_err(Wg, Wo) <= W_TOL
            assert colscaled_max_rel_err(Hg, Ho) <= W_TOL


# Every layout strategy on the same problem: automatic, global-memory gathers,
# LDS staging with small tiles (several tiles per side, per-tile partials and the
# combine), and very few persistent workgroups (long unit loops per wave).
LAYOUTS = {
    "auto": dict(),
    "global": dict(gather_mode=(1, 1)),
    "tiled": dict(gather_mode=(2, 2), tile_width=(192, 128)),
    "tiled_odd": dict(gather_mode=(2, 2), tile_width=(100, 333), workgroups=3),
    "mixed": dict(gather_mode=(1, 2), tile_width=(0, 64), workgroups=1),
    # Hot layouts: a few leading columns staged, the rest gathered from global memory
    # (widths 64 and 96 of 900 and 1500), and the widest hot width, which stages all
    # but the last partial group of 32 columns.
    "hot": dict(gather_mode=(3, 3), tile_width=(64, 96)),
    "hot_wide": dict(gather_mode=(3, 3), workgroups=3),
    "hot_mixed": dict(gather_mode=(2, 3), tile_width=(128, 32), workgroups=1),
}


@pytest.mark.parametrize("name", list(LAYOUTS))
def test_layout_strategies_match_oracle(name):
    from paper_1511_02433_amd.ccdpp import make_options
    # A few heavy rows plus many short ones, so long segments and every lane-group
    # class occur on the user side; item lengths follow from the random columns.
    lens = [850, 700, 300, 40] + list(np.random.default_rng(31).integers(0, 80, 1496))
    row, col, val, H0 = synth.lengths_problem(lens, 900, 4, seed=32)
    print(f"case: layout {name} nnz={row.size}", flush=True)
    opts = make_options(**LAYOUTS[name])
    g = CCDPP(1500, 900, 4, 0.1, row, col, val, opts=opts)
    info = g.info()
    print({k: v for k, v in info.items() if k.startswith(("u_", "v_"))})
    g.set_factors(np.zeros((1500, 4), np.float32), H0)
    o = Oracle(1500, 900, 4, 0.1, row, col, val, H0)
    for outer in range(2):
        g.run(1, 2)
        o.run(1, 2)
        Wg, Hg = g.factors()
        Wo, Ho = o.factors()
        ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
        print(f"outer {outer}: W err {ew:.3e}  H err {eh:.3e}")
        if outer == 0:
            assert ew <= W_TOL and eh <= W_TOL
    assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    assert g.check_consistency() == 0
    if name == "tiled":
        assert info["u_tiles"] > 1 and info["v_tiles"] > 1
    if name == "global":
        assert info["u_gather"] == 1 and info["v_gather"] == 1
    if name.startswith("hot"):
        assert info["v_gather"] == 3
    if name == "auto":
        # Short rows at every share boundary: the workgroups finish the rows cut between
        # their waves themselves, and no combine kernel runs on either side.
        for side in "uv":
            assert info[f"{side}_rows_finished_in_pass"] > 0 and info[f"{side}_rows_combined"] == 0


@pytest.mark.parametrize("tiles", ["one", "several"])
def test_cache_policies_give_identical_results(tiles):
    # The cache policy only changes how the residual stream is loaded and stored, so
    # every policy gives bitwise the same factors and residual.  "one": one tile per
    # side (the kernels for P == 1); "several": several tiles per side.
    from paper_1511_02433_amd.ccdpp import CCDPPError, CCDPP_EINVAL, make_options
    lens = [850, 700, 300, 40] + list(np.random.default_rng(31).integers(0, 80, 1496))
    row, col, val, H0 = synth.lengths_problem(lens, 900, 4, seed=32)
    tw = (0, 0) if tiles == "one" else (192, 128)
    print(f"case: cache policies, {tiles} tile(s) per side", flush=True)
    ref = None
    for cache in [(1, 1), (0, 0), (2, 2), (3, 3), (2, 1), (1, 3), (3, 2)]:
        g = CCDPP(1500, 900, 4, 0.1, row, col, val,
                  opts=make_options(gather_mode=(2, 2), tile_width=tw, cache=cache))
        info = g.info()
        assert (info["u_tiles"] == 1) == (tiles == "one")
        want = cache if cache != (0, 0) else (3, 3)  # automatic: the streams fit the cache
        assert (info["u_cache"], info["v_cache"]) == want
        g.set_factors(np.zeros((1500, 4), np.float32), H0)
        g.run(1, 2)
        first = g.factors()
        g.run(1, 2)
        out = first + g.factors() + (g.residual(),)
        assert g.check_consistency() == 0
        rmse = g.train_rmse()
        g.run(1, 1)        # one inner iteration: automatic write-back stores off
        g.ccd_run(1)       # element-wise CCD on the same copies
        out += g.factors() + (g.residual(),)
        assert g.check_consistency() == 0
        g.close()
        if ref is None:
            ref = out
            o = Oracle(1500, 900, 4, 0.1, row, col, val, H0)
            o.run(1, 2)
            Wo, Ho = o.factors()
            assert colscaled_max_rel_err(first[0], Wo) <= W_TOL
            assert colscaled_max_rel_err(first[1], Ho) <= W_TOL
            o.run(1, 2)
            assert abs(rmse - o.train_rmse()) <= RMSE_TOL
        else:
            for a, b in zip(ref, out):
                assert np.array_equal(a, b), f"cache {cache} differs"
    # Write-back policies need a tiled float copy.
    for kw in (dict(gather_mode=(1, 1), cache=(3, 1)), dict(gather_mode=(3, 3), cache=(1, 2)),
               dict(precision=1, cache=(2, 2))):
        with pytest.raises(CCDPPError) as ei:
            CCDPP(1500, 900, 4, 0.1, row, col, val, opts=make_options(**kw))
        assert ei.value.code == CCDPP_EINVAL and "cache policy" in str(ei.value)
    # Automatic choice elsewhere: copies that are not tiled, and double precision, stream.
    for kw in (dict(gather_mode=(1, 3)), dict(precision=1)):
        g = CCDPP(1500, 900, 4, 0.1, row, col, val, opts=make_options(**kw))
        info = g.info()
        assert (info["u_cache"], info["v_cache"]) == (1, 1)
        g.close()


@pytest.mark.parametrize("case", ["one_tile", "tiles", "double", "mixed_gaps"])
def test_index_coding_gives_identical_results(case):
    # Delta-coded index windows decode to the plain indices, so the passes, the
    # residual rebuild of set_factors and element-wise CCD give bitwise the same
    # results with and without them.  "mixed_gaps": rows of 1 to 5000 entries over
    # 6000 columns, so that some windows have steps past 2047 and stay plain.
    from paper_1511_02433_amd.ccdpp import make_options
    if case == "mixed_gaps":
        lens = [5000, 3000, 2049, 1025, 1024, 513, 200, 64, 9, 1, 0] * 3
        m, n, k = len(lens), 6000, 3
        row, col, val, H0 = synth.lengths_problem(lens, n, k, seed=41)
    else:
        lens = [850, 700, 300, 40] + list(np.random.default_rng(31).integers(0, 80, 1496))
        m, n, k = 1500, 900, 4
        row, col, val, H0 = synth.lengths_problem(lens, n, k, seed=32)
    # Streaming copies: the automatic choice codes no window of a copy that stays cached.
    kw = {"one_tile": dict(gather_mode=(2, 2)), "tiles": dict(gather_mode=(2, 2), tile_width=(192, 128)),
          "double": dict(gather_mode=(2, 2), precision=1), "mixed_gaps": dict()}[case]
    kw["cache"] = (1, 1)
    print(f"case: index coding, {case}", flush=True)
    W1 = (np.random.default_rng(5).standard_normal((m, k)) * 0.1).astype(np.float32)
    outs = []
    for coding in [(1, 1), (0, 0)]:
        g = CCDPP(m, n, k, 0.1, row, col, val, opts=make_options(index_coding=coding, **kw))
        info = g.info()
        print({key: v for key, v in info.items() if "windows" in key})
        if coding == (1, 1):
            assert info["u_delta_windows"] == 0 and info["v_delta_windows"] == 0
        else:
            assert info["u_delta_windows"] > 0 and info["v_delta_windows"] > 0
        g.set_factors(np.zeros((m, k), np.float32), H0)
        g.run(1, 2)
        out = list(g.factors())
        g.set_factors(W1, H0)  # rebuilds the residual from the stored indices
        out.append(g.residual())
        g.run(1, 3)
        g.ccd_run(1)
        out += list(g.factors()) + [g.residual()]
        assert g.check_consistency() == 0
        g.close()
        outs.append(out)
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("layout", ["auto", "global", "hot"])
@pytest.mark.parametrize("transpose", [False, True])
def test_short_segments_fill_windows(layout, transpose):
    # Rows of 1..8 entries: every segment fills one lane after alignment padding, so
    # full windows hold 64 segment starts (the last lane's segment lies past the
    # window's row-scalar slots).  40,000 columns need 32-bit indices outside tiles.
    # Tiles of them would hold about one entry per row, so the automatic layout of
    # that side is hot: the plain passes stage all 40,000 columns, the first passes
    # (two or three vectors) the leading 20,416 or 13,568, and gather the rest,
    # swizzled indices included, from global memory.  "hot" stages only 4,096.
    from paper_1511_02433_amd.ccdpp import make_options
    lens = list(np.random.default_rng(51).integers(1, 9, 6000))
    row, col, val, H0 = synth.lengths_problem(lens, 40_000, 3, seed=52)
    m, n = len(lens), 40_000
    if transpose:
        row, col = col, row
        m, n = n, m
        H0 = (np.random.default_rng(53).standard_normal((n, 3)) * 0.1).astype(np.float32)
    print(f"case: short segments layout={layout} transpose={transpose} nnz={row.size}",
          flush=True)
    opts = {"global": make_options(gather_mode=(1, 1)),
            "hot": make_options(gather_mode=(3, 3), tile_width=(4096, 4096)),
            "auto": make_options()}[layout]
    g = CCDPP(m, n, 3, 0.1, row, col, val, opts=opts)
    info = g.info()
    print({k: v for k, v in info.items() if k.startswith(("u_", "v_"))})
    wide = "v" if transpose else "u"  # the side that gathers over 40,000 columns
    assert info[f"{wide}_gather"] == {"global": 1, "hot": 3, "auto": 3}[layout]
    g.set_factors(np.zeros((m, 3), np.float32), H0)
    o = Oracle(m, n, 3, 0.1, row, col, val, H0)
    g.run(1, 2)
    o.run(1, 2)
    Wg, Hg = g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
    print(f"W err {ew:.3e}  H err {eh:.3e}")
    assert ew <= W_TOL and eh <= W_TOL
    g.run(1, 2)
    o.run(1, 2)
    assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    assert g.check_consistency() == 0


def test_heavy_rows_in_tiles_and_layout_equivalence():
    # Rows far longer than kGroupMaxLen inside tiles, plus the same problem under two
    # layouts: results agree to summation-order rounding.  With one tile per side,
    # rows cut between the waves of a workgroup are finished by the pass itself, and
    # rows too long to keep inside one workgroup's share by the combine kernel.
    from paper_1511_02433_amd.ccdpp import make_options
    lens = [5000, 3000, 2049, 1025, 1024, 513, 200, 64, 9, 1, 0] * 3
    row, col, val, H0 = synth.lengths_problem(lens, 6000, 3, seed=41)
    m = len(lens)
    print("case: heavy rows in tiles", flush=True)
    res = []
    for opts in (make_options(), make_options(gather_mode=(2, 2), tile_width=(512, 16))):
        g = CCDPP(m, 6000, 3, 0.05, row, col, val, opts=opts)
        info = g.info()
        print({k: v for k, v in info.items() if k.startswith(("u_", "v_"))})
        if info["u_tiles"] == 1:
            # Rows of 5000 entries in shares of about 8000: the shares stay balanced and
            # the combine kernel finishes every cut row.
            assert info["u_rows_finished_in_pass"] == 0 and info["u_rows_combined"] > 0
        g.set_factors(np.zeros((m, 3), np.float32), H0)
        g.run(1, 3)
        res.append(g.factors())
        assert g.check_consistency() == 0
    o = Oracle(m, 6000, 3, 0.05, row, col, val, H0)
    o.run(1, 3)
    Wo, Ho = o.factors()
    for W, H in res:
        assert colscaled_max_rel_err(W, Wo) <= W_TOL and colscaled_max_rel_err(H, Ho) <= W_TOL
