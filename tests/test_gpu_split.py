"""The split item-major copy against the fp64 oracle.

When tiles of the whole item-major copy would hold too few entries per row
segment, the copy may be split: its items with the most ratings are tiled (all
their gathers from LDS) and the others kept in a hot layout (the most frequent
users staged, the others gathered from global memory).  The two parts are one
copy of the residual: one value array, one map to the user-major copy, one pass
after the other.  The problem here has 40 items of 3,000 ratings over 60,000
users and 19,960 items of 1 to 6 ratings, so the automatic layout splits it;
forced splits cover one tiled item, all but one, and points in between.

Checked: W and H within 1e-3 of the oracle after one outer iteration (1e-9 in
float64), the training RMSE within 1e-4 after the next, the two residual copies
bitwise equal, the residual rebuild of set_factors, element-wise CCD (Algorithm
2) over the split copy, and bitwise determinism.
"""
import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP, CCDPPError, CCDPP_EINVAL, make_options
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

W_TOL = 1e-3
RMSE_TOL = 1e-4
M, N, K = 60_000, 20_000, 4


def _problem():
    lens = [3000] * 40 + list(np.random.default_rng(61).integers(1, 7, N - 40))
    # Rows of lengths_problem are items here; transposed, users are rows.
    irow, ucol, val, _ = synth.lengths_problem(lens, M, K, seed=62)
    H0 = (np.random.default_rng(63).standard_normal((N, K)) * 0.1).astype(np.float32)
    return ucol, irow, val, H0


PROB = None


def _prob():
    global PROB
    if PROB is None:
        PROB = _problem()
    return PROB


def _run_case(opts, inner=2, tol=W_TOL, precision_note=""):
    row, col, val, H0 = _prob()
    g = CCDPP(M, N, K, 0.1, row, col, val, opts=opts)
    info = g.info()
    print({k: v for k, v in info.items() if k.startswith(("v_", "v2_"))}, flush=True)
    g.set_factors(np.zeros((M, K), np.float32), H0)
    o = Oracle(M, N, K, 0.1, row, col, val, H0)
    g.run(1, inner)
    o.run(1, inner)
    Wg, Hg = g.factors_f64() if tol < 1e-6 else g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(Wg, Wo), colscaled_max_rel_err(Hg, Ho)
    print(f"{precision_note}W err {ew:.3e}  H err {eh:.3e}", flush=True)
    assert ew <= tol and eh <= tol
    g.run(1, inner)
    o.run(1, inner)
    assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    assert g.check_consistency() == 0
    return g, o, info


@pytest.mark.parametrize("split", [0, 1, 40, 1000, N - 1, -1])
def test_split_item_major_copy_matches_oracle(split):
    print(f"case: split_rows={split}", flush=True)
    g, o, info = _run_case(make_options(split_rows=split))
    if split == 0:
        # The automatic layout splits this copy, tiling the 40 long items.
        assert 0 < info["v_split_rows"] <= 400
    elif split == -1:
        assert info["v_split_rows"] == 0 and info["v_gather"] == 3
    else:
        assert info["v_split_rows"] == split
    if info["v_split_rows"]:
        assert info["v_gather"] == 2 and info["v2_gather"] == 3
        assert info["v_tiles"] > 1
    g.close()
    o.close()


def test_split_copy_in_float64():
    print("case: split_rows=40 float64", flush=True)
    g, o, info = _run_case(make_options(split_rows=40, precision=1), tol=1e-9, precision_note="f64 ")
    assert info["v_split_rows"] == 40 and info["value_bytes"] == 8
    g.close()
    o.close()


@pytest.mark.parametrize("split", [0, 1000])
def test_split_copy_elementwise_ccd_and_rebuild(split):
    row, col, val, H0 = _prob()
    print(f"case: element-wise CCD and rebuild, split_rows={split}", flush=True)
    g = CCDPP(M, N, K, 0.1, row, col, val, opts=make_options(split_rows=split))
    assert g.info()["v_split_rows"] > 0
    g.set_factors(np.zeros((M, K), np.float32), H0)
    o = Oracle(M, N, K, 0.1, row, col, val, H0)
    g.ccd_run(1)
    o.ccd_run(1)
    Wg, Hg = g.factors()
    Wo, Ho = o.factors()
    assert colscaled_max_rel_err(Wg, Wo) <= W_TOL and colscaled_max_rel_err(Hg, Ho) <= W_TOL
    assert g.check_consistency() == 0
    # CCD++ after element-wise CCD on the same copies, then the rebuild of the residual.
    g.run(1, 2)
    o.run(1, 2)
    assert abs(g.train_rmse() - o.train_rmse()) <= RMSE_TOL
    W, H = g.factors()
    g.set_factors(W, H)
    ref = val.astype(np.float64) - np.einsum("ek,ek->e", W[row].astype(np.float64),
                                             H[col].astype(np.float64))
    R = g.residual().astype(np.float64)
    assert np.abs(R - ref).max() <= 1e-6 * np.abs(val).max()
    assert g.check_consistency() == 0
    g.close()
    o.close()


def test_split_copy_is_deterministic():
    row, col, val, H0 = _prob()
    print("case: split determinism", flush=True)
    outs = []
    for _ in range(2):
        g = CCDPP(M, N, K, 0.1, row, col, val, opts=make_options(split_rows=40))
        g.set_factors(np.zeros((M, K), np.float32), H0)
        g.run(2, 3)
        outs.append(g.factors() + (g.residual(),))
        g.close()
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_split_rows_arguments():
    row, col, val, _ = _prob()
    for kw in (dict(split_rows=N), dict(split_rows=-2), dict(split_rows=5, gather_mode=(0, 3))):
        with pytest.raises(CCDPPError) as ei:
            CCDPP(M, N, K, 0.1, row, col, val, opts=make_options(**kw))
        assert ei.value.code == CCDPP_EINVAL and "split_rows" in str(ei.value)


def test_split_copy_cache_policies_and_index_coding_are_bitwise_neutral():
    """On a split copy, the tiled part takes the write-back policies and delta-coded
    indices, the hot part streams; none of them changes a bit of the results."""
    row, col, val, H0 = _prob()
    print("case: split copy, cache policies and index coding", flush=True)
    ref = None
    for kw in (dict(cache=(1, 1), index_coding=(1, 1)), dict(cache=(1, 1)), dict(cache=(1, 2)),
               dict(cache=(1, 3)), dict(cache=(2, 2), index_coding=(0, 1))):
        g = CCDPP(M, N, K, 0.1, row, col, val, opts=make_options(split_rows=40, **kw))
        info = g.info()
        assert info["v_split_rows"] == 40 and info["v2_cache"] == 1
        assert info["v_cache"] == kw["cache"][1]
        g.set_factors(np.zeros((M, K), np.float32), H0)
        g.run(1, 2)
        g.run(1, 1)
        g.ccd_run(1)
        out = g.factors() + (g.residual(),)
        assert g.check_consistency() == 0
        g.close()
        if ref is None:
            ref = out
        else:
            for a, b in zip(ref, out):
                assert np.array_equal(a, b), f"{kw} differs"
