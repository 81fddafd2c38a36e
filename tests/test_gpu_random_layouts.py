"""Seeded random combinations of problem shape and layout options against the fp64
oracle: row lengths from one to the column count, empty rows and columns, every
gather mode with forced tile and hot widths, workgroup counts from 1 to 64, segment
weights, both index codings, the cache policies a copy allows, forced splits of the
item-major copy, float and double, lambda from 0.01 to 1.  Each case: W and H
after one outer iteration, the training RMSE after a second, then, from the oracle's
factors, W and H after an outer iteration of element-wise CCD on the same handle,
and bitwise agreement of the two residual copies throughout."""
import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP, make_options
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

CASES = 64
LARGER = 48  # cases from here on: up to 30,000 rows or columns and 400,000 entries


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    big = seed >= LARGER
    m = int(rng.integers(1, 30_000 if big else 2500))
    n = int(rng.integers(1, 30_000 if big else 2500))
    # heavy-tailed row lengths, some rows empty, capped by the column count
    lens = np.minimum(n, np.floor(rng.pareto(1.2, m) * rng.integers(1, 12))).astype(int)
    lens[rng.random(m) < 0.1] = 0
    while lens.sum() > (400_000 if big else 60_000):
        lens //= 2
    k = int(rng.choice([1, 2, 3, 5, 8]))
    inner = int(rng.choice([1, 2, 3]))
    # No lambda = 0 here: a row (or column) with one entry is then fitted exactly, its
    # residual is rounding noise, and a later feature divides that noise by noise (one
    # case: a column 0 in the oracle, 0.2 here, in double; W off by 6e-3 in float).
    # lambda = 0 has tests of its own (empty rows, reading A-6).
    lam = float(rng.choice([0.01, 0.05, 1.0]))
    prec = int(rng.random() < 0.3)
    gm = [int(rng.choice([0, 1, 2, 3])) for _ in range(2)]
    tw = [0, 0]
    for side in (0, 1):
        cols = n if side == 0 else m
        if gm[side] == 2 and rng.random() < 0.7:
            tw[side] = int(rng.integers(1, max(2, min(cols, 4000))))
        elif gm[side] == 3 and cols >= 64 and rng.random() < 0.7:
            tw[side] = 32 * int(rng.integers(1, max(2, min(cols // 32, 120))))
    cache = [0, 0]
    for side in (0, 1):
        if gm[side] == 2 and prec == 0:
            cache[side] = int(rng.choice([0, 1, 2, 3]))
    split = 0
    if gm[1] == 0 and n >= 2:
        split = int(rng.choice([0, -1, int(rng.integers(1, n))]))
    opts = make_options(gather_mode=tuple(gm), tile_width=tuple(tw),
                        workgroups=int(rng.choice([0, 1, 2, 5, 13, 64])),
                        seg_weight=int(rng.choice([0, -1, 1, 16])), precision=prec,
                        cache=tuple(cache), index_coding=(int(rng.integers(0, 2)), int(rng.integers(0, 2))),
                        split_rows=split)
    desc = (f"m={m} n={n} k={k} inner={inner} lam={lam} prec={prec} gather={gm} tile={tw} "
            f"cache={cache} split={split}")
    return m, n, k, inner, lam, prec, lens, opts, desc


@pytest.mark.parametrize("seed", range(CASES))
def test_random_layout(seed):
    m, n, k, inner, lam, prec, lens, opts, desc = _case(seed)
    row, col, val, H0 = synth.lengths_problem(list(lens), n, k, seed=2000 + seed)
    print(f"case {seed}: {desc} nnz={row.size}", flush=True)
    g = CCDPP(m, n, k, lam, row, col, val, opts=opts)
    o = Oracle(m, n, k, lam, row, col, val, H0)
    W0 = np.zeros((m, k), np.float32)
    if prec:
        g.set_factors_f64(W0.astype(np.float64), H0.astype(np.float64))
    else:
        g.set_factors(W0, H0)
    g.run(1, inner)
    o.run(1, inner)
    W, H = g.factors_f64() if prec else g.factors()
    Wo, Ho = o.factors()
    tol = 1e-9 if prec else 1e-3
    ew, eh = colscaled_max_rel_err(W, Wo), colscaled_max_rel_err(H, Ho)
    print(f"  W err {ew:.2e}  H err {eh:.2e}", flush=True)
    assert ew <= tol and eh <= tol
    assert g.check_consistency() == 0
    g.run(1, inner)
    o.run(1, inner)
    if row.size:
        assert abs(g.train_rmse() - o.train_rmse()) <= (1e-9 if prec else 1e-4)
    assert g.check_consistency() == 0
    # Then one outer iteration of element-wise CCD (Algorithm 2) on the same copies,
    # both sides starting from the oracle's factors (in the handle's precision).
    Ws, Hs = o.factors()
    o.close()
    if not prec:
        Ws, Hs = Ws.astype(np.float32), Hs.astype(np.float32)
        g.set_factors(Ws, Hs)
    else:
        g.set_factors_f64(Ws, Hs)
    o = Oracle(m, n, k, lam, row, col, val, Hs, W0=Ws)
    g.ccd_run(1)
    o.ccd_run(1)
    W, H = g.factors_f64() if prec else g.factors()
    Wo, Ho = o.factors()
    ew, eh = colscaled_max_rel_err(W, Wo), colscaled_max_rel_err(H, Ho)
    print(f"  element-wise CCD: W err {ew:.2e}  H err {eh:.2e}", flush=True)
    assert ew <= tol and eh <= tol
    assert g.check_consistency() == 0
    g.close()
    o.close()
