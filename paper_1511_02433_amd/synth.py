"""Seeded synthetic rating matrices shaped like the workloads of the CCD++ study.

This module only draws inputs: observed positions Omega, rating values A_ij and
the initial factor H0.  It holds none of the factorization's arithmetic, so the
CPU oracle and the GPU library can both be fed from it without sharing any part
of the method.

The paper evaluates on the Netflix ratings (Section 8: 100,480,507 ratings of
480,189 users on 17,770 movies).  That data is not available here, so every
workload is synthetic: the "large" workload takes the Netflix shape (m, n, nnz)
with power-law user and item degrees, and the other workloads are a small
uniform case, a medium power-law case and a very large power-law case.

Degree model ("Zipf(alpha)" with a minimum, a maximum and an exact total):
the rank curve d_r = clamp(C * r**-alpha, d_min, d_max), r = 1..count, with C
found by bisection so that the rounded curve sums to the requested total
(largest-remainder rounding), assigned to ids by a seeded permutation.  Row
(user) degrees are exact; each row then draws its distinct columns by weighted
sampling without replacement, with column weights from the items' own rank
curve, so item degrees follow that curve approximately.

Weighted sampling without replacement is done as successive sampling: i.i.d.
draws from the column distribution, rejecting columns already present in the
row, until the row holds its degree.  Draws are made in batches of the current
deficit, which accepts exactly the same sets as drawing one at a time.  Rows
asking for more than a quarter of all columns use the equivalent exponential-
key (Efraimidis-Spirakis) selection instead, which needs no rejection loop.
"""
from __future__ import annotations

import hashlib
import json
import math
import os
import sys
import time
from dataclasses import dataclass, field

import numpy as np

BASE_SEED = 151102433


@dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    m: int
    n: int
    nnz: int                 # training entries (exact)
    holdout: int             # extra distinct entries, disjoint from training
    k: int
    lam: float
    outer: int
    inner: int
    kind: str                # "uniform" | "powerlaw"
    alpha_u: float = 0.0
    alpha_i: float = 0.0
    dmin_u: int = 1
    dmin_i: int = 1
    dmax_u: int = 0          # 0 -> floor(n / 2)
    dmax_i: int = 0          # 0 -> floor(m / 2)
    values: str = "lowrank"  # value model, see _values()
    extra: dict = field(default_factory=dict)

    def describe(self) -> str:
        return (f"{self.name}: m={self.m} n={self.n} nnz={self.nnz} holdout={self.holdout} "
                f"k={self.k} lambda={self.lam} outer={self.outer} inner={self.inner}")


WORKLOADS = {
    # 2,000 x 1,000, 50,000 uniform distinct positions, rank-8 values plus noise.
    "tiny": Workload("tiny", 0, 2000, 1000, 50_000, 2_500, 8, 0.05, 5, 3, "uniform",
                     values="tiny"),
    # 71,567 x 10,681, 10,000,054 entries, Zipf(1.2) both sides, users >= 20.
    "medium": Workload("medium", 1, 71_567, 10_681, 10_000_054, 0, 40, 0.05, 10, 3,
                       "powerlaw", alpha_u=1.2, alpha_i=1.2, dmin_u=20, dmin_i=1,
                       values="halfstar"),
    # Netflix shape: 480,189 x 17,770, 100,480,507 entries; users Zipf(1.1) up to
    # 17,000, items Zipf(0.9) from 3 up to 230,000; integer stars 1..5.
    "large": Workload("large", 2, 480_189, 17_770, 100_480_507, 1_400_000, 40, 0.05, 10, 3,
                      "powerlaw", alpha_u=1.1, alpha_i=0.9, dmin_u=1, dmin_i=3,
                      dmax_u=17_000, dmax_i=230_000, values="stars"),
    # 1,000,990 x 624,961, 252,800,275 entries; users Zipf(1.0), items Zipf(1.3);
    # integer scores 0..100.
    "vlarge": Workload("vlarge", 4, 1_000_990, 624_961, 252_800_275, 0, 40, 1.0, 5, 3,
                       "powerlaw", alpha_u=1.0, alpha_i=1.3, values="score100"),
}
# The rank sweep reuses the large matrix with k in {10, 40, 100} and 5 x 3 iterations.
RANK_SWEEP = (10, 40, 100)


def _streams(config_id: int):
    ss = np.random.SeedSequence([BASE_SEED, config_id]).spawn(5)
    # 0: degree permutations, 1: positions, 2: values, 3: holdout split, 4: H0
    return [np.random.Generator(np.random.PCG64(s)) for s in ss]


def _log(msg: str, verbose: bool):
    if verbose:
        print(f"[synth] {msg}", file=sys.stderr, flush=True)


def rank_curve(count: int, total: int, alpha: float, dmin: int, dmax: int) -> np.ndarray:
    """Integer degrees on a clamped power-law rank curve summing exactly to ``total``."""
    if not (dmin * count <= total <= dmax * count):
        raise ValueError("degree bounds cannot reach the requested total")
    r = np.arange(1, count + 1, dtype=np.float64)
    base = r ** (-alpha)

    def curve(c):
        return np.clip(c * base, dmin, dmax)

    lo, hi = 0.0, float(dmax) / base[-1] * 2.0 + 1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if curve(mid).sum() < total:
            lo = mid
        else:
            hi = mid
    d = curve(hi)
    fl = np.floor(d)
    short = int(total - fl.sum())
    if short < 0:
        raise RuntimeError("bisection overshoot")
    frac = d - fl
    if short > 0:
        order = np.argsort(-frac, kind="stable")
        fl[order[:short]] += 1
    out = fl.astype(np.int64)
    assert out.sum() == total and out.min() >= dmin and out.max() <= dmax
    return out


def _sorted_uniforms(counts: np.ndarray, rng: np.random.Generator) -> np.ndarray:
    """For each segment of length counts[s], that many sorted U(0,1) values (exponential spacings)."""
    tot = int(counts.sum())
    seg = counts + 1
    e = rng.standard_exponential(int(seg.sum()))
    cs = np.cumsum(e)
    ends = np.cumsum(seg) - 1                      # index of each segment's last spacing
    starts = ends - seg + 1
    base = np.where(starts > 0, cs[starts - 1], 0.0)
    total = cs[ends] - base
    owner = np.repeat(np.arange(len(counts)), seg)
    keep = np.ones(len(e), dtype=bool)
    keep[ends] = False
    u = (cs[keep] - base[owner[keep]]) / total[owner[keep]]
    assert u.size == tot
    return u


def _sample_positions(deg: np.ndarray, q: np.ndarray, rng: np.random.Generator,
                      verbose: bool) -> tuple[np.ndarray, np.ndarray]:
    """Distinct (row, col) per row: deg[r] columns, weighted by q, without replacement."""
    m = deg.size
    n = q.size
    cdf = np.cumsum(q, dtype=np.float64)
    cdf /= cdf[-1]
    heavy = deg > n // 4
    rows_out, cols_out = [], []

    # Exact exponential-key selection for very heavy rows.
    for r in np.flatnonzero(heavy):
        key = np.log(rng.random(n)) / q
        pick = np.argpartition(-key, deg[r] - 1)[: deg[r]]
        pick.sort()
        rows_out.append(np.full(pick.size, r, dtype=np.int32))
        cols_out.append(pick.astype(np.int32))

    light = np.flatnonzero(~heavy)
    need = deg[light].astype(np.int64)
    # First draw: sorted uniforms per row, so duplicate columns are adjacent.
    u = _sorted_uniforms(need, rng)
    cols = np.searchsorted(cdf, u, side="right").astype(np.int64)
    np.minimum(cols, n - 1, out=cols)
    rows = np.repeat(light.astype(np.int64), need)
    keys = rows * n + cols
    del u, cols, rows
    keep = np.ones(keys.size, dtype=bool)
    keep[1:] = keys[1:] != keys[:-1]
    keys = keys[keep]
    del keep
    krow = keys // n
    got = np.bincount(krow, minlength=m)
    deficit = np.where(heavy, 0, deg - got)
    # Rows already complete are set aside; only deficient rows are redrawn.  Their
    # entries are kept as one sorted array (`work`) plus a smaller sorted array of the
    # entries added since it was last merged (`fresh`), so that a round costs about
    # as much as its own draws; each row remembers the round that completed it.
    short = deficit > 0
    sel = short[krow]
    done0 = keys[~sel]
    work = keys[sel]
    del keys, krow, sel
    fresh = np.zeros(0, dtype=np.int64)
    fin_round = np.zeros(m, dtype=np.int32)

    def held_in(arr, x):
        if arr.size == 0:
            return np.zeros(x.size, dtype=bool)
        pos = np.searchsorted(arr, x)
        h = np.zeros(x.size, dtype=bool)
        inside = pos < arr.size
        h[inside] = arr[pos[inside]] == x[inside]
        return h

    def merged(a, b):
        return np.insert(a, np.searchsorted(a, b), b)

    rounds = 0
    while deficit.sum() > 0:
        rounds += 1
        bad = np.flatnonzero(deficit > 0)
        add_u = _sorted_uniforms(deficit[bad], rng)
        add_c = np.minimum(np.searchsorted(cdf, add_u, side="right"), n - 1).astype(np.int64)
        add_r = np.repeat(bad.astype(np.int64), deficit[bad])
        # The draws come sorted (rows ascending, columns ascending inside a row).
        add = add_r * n + add_c
        del add_u, add_c, add_r
        keep = np.ones(add.size, dtype=bool)
        keep[1:] = add[1:] != add[:-1]
        add = add[keep]
        add = add[~(held_in(work, add) | held_in(fresh, add))]
        fresh = merged(fresh, add)
        if fresh.size > work.size // 8:
            work = merged(work, fresh)
            fresh = np.zeros(0, dtype=np.int64)
        deficit[bad] -= np.bincount(add // n, minlength=m)[bad]
        fin_round[bad[deficit[bad] == 0]] = rounds
        if rounds > 10_000:
            raise RuntimeError("successive sampling did not converge")
    work = merged(work, fresh)
    # Rows in the order they were completed, each row's entries in column order.
    done = [done0, work[np.argsort(fin_round[work // n], kind="stable")]]
    del work, fresh
    keys = np.concatenate(done)
    _log(f"positions: {keys.size + sum(c.size for c in cols_out)} drawn, {rounds} top-up rounds", verbose)
    rows_out.append((keys // n).astype(np.int32))
    cols_out.append((keys % n).astype(np.int32))
    return np.concatenate(rows_out), np.concatenate(cols_out)


def _latent_dot(rows, cols, X, Y, chunk=1 << 21):
    out = np.empty(rows.size, dtype=np.float64)
    for s in range(0, rows.size, chunk):
        e = min(rows.size, s + chunk)
        out[s:e] = np.einsum("ij,ij->i", X[rows[s:e]], Y[cols[s:e]])
    return out


def _values(w: Workload, rows, cols, rng) -> np.ndarray:
    if w.values == "tiny":
        # W*, H* rank 8 with entries of variance 1/sqrt(8); A = (W* H*^T)_ij + N(0, 0.1^2).
        r = 8
        sd = (1.0 / math.sqrt(r)) ** 0.5
        X = rng.standard_normal((w.m, r)) * sd
        Y = rng.standard_normal((w.n, r)) * sd
        a = _latent_dot(rows, cols, X, Y) + rng.standard_normal(rows.size) * 0.1
        return a.astype(np.float32)
    # Rank-20 latent score with entries of variance 1/sqrt(20) (so Var s ~ 1), plus N(0, 0.8^2).
    r = 20
    sd = (1.0 / math.sqrt(r)) ** 0.5
    X = (rng.standard_normal((w.m, r)) * sd).astype(np.float32)
    Y = (rng.standard_normal((w.n, r)) * sd).astype(np.float32)
    s = _latent_dot(rows, cols, X, Y)
    s += rng.standard_normal(rows.size) * 0.8
    if w.values == "halfstar":
        a = np.clip(np.round(2.0 * (3.5 + s)) / 2.0, 0.5, 5.0)
        return a.astype(np.float32)
    z = s / math.sqrt(1.64)
    if w.values == "stars":
        # Empirical quantile thresholds -> marginal (0.05, 0.10, 0.29, 0.34, 0.22) over 1..5.
        th = np.quantile(z, [0.05, 0.15, 0.44, 0.78])
        a = 1.0 + np.searchsorted(th, z, side="right")
        return a.astype(np.float32)
    if w.values == "score100":
        return np.clip(np.round(50.0 + 25.0 * z), 0.0, 100.0).astype(np.float32)
    raise ValueError(w.values)


@dataclass
class Dataset:
    workload: Workload
    row: np.ndarray      # int32 [nnz]  0-based user ids
    col: np.ndarray      # int32 [nnz]  0-based item ids
    val: np.ndarray      # float32 [nnz]
    test_row: np.ndarray
    test_col: np.ndarray
    test_val: np.ndarray
    H0: np.ndarray       # float32 [n, k] row-major, N(0, 0.01) i.e. sd 0.1

    def h0(self, k: int) -> np.ndarray:
        """H0 for another rank k (same stream; the first columns agree for any k)."""
        rng = _streams(self.workload.config_id)[4]
        return _h0(rng, self.workload.n, k)


def _h0(rng, n, k):
    kmax = max(k, 100)
    full = rng.standard_normal((n, kmax), dtype=np.float32) * np.float32(0.1)
    return np.ascontiguousarray(full[:, :k])


def generate(name: str, verbose: bool = False) -> Dataset:
    w = WORKLOADS[name]
    g_deg, g_pos, g_val, g_hold, g_h0 = _streams(w.config_id)
    total = w.nnz + w.holdout
    t0 = time.time()
    if w.kind == "uniform":
        flat = g_pos.choice(w.m * w.n, size=total, replace=False)
        rows = (flat // w.n).astype(np.int32)
        cols = (flat % w.n).astype(np.int32)
    else:
        dmax_u = w.dmax_u or w.n // 2
        dmax_i = w.dmax_i or w.m // 2
        deg_u = rank_curve(w.m, total, w.alpha_u, w.dmin_u, dmax_u)[g_deg.permutation(w.m)]
        q = rank_curve(w.n, total, w.alpha_i, w.dmin_i, dmax_i)[g_deg.permutation(w.n)]
        _log(f"{name}: degrees u[{deg_u.min()}..{deg_u.max()}] i-target[{q.min()}..{q.max()}] "
             f"({time.time() - t0:.1f}s)", verbose)
        rows, cols = _sample_positions(deg_u, q.astype(np.float64), g_pos, verbose)
    _log(f"{name}: positions done ({time.time() - t0:.1f}s)", verbose)
    vals = _values(w, rows, cols, g_val)
    _log(f"{name}: values done ({time.time() - t0:.1f}s)", verbose)
    if w.holdout:
        pick = np.zeros(total, dtype=bool)
        pick[g_hold.choice(total, size=w.holdout, replace=False)] = True
        tr, te = ~pick, pick
    else:
        tr = np.ones(total, dtype=bool)
        te = ~tr
    H0 = _h0(g_h0, w.n, w.k)
    ds = Dataset(w, np.ascontiguousarray(rows[tr]), np.ascontiguousarray(cols[tr]),
                 np.ascontiguousarray(vals[tr]), np.ascontiguousarray(rows[te]),
                 np.ascontiguousarray(cols[te]), np.ascontiguousarray(vals[te]), H0)
    assert ds.row.size == w.nnz
    _log(f"{name}: generated in {time.time() - t0:.1f}s", verbose)
    return ds


_FIELDS = ("row", "col", "val", "test_row", "test_col", "test_val", "H0")


def cache_dir() -> str:
    return os.environ.get("CCDPP_SYNTH_CACHE", os.path.join("/tmp", "ccdpp_synth_cache"))


def load(name: str, verbose: bool = False, use_cache: bool = True) -> Dataset:
    """Generate (or load from the on-disk cache) the named workload."""
    w = WORKLOADS[name]
    d = os.path.join(cache_dir(), f"{name}_v1")
    man = os.path.join(d, "manifest.json")
    if use_cache and os.path.exists(man):
        with open(man) as f:
            meta = json.load(f)
        arrs = {k: np.load(os.path.join(d, k + ".npy"), mmap_mode=None) for k in _FIELDS}
        ok = all(meta.get(k) == _digest(arrs[k]) for k in ("row", "col", "val"))
        if ok:
            _log(f"{name}: loaded from cache {d}", verbose)
            return Dataset(w, **arrs)
    ds = generate(name, verbose=verbose)
    if use_cache:
        os.makedirs(d, exist_ok=True)
        meta = {}
        for k in _FIELDS:
            a = getattr(ds, k)
            np.save(os.path.join(d, k + ".npy"), a)
            if k in ("row", "col", "val"):
                meta[k] = _digest(a)
        with open(man, "w") as f:
            json.dump(meta, f)
    return ds


def _digest(a: np.ndarray) -> str:
    h = hashlib.sha256()
    h.update(str(a.dtype).encode())
    h.update(str(a.shape).encode())
    # Sampled digest: the first, middle and last MiB plus the size.  Enough to catch a
    # stale or truncated cache without rehashing gigabytes on every load.
    b = a.view(np.uint8).reshape(-1)
    for s in (0, max(0, b.size // 2 - (1 << 19)), max(0, b.size - (1 << 20))):
        h.update(b[s:s + (1 << 20)].tobytes())
    return h.hexdigest()


def small_random(m: int, n: int, nnz: int, k: int, seed: int, allow_empty: bool = True):
    """A small uniform random problem for unit tests: distinct positions, N(0,1) values,
    H0 ~ N(0, 0.01).  Returns (row, col, val, H0)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    flat = rng.choice(m * n, size=nnz, replace=False)
    row = (flat // n).astype(np.int32)
    col = (flat % n).astype(np.int32)
    val = rng.standard_normal(nnz).astype(np.float32)
    H0 = (rng.standard_normal((n, k)) * 0.1).astype(np.float32)
    return row, col, val, H0


def lengths_problem(row_lengths, n: int, k: int, seed: int):
    """Rows with exactly the given lengths (columns drawn uniformly without replacement),
    for exercising every scheduling class of a kernel.  Returns (row, col, val, H0)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    rows, cols = [], []
    for i, L in enumerate(row_lengths):
        if L > n:
            raise ValueError("row longer than the number of columns")
        c = rng.choice(n, size=L, replace=False)
        rows.append(np.full(L, i, dtype=np.int32))
        cols.append(c.astype(np.int32))
    row = np.concatenate(rows) if rows else np.zeros(0, np.int32)
    col = np.concatenate(cols) if cols else np.zeros(0, np.int32)
    perm = rng.permutation(row.size)
    row, col = row[perm], col[perm]
    val = rng.standard_normal(row.size).astype(np.float32)
    H0 = (rng.standard_normal((n, k)) * 0.1).astype(np.float32)
    return row, col, val, H0
