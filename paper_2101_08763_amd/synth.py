"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module only draws random numbers; it holds none of the method's
arithmetic, and neither the GPU library nor the oracle imports it.  The paper
evaluates on randomly generated problems whose distribution it does not state
(Section V); the named workloads below stand in for them.

Draw order for every workload (NumPy PCG64, ``numpy.random.default_rng(seed)``):

1. cluster means, shape (C, d): ``5 * standard_normal`` (covariance 25 I);
2. cluster labels, shape (n,): ``integers(0, C)``;
3. points: ``means[labels] + standard_normal((n, d))`` (sigma = 1);
   i.i.d. workloads skip steps 1-2 and use ``standard_normal((n, d))``;
4. sets: one ``choice(n, k, replace=False)`` per set, in set order (the
   paper-shaped sweep below draws its larger batches differently).
   Greedy workloads draw the base set S with ``choice(n, |S|)`` and then
   ``choice(n, l + |S|)`` candidates, drop the ones in S and keep the first l.

All normals are drawn directly as float32.  Reduced-precision runs round the
same float32 array to fp16 / bf16 (round-to-nearest-even).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PRECISIONS = ("fp32", "fp16", "bf16")


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    d: int
    l: int
    k: int                      # set size for eval; |S| for gain
    clusters: int               # 0 = i.i.d. N(0, 1)
    seed: int
    precision: str = "fp32"
    mode: str = "eval"          # "eval" or "gain"
    note: str = ""

    @property
    def terms(self) -> int:
        """(point, exemplar) pairs one call scores: n*k*l, with k+1 per gain set."""
        kk = self.k + 1 if self.mode == "gain" else self.k
        return self.n * kk * self.l


WORKLOADS = {
    "tiny": Workload("tiny", 1000, 8, 16, 5, 0, 0, "fp32", "eval",
                     "1 000 points, d=8, i.i.d. N(0,1); 16 sets of 5"),
    "mix50k": Workload("mix50k", 50_000, 32, 256, 10, 10, 1, "fp32", "eval",
                       "50 000 points, d=32, 10-Gaussian mixture; 256 sets of 10"),
    "greedy200k": Workload("greedy200k", 200_000, 100, 4096, 19, 50, 2, "fp32", "gain",
                           "200 000 points, d=100, 50-Gaussian mixture; |S|=19, 4096 candidates"),
    "large1m": Workload("large1m", 1_000_000, 256, 2048, 32, 100, 4, "fp16", "eval",
                        "1 000 000 points, d=256, 100-Gaussian mixture, fp16; 2048 sets of 32"),
}
# The d/precision sweep; bf16 storage is measured beside the fp16 lines.
for _d in (2, 16, 128, 512):
    for _p in ("fp32", "fp16", "bf16"):
        _w = Workload(f"sweep_d{_d}_{_p}", 100_000, _d, 1024, 16, 0, 3, _p, "eval",
                      f"100 000 points, d={_d}, i.i.d. N(0,1), {_p}; 1024 sets of 16")
        WORKLOADS[_w.name] = _w


@dataclass
class Problem:
    workload: Workload
    X: np.ndarray                      # (n, d) float32, before any rounding
    sets: np.ndarray | None = None     # (l, k) int32 (eval)
    S: np.ndarray | None = None        # (|S|,) int32 (gain)
    cands: np.ndarray | None = None    # (l,) int32 (gain)
    extra: dict = field(default_factory=dict)


def points(rng: np.random.Generator, n: int, d: int, clusters: int) -> np.ndarray:
    if clusters <= 0:
        return rng.standard_normal((n, d), dtype=np.float32)
    means = 5.0 * rng.standard_normal((clusters, d), dtype=np.float32)
    labels = rng.integers(0, clusters, size=n)
    X = rng.standard_normal((n, d), dtype=np.float32)
    X += means[labels]
    return X


def draw_sets(rng: np.random.Generator, n: int, l: int, k: int) -> np.ndarray:
    sets = np.empty((l, k), dtype=np.int32)
    for j in range(l):
        sets[j] = rng.choice(n, size=k, replace=False)
    return sets


def draw_greedy(rng: np.random.Generator, n: int, base: int, l: int):
    S = rng.choice(n, size=base, replace=False).astype(np.int32)
    pool = rng.choice(n, size=min(n, l + base), replace=False).astype(np.int32)
    cands = pool[~np.isin(pool, S)][:l]
    return S, np.ascontiguousarray(cands, dtype=np.int32)


def make(workload: Workload | str) -> Problem:
    w = WORKLOADS[workload] if isinstance(workload, str) else workload
    rng = np.random.default_rng(w.seed)
    X = points(rng, w.n, w.d, w.clusters)
    if w.mode == "gain":
        S, cands = draw_greedy(rng, w.n, w.k, w.l)
        return Problem(w, X, S=S, cands=cands)
    return Problem(w, X, sets=draw_sets(rng, w.n, w.l, w.k))


def random_problem(n: int, d: int, l: int, k: int, seed: int, clusters: int = 0,
                   replace: bool = False) -> Problem:
    """Small ad-hoc problem with the same recipe (tests)."""
    rng = np.random.default_rng(seed)
    X = points(rng, n, d, clusters)
    if replace or k > n:
        sets = rng.integers(0, n, size=(l, k)).astype(np.int32)
    else:
        sets = draw_sets(rng, n, l, k)
    w = Workload(f"random_n{n}_d{d}_l{l}_k{k}_s{seed}", n, d, l, k, clusters, seed)
    return Problem(w, X, sets=sets)


def rounded(X: np.ndarray, precision: str):
    """(storage array for the GPU, exact float64 copy of the values it holds).

    fp32 keeps X; fp16 rounds with NumPy (RNE); bf16 rounds with torch (RNE)
    and returns a torch CPU tensor as storage.
    """
    if precision == "fp32":
        Xs = np.ascontiguousarray(X, dtype=np.float32)
        return Xs, Xs.astype(np.float64)
    if precision == "fp16":
        Xs = np.ascontiguousarray(X.astype(np.float16))
        return Xs, Xs.astype(np.float64)
    if precision == "bf16":
        import torch
        Xs = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).to(torch.bfloat16)
        return Xs, Xs.to(torch.float64).numpy()
    raise ValueError(f"unknown precision {precision!r}")


# ---------------------------------------------------------------------------
# The scaling experiment of Section V-A: d = 100, a default problem of
# n = 50 000 points, l = 5 000 sets, k = 10 members, and three series that
# vary one of n, l, k over 15 uniformly spaced values of an interval while the
# other two keep their defaults.  The paper states no distribution; points
# are i.i.d. N(0, 1) here, ``default_rng(seed).standard_normal((n, 100))``
# (so every n of the series is a prefix of the largest array).  Sets come
# from ``default_rng(seed + 1)``: ``integers(0, n, (l, k))``, then, for the
# rows that still hold a repeat (in row order), every member equal to an
# earlier one of its row (ranked by a stable sort of the row) is redrawn with
# ``integers(0, n)`` in row-major order, until every row holds k distinct
# points.
# ---------------------------------------------------------------------------
PAPER_SWEEP_D = 100
PAPER_SWEEP_DEFAULT = {"n": 50_000, "l": 5_000, "k": 10}
PAPER_SWEEP_RANGE = {"n": (1_000, 400_000), "l": (1_000, 40_000), "k": (10, 500)}
PAPER_SWEEP_POINTS = 15
PAPER_SWEEP_SEED = 5


def paper_sweep(axis: str) -> list[dict]:
    """The 15 (n, l, k) points of one series of Section V-A."""
    lo, hi = PAPER_SWEEP_RANGE[axis]
    out = []
    for v in np.linspace(lo, hi, PAPER_SWEEP_POINTS):
        pt = dict(PAPER_SWEEP_DEFAULT)
        pt[axis] = int(round(float(v)))
        out.append(pt)
    return out


def draw_sets_redraw(rng: np.random.Generator, n: int, l: int, k: int) -> np.ndarray:
    if k > n:
        raise ValueError("k distinct members need k <= n")
    sets = rng.integers(0, n, size=(l, k), dtype=np.int64)
    rows = np.arange(l)
    while rows.size:
        sub = sets[rows]
        order = np.argsort(sub, axis=1, kind="stable")
        srt = np.take_along_axis(sub, order, axis=1)
        rep_sorted = np.zeros(srt.shape, dtype=bool)
        rep_sorted[:, 1:] = srt[:, 1:] == srt[:, :-1]
        bad = rep_sorted.any(axis=1)
        if not bad.any():
            break
        rep = np.zeros_like(rep_sorted)
        np.put_along_axis(rep, order, rep_sorted, axis=1)
        sub[rep] = rng.integers(0, n, size=int(rep.sum()))
        sets[rows] = sub
        rows = rows[bad]
    return np.ascontiguousarray(sets, dtype=np.int32)


def paper_sweep_points(n: int, seed: int = PAPER_SWEEP_SEED) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal((n, PAPER_SWEEP_D), dtype=np.float32)


def paper_sweep_problem(n: int, l: int, k: int, seed: int = PAPER_SWEEP_SEED,
                        X: np.ndarray | None = None) -> Problem:
    """One point of the series; ``X`` may be the points of a larger n of the
    same seed (its first n rows are used)."""
    X = paper_sweep_points(n, seed) if X is None else np.ascontiguousarray(X[:n])
    if X.shape != (n, PAPER_SWEEP_D):
        raise ValueError("X holds fewer than n points")
    w = Workload(f"paper_n{n}_l{l}_k{k}", n, PAPER_SWEEP_D, l, k, 0, seed, "fp32", "eval",
                 f"{n} points, d=100, i.i.d. N(0,1); {l} sets of {k} (Section V-A series)")
    return Problem(w, X, sets=draw_sets_redraw(np.random.default_rng(seed + 1), n, l, k))
