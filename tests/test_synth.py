"""The seeded workload generator (CPU only)."""
import numpy as np
import pytest

from paper_2101_08763_amd import synth


def test_tiny_shapes_and_determinism():
    a = synth.make("tiny")
    b = synth.make("tiny")
    assert a.X.shape == (1000, 8) and a.X.dtype == np.float32
    assert a.sets.shape == (16, 5) and a.sets.dtype == np.int32
    assert np.array_equal(a.X, b.X) and np.array_equal(a.sets, b.sets)
    for s in a.sets:
        assert len(set(s.tolist())) == 5 and s.min() >= 0 and s.max() < 1000


def test_mixture_has_cluster_structure():
    p = synth.make("mix50k")
    assert p.X.shape == (50_000, 32) and p.sets.shape == (256, 10)
    norms = (p.X.astype(np.float64) ** 2).sum(1)
    assert 20 * 32 < norms.mean() < 32 * 32  # means ~N(0, 25 I) plus unit noise


def test_greedy_candidates_exclude_base():
    w = synth.Workload("g", 5000, 4, 300, 19, 5, 2, "fp32", "gain")
    p = synth.make(w)
    assert p.S.shape == (19,) and p.cands.shape == (300,)
    assert not np.isin(p.cands, p.S).any()
    assert len(np.unique(p.cands)) == 300


@pytest.mark.parametrize("prec", synth.PRECISIONS)
def test_rounding_is_exact_upcast(prec):
    X = synth.make("tiny").X
    Xs, X64 = synth.rounded(X, prec)
    assert X64.dtype == np.float64 and X64.shape == X.shape
    if prec == "fp32":
        assert np.array_equal(X64, X.astype(np.float64))
    else:
        assert np.abs(X64 - X).max() < 2e-2 * np.abs(X).max()


def test_paper_sweep_series():
    """Section V-A: 15 uniformly spaced values per series, the other two
    parameters at n = 50 000, l = 5 000, k = 10."""
    n = [p["n"] for p in synth.paper_sweep("n")]
    assert n[0] == 1000 and n[-1] == 400_000 and len(n) == 15 and len(set(np.diff(n))) == 1
    k = [p["k"] for p in synth.paper_sweep("k")]
    assert k == list(range(10, 501, 35))
    l = [p["l"] for p in synth.paper_sweep("l")]
    assert l[0] == 1000 and l[-1] == 40_000 and np.all(np.abs(np.diff(np.diff(l))) <= 1)
    for p in synth.paper_sweep("l"):
        assert p["n"] == 50_000 and p["k"] == 10


def test_paper_sweep_sets_distinct_and_prefix():
    p = synth.paper_sweep_problem(300, 200, 40)
    assert p.X.shape == (300, 100) and p.sets.shape == (200, 40) and p.sets.dtype == np.int32
    for s in p.sets:
        assert len(set(s.tolist())) == 40 and s.min() >= 0 and s.max() < 300
    big = synth.paper_sweep_points(1000)
    q = synth.paper_sweep_problem(300, 200, 40, X=big)
    assert np.array_equal(p.X, q.X) and np.array_equal(p.sets, q.sets)
    full = synth.paper_sweep_problem(50, 3, 50)
    assert all(sorted(s.tolist()) == list(range(50)) for s in full.sets)
