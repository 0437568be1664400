"""Pins that tie the CPU oracle to the paper and to mathematics, not to itself.

Each pin takes an oracle handle and raises AssertionError when the oracle
disagrees with something fixed independently of it:

- hand-derived exact values of Eq. (3)/(4) on tiny inputs (tests/golden);
- the boundary values the paper states for f: f(empty) = 0, and f is largest
  at S = V where it equals L({e0});
- monotonicity (Definition 3) and submodularity (Definition 2, Eq. (1)) by
  brute force over every pair of subsets of a tiny ground set;
- the loss as a nearest-neighbour query answered by a k-d tree (SciPy), an
  algorithm that shares nothing with the oracle's direct loop;
- closed forms (one-point ground set, k = 1 through the norm expansion),
  exact scaling by 2, order invariance, the greedy multiset of Section IV-A;
- Algorithm 1 against a hand-worked run and against the (1 - 1/e) bound of
  Section III over brute-force optima.

The same battery runs against deliberately broken builds of the oracle
(tests/test_oracle_mutants.py) to show that each planted mistake trips a pin.
"""
from __future__ import annotations

import itertools
import json
import os

import numpy as np
from scipy.spatial import cKDTree

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")
RTOL = 1e-12


def _close(a, b, rtol=RTOL, atol=0.0, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    ok = np.all(np.abs(a - b) <= rtol * np.abs(b) + atol)
    assert ok, f"{what}: got {a!r}, expected {b!r}"


def _rng_points(seed, n, d, scale=1.0):
    rng = np.random.default_rng(seed)
    return scale * rng.standard_normal((n, d))


def pin_worked_examples(o):
    """Exact rationals of Eq. (3)/(4) for three hand-worked ground sets."""
    g = json.load(open(GOLDEN))
    for ex in g["examples"]:
        V = np.array(ex["V"], dtype=np.float64)
        num, den = ex["loss_e0"]
        _close(o.loss_e0(V), num / den, what="L({e0})")
        by_size = {}
        for item in ex["f"]:
            by_size.setdefault(len(item["S"]), []).append(item)
        for size, items in by_size.items():
            sets = np.array([it["S"] for it in items], dtype=np.int32).reshape(len(items), size)
            got = o.eval(V, sets, 1)
            want = [it["value"][0] / it["value"][1] for it in items]
            _close(got, want, atol=1e-14, what=f"f on {ex['V']} size {size}")
    gg = g["gain"]
    got = o.gain(np.array(gg["V"], float), gg["S"], gg["cands"], 1)
    _close(got, [a / b for a, b in gg["value"]], what="greedy multiset")
    gr = g["greedy"]
    S, f = o.greedy(np.array(gr["V"], float), gr["K"], 1)
    assert list(S) == gr["S"], f"greedy order {list(S)}"
    _close(f, [a / b for a, b in gr["f"]], what="greedy values")


def pin_empty_and_full(o):
    """f(empty) = 0 and f(V) = L({e0}) (statements after Eq. (4))."""
    for seed, (n, d) in enumerate([(5, 1), (9, 3), (17, 8)]):
        V = _rng_points(seed, n, d, 3.0)
        empty = o.eval(V, np.zeros((2, 0), np.int32), 1)
        assert np.all(empty == 0.0), f"f(empty) = {empty}"
        full = o.eval(V, np.arange(n, dtype=np.int32)[None, :], 1)
        _close(full, [o.loss_e0(V)], what="f(V)")


def _all_subsets(o, V):
    n = V.shape[0]
    f = np.empty(1 << n)
    for r in range(n + 1):
        combos = list(itertools.combinations(range(n), r))
        sets = np.array(combos, dtype=np.int32).reshape(len(combos), r)
        vals = o.eval(V, sets, 1)
        for c, v in zip(combos, vals):
            f[sum(1 << i for i in c)] = v
    return f


def pin_monotone_submodular_bruteforce(o):
    """Definition 3 and Eq. (1) on every subset pair of tiny ground sets."""
    for seed, (n, d) in enumerate([(6, 1), (7, 2), (7, 3)]):
        V = _rng_points(100 + seed, n, d, 2.0)
        f = _all_subsets(o, V)
        le0 = o.loss_e0(V)
        tol = 1e-12 * max(le0, 1.0)
        full = (1 << n) - 1
        assert abs(f[0]) <= tol, "f(empty) != 0"
        assert abs(f[full] - le0) <= tol, "f(V) != L({e0})"
        assert np.all(f >= -tol) and np.all(f <= le0 + tol), "f outside [0, L({e0})]"
        for B in range(1 << n):
            A = B
            while True:  # every A subset of B
                for e in range(n):
                    if B >> e & 1:
                        continue
                    dA = f[A | 1 << e] - f[A]
                    dB = f[B | 1 << e] - f[B]
                    assert dA >= -tol, f"not monotone at A={A:b}, e={e}"
                    assert dA >= dB - tol, f"not submodular: A={A:b} B={B:b} e={e}"
                if A == 0:
                    break
                A = (A - 1) & B


def pin_kdtree_nearest_neighbour(o):
    """L(S u {e0}) as squared nearest-neighbour distances from a k-d tree."""
    cases = [(300, 2, 40, 5, 1.0, 0), (257, 7, 16, 12, 4.0, 1), (120, 16, 9, 3, 0.5, 2)]
    for n, d, l, k, scale, seed in cases:
        rng = np.random.default_rng(200 + seed)
        V = scale * rng.standard_normal((n, d))
        sets = rng.integers(0, n, size=(l, k)).astype(np.int32)
        got = o.eval(V, sets, 2)
        le0 = np.mean(np.linalg.norm(V, axis=1) ** 2)
        want = []
        for s in sets:
            pts = np.vstack([np.zeros((1, d)), V[s]])
            dist, _ = cKDTree(pts).query(V, k=1)
            want.append(le0 - np.mean(dist ** 2))
        _close(got, want, rtol=1e-9, atol=1e-11 * le0, what="k-d tree")


def pin_closed_forms(o):
    """One-point ground set: f({v}) = ||v||^2.  k = 1 through the norm
    expansion ||v-s||^2 = ||v||^2 - 2<v,s> + ||s||^2, which turns
    min(||v||^2, ||v-s||^2) into ||v||^2 - 2 max(0, <v,s> - ||s||^2/2)."""
    v = np.array([[3.0, -4.0, 12.0]])
    _close(o.eval(v, [[0]], 1), [169.0], what="n=1")
    _close(o.sqnorm(np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 0.0]])), [25.0, 1.0, 0.0], what="sqnorm")
    rng = np.random.default_rng(7)
    V = rng.standard_normal((200, 5)) * 2.0
    s_idx = np.arange(0, 200, 13, dtype=np.int32)
    got = o.eval(V, s_idx[:, None], 1)
    want = []
    for s in s_idx:
        h = V @ V[s] - 0.5 * V[s] @ V[s]
        want.append(2.0 * np.mean(np.maximum(0.0, h)))
    _close(got, want, rtol=1e-10, atol=1e-12, what="k=1 clamp form")


def pin_scaling_and_order(o):
    """f(2V) = 4 f(V) exactly; slot order and duplicates leave f unchanged;
    relabelling the ground points leaves f unchanged up to summation order."""
    rng = np.random.default_rng(11)
    V = rng.standard_normal((150, 6))
    sets = rng.integers(0, 150, size=(8, 7)).astype(np.int32)
    f1 = o.eval(V, sets, 1)
    assert np.array_equal(o.eval(2.0 * V, sets, 1), 4.0 * f1), "scaling by 2"
    assert np.array_equal(o.eval(V, sets[:, ::-1].copy(), 1), f1), "slot order"
    dup = np.concatenate([sets, sets[:, :3]], axis=1)
    assert np.array_equal(o.eval(V, dup, 1), f1), "duplicate members"
    perm = rng.permutation(150)
    inv = np.argsort(perm)
    _close(o.eval(V[perm], inv[sets].astype(np.int32), 1), f1, rtol=1e-12, what="relabelling")


def pin_threads_and_gain(o):
    """Multi-thread = single-thread bitwise; greedy scoring = direct f(S u {c})."""
    rng = np.random.default_rng(12)
    V = rng.standard_normal((400, 4))
    sets = rng.integers(0, 400, size=(37, 6)).astype(np.int32)
    assert np.array_equal(o.eval(V, sets, 1), o.eval(V, sets, 4)), "threads"
    S = np.array([3, 77, 150], np.int32)
    c = np.array([0, 3, 399, 150, 12], np.int32)
    direct = o.eval(V, np.concatenate([np.tile(S, (5, 1)), c[:, None]], axis=1), 1)
    assert np.array_equal(o.gain(V, S, c, 1), direct), "gain vs eval"
    fS = o.eval(V, S[None, :], 1)[0]
    g = o.gain(V, S, c, 1)
    assert g[1] == fS and g[3] == fS, "candidate already in S"
    g0 = o.gain(V, np.zeros(0, np.int32), c, 1)
    assert np.array_equal(g0, o.eval(V, c[:, None], 1)), "empty base set"


def pin_invalid_index(o):
    """An index outside [0, n) other than the empty slot -1 poisons only its
    own set."""
    V = _rng_points(13, 20, 3)
    sets = np.array([[1, 2], [3, 20], [-2, 0], [4, 5]], np.int32)
    got = o.eval(V, sets, 1)
    assert np.isnan(got[1]) and np.isnan(got[2]), "out-of-range index"
    _close(got[[0, 3]], o.eval(V, sets[[0, 3]], 1), what="other sets")


def pin_empty_slots(o):
    """Sets of different sizes padded with -1 (blank fields) score exactly as
    the unpadded sets; an all-blank set scores f(empty) = 0."""
    rng = np.random.default_rng(14)
    V = rng.standard_normal((60, 2))
    sizes = [4, 3, 5, 0, 1]
    k = max(sizes)
    padded = np.full((len(sizes), k), -1, np.int32)
    want = []
    for j, sz in enumerate(sizes):
        members = rng.choice(60, sz, replace=False).astype(np.int32)
        padded[j, :sz] = members
        rng.shuffle(padded[j])
        want.append(o.eval(V, members[None, :], 1)[0] if sz else 0.0)
    got = o.eval(V, padded, 1)
    assert np.array_equal(got, np.asarray(want)), f"blank fields: {got} vs {want}"


def pin_greedy_guarantee(o):
    """Algorithm 1 reaches at least (1 - 1/e) of the best size-K subset
    (Section III), checked against brute force; each round's value is f of
    the prefix, and f never decreases."""
    for seed, (n, d, K) in enumerate([(8, 2, 3), (9, 3, 4), (7, 1, 2)]):
        V = _rng_points(300 + seed, n, d, 2.0)
        S, f = o.greedy(V, K, 1)
        assert len(set(S.tolist())) == K, "greedy repeated a point"
        for i in range(K):
            _close([f[i]], o.eval(V, S[None, :i + 1], 1), what="greedy prefix value")
        assert np.all(np.diff(f) >= -1e-12), "greedy values decrease"
        combos = np.array(list(itertools.combinations(range(n), K)), np.int32)
        best = o.eval(V, combos, 1).max()
        assert f[-1] >= (1 - np.exp(-1)) * best - 1e-12, "greedy below (1 - 1/e) OPT"


PINS = [pin_worked_examples, pin_empty_and_full, pin_monotone_submodular_bruteforce,
        pin_kdtree_nearest_neighbour, pin_closed_forms, pin_scaling_and_order,
        pin_threads_and_gain, pin_invalid_index, pin_empty_slots, pin_greedy_guarantee]
