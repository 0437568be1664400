"""GPU Greedy optimizer (Algorithm 1, exemplar_greedy) against the CPU fp64
oracle and against exemplar_gain.

A greedy run is judged round by round on the prefix the GPU chose: its pick
must be a best candidate of the oracle's scores for that prefix up to twice
the fp32 tolerance of test_parity_gpu.py (a near-tie may go either way), and
f_out must be f of the prefix within that tolerance.  Where the oracle's
best and second-best scores of every round are far apart, the sequence must
equal the oracle's own greedy run exactly.  Ties are broken by the lowest
index on both sides: exact ties are checked on duplicated points and on the
hand-worked run of tests/golden.
"""
import json
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2101_08763_amd import api, synth

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-7
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.load()
    return torch


@pytest.fixture(scope="module")
def orc():
    return oracle.load()


@pytest.fixture(autouse=True)
def _clean_env(monkeypatch):
    monkeypatch.delenv("EXEMCL_PATH", raising=False)
    monkeypatch.delenv("EXEMCL_WORKSPACE_LIMIT", raising=False)


def run_greedy(torch, Vg, K):
    S, f = api.exemplar_greedy(Vg, K)
    torch.cuda.synchronize()
    return S.cpu().numpy(), f.cpu().numpy()


def gpu_points(torch, X):
    X32 = np.ascontiguousarray(X, dtype=np.float32)
    return torch.from_numpy(X32).cuda(), X32.astype(np.float64)


def test_worked_example(torch_gpu):
    g = json.load(open(GOLDEN))["greedy"]
    Vg, _ = gpu_points(torch_gpu, np.array(g["V"], float))
    S, f = run_greedy(torch_gpu, Vg, g["K"])
    assert S.tolist() == g["S"], S
    want = np.array([a / b for a, b in g["f"]])
    assert np.all(np.abs(f - want) <= RTOL * want), (f, want)


@pytest.mark.parametrize("d", [1, 7, 100, 300])
def test_rounds_against_oracle(torch_gpu, orc, d):
    torch = torch_gpu
    n, K = 1500, 6
    p = synth.random_problem(n, d, 1, 1, seed=70 + d, clusters=5)
    Vg, X64 = gpu_points(torch, p.X)
    say(f"  greedy n={n} d={d} K={K}")
    S, f = run_greedy(torch, Vg, K)
    assert len(set(S.tolist())) == K and S.min() >= 0 and S.max() < n
    le0 = orc.loss_e0(X64)
    for i in range(K):
        prefix = S[:i]
        cands = np.setdiff1d(np.arange(n), prefix).astype(np.int32)
        sc = orc.gain(X64, prefix, cands)
        best = sc.max()
        mine = sc[np.searchsorted(cands, S[i])]
        tol = RTOL * abs(best) + ATOL * le0
        assert mine >= best - 2 * tol, f"round {i}: picked {mine} vs best {best}"
        assert abs(f[i] - mine) <= tol, f"round {i}: f_out {f[i]} vs oracle {mine}"
    assert np.all(np.diff(f) >= -RTOL * f[-1])
    # The oracle's own run: equal up to the first round without a clear winner.
    So, fo = orc.greedy(X64, K)
    for i in range(K):
        prefix = So[:i]
        cands = np.setdiff1d(np.arange(n), prefix).astype(np.int32)
        sc = np.sort(orc.gain(X64, prefix, cands))
        if sc[-1] - sc[-2] <= 4 * (RTOL * abs(sc[-1]) + ATOL * le0):
            say(f"  near-tie in round {i}: sequences compared up to it")
            break
        assert S[i] == So[i], f"round {i}: GPU {S[i]} vs oracle {So[i]}"


def test_rounds_match_gain_bitwise(torch_gpu, monkeypatch):
    """Round i's scores are exemplar_gain's for the prefix S[:i], bit for bit,
    also when the candidates are scored in several chunks."""
    torch = torch_gpu
    n, d, K = 5000, 64, 8
    p = synth.random_problem(n, d, 1, 1, seed=80, clusters=4)
    Vg, _ = gpu_points(torch, p.X)
    S, f = run_greedy(torch, Vg, K)
    allc = torch.arange(n, dtype=torch.int32, device="cuda")
    for i in range(K):
        sc = api.exemplar_gain(Vg, torch.from_numpy(S[:i].copy()).cuda(), allc)
        sc = sc.cpu().numpy()
        masked = sc.copy()
        masked[S[:i]] = -np.inf
        assert int(np.argmax(masked)) == S[i], f"round {i}"
        assert sc[S[i]] == f[i], f"round {i}: {sc[S[i]]} vs {f[i]}"
    _, ws = api.exemplar_plan(n, d, n, 1)
    monkeypatch.setenv("EXEMCL_WORKSPACE_LIMIT", str(ws // 3 + 200000))
    S2, f2 = run_greedy(torch, Vg, K)
    assert np.array_equal(S, S2) and np.array_equal(f, f2), "chunked candidates"
    monkeypatch.setenv("EXEMCL_WORKSPACE_LIMIT", "4096")
    with pytest.raises(api.ExemclError) as ei:
        run_greedy(torch, Vg, K)
    assert ei.value.status == api.EXEMCL_ENOMEM


def test_duplicates_and_all_rounds(torch_gpu, orc):
    """V holds every point twice.  The first 50 rounds take one copy of each
    (the lower index of an exact tie), the last 50 score exactly f(V) and go
    in index order; f(V) = L({e0})."""
    torch = torch_gpu
    base = np.random.default_rng(90).standard_normal((50, 5))
    X = np.concatenate([base, base])
    Vg, X64 = gpu_points(torch, X)
    S, f = run_greedy(torch, Vg, 100)
    assert sorted(S[:50].tolist()) == list(range(50)), S[:50]
    assert S[50:].tolist() == list(range(50, 100)), S[50:]
    assert np.all(f[50:] == f[49])
    le0 = orc.loss_e0(X64)
    assert abs(f[49] - le0) <= RTOL * le0
    assert np.all(np.diff(f) >= -RTOL * le0)


def test_single_point_and_repeat(torch_gpu, orc):
    torch = torch_gpu
    Vg, X64 = gpu_points(torch, np.array([[3.0, -4.0]]))
    S, f = run_greedy(torch, Vg, 1)
    assert S.tolist() == [0] and f[0] == 25.0
    p = synth.random_problem(777, 33, 1, 1, seed=91)
    Vg, _ = gpu_points(torch, p.X)
    a = run_greedy(torch, Vg, 5)
    b = run_greedy(torch, Vg, 5)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), "repeat"
