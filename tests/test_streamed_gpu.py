"""Out-of-core evaluation (V in host memory, streamed in row blocks) against
the CPU fp64 oracle and against the in-HBM path, through the C ABI.

Same tolerances as tests/test_parity_gpu.py.  The streamed result groups the
sum over points by row blocks, so it equals exemplar_eval within tolerance,
not bitwise; index handling (NaN sets, empty slots) is exact.
"""
import numpy as np
import pytest

from paper_2101_08763_amd import api, synth
from test_parity_gpu import ATOL, RTOL, check, exact, gpu_eval, say, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.load()
    return torch


@pytest.fixture(scope="module")
def orc():
    import oracle
    return oracle.load()


def host_tensors(torch, X, sets, prec, pinned=False):
    Xs, X64 = synth.rounded(X, prec)
    V = (Xs if isinstance(Xs, torch.Tensor) else torch.from_numpy(Xs)).contiguous()
    if pinned:
        V = V.pin_memory()
    S = torch.from_numpy(np.ascontiguousarray(sets, dtype=np.int32))
    return V, S, X64


def streamed(V, S, rows):
    return api.exemplar_eval_streamed(V, S, rows_per_block=rows).numpy().astype(np.float64)


# Several blocks with a ragged last one, every storage type, dimensions with
# and without padded rows (and a half last k-block for fp16/bf16 at d = 100).
@pytest.mark.parametrize("prec", ["fp32", "fp16", "bf16"])
@pytest.mark.parametrize("d", [8, 33, 100, 128, 600])
def test_streamed_matches_oracle(torch_gpu, orc, prec, d):
    torch = torch_gpu
    n, l, k = 5003, 70, 7
    p = synth.random_problem(n, d, l, k, seed=3000 + d, clusters=4)
    V, S, X64 = host_tensors(torch, p.X, p.sets, prec)
    say(f"streamed prec={prec} n={n} d={d} l={l} k={k}")
    want = orc.eval(X64, p.sets, 8)
    le0 = orc.loss_e0(X64)
    for rows in (600, 2048, 0):
        check(streamed(V, S, rows), want, le0, prec, f"d={d} rows_per_block={rows}")


def test_streamed_pinned_and_pageable_agree(torch_gpu, orc):
    """Pinned V is copied to the device directly, pageable V through the
    library's staging buffers: same blocks, same kernels, bitwise the same."""
    torch = torch_gpu
    p = synth.random_problem(7000, 64, 40, 9, seed=31, clusters=3)
    Vp, S, X64 = host_tensors(torch, p.X, p.sets, "fp32", pinned=True)
    Vq, _, _ = host_tensors(torch, p.X, p.sets, "fp32")
    a, b = streamed(Vp, S, 1000), streamed(Vq, S, 1000)
    assert np.array_equal(a, b)
    check(a, orc.eval(X64, p.sets, 8), orc.loss_e0(X64), "fp32", "pinned")


def test_streamed_agrees_with_device_path(torch_gpu):
    torch = torch_gpu
    p = synth.random_problem(20000, 128, 300, 10, seed=32, clusters=6)
    for prec in ("fp32", "fp16"):
        V, S, _ = host_tensors(torch, p.X, p.sets, prec)
        Vg, _ = to_gpu(torch, p.X, prec)
        dev = gpu_eval(torch, Vg, p.sets)
        got = streamed(V, S, 4096)
        err = np.abs(got - dev)
        say(f"  {prec}: streamed vs exemplar_eval max rel {np.max(err / np.abs(dev)):.2e}")
        assert np.all(err <= RTOL[prec] * np.abs(dev) + ATOL[prec] * float(np.max(dev)))


def test_streamed_index_edge_cases(torch_gpu, orc):
    """Empty slots, an all-empty set, invalid indices (NaN only for their own
    set), duplicates, n = 1, k = 0."""
    torch = torch_gpu
    n, d = 3001, 24
    p = synth.random_problem(n, d, 6, 5, seed=33)
    sets = p.sets.copy()
    sets[1, 2:] = -1          # shorter set
    sets[2, :] = -1           # all empty: f = 0
    sets[3, 1] = n            # invalid: NaN
    sets[4, 0] = -7           # invalid: NaN
    sets[5, :] = sets[5, 0]   # duplicates
    V, S, X64 = host_tensors(torch, p.X, sets, "fp32")
    got = streamed(V, S, 512)
    want = orc.eval(X64, sets, 8)
    assert np.isnan(got[3]) and np.isnan(got[4]) and not np.isnan(got[[0, 1, 2, 5]]).any()
    assert got[2] == 0.0
    check(got, want, orc.loss_e0(X64), "fp32", "edge cases")
    # n = 1 with S = {v}: f = ||v||^2
    v = np.array([[1.5, -2.0, 0.25]], np.float32)
    V1, S1, _ = host_tensors(torch, v, np.zeros((1, 1), np.int32), "fp32")
    assert abs(streamed(V1, S1, 0)[0] - float((v.astype(np.float64) ** 2).sum())) <= 1e-6
    # k = 0: every set scores 0
    V0, S0, _ = host_tensors(torch, p.X, np.zeros((4, 0), np.int32), "fp32")
    assert np.array_equal(streamed(V0, S0, 0), np.zeros(4))


def test_streamed_workspace_limit(torch_gpu, monkeypatch):
    torch = torch_gpu
    p = synth.random_problem(4000, 32, 20, 4, seed=34)
    V, S, _ = host_tensors(torch, p.X, p.sets, "fp32")
    monkeypatch.setenv("EXEMCL_WORKSPACE_LIMIT", "4096")
    with pytest.raises(api.ExemclError) as ei:
        streamed(V, S, 0)
    assert ei.value.status == api.EXEMCL_ENOMEM


@pytest.mark.slow
def test_streamed_large1m_sampled(torch_gpu, large1m_ref):
    """The 1 000 000-point d = 256 fp16 workload streamed from host memory in
    blocks of 131 072 points, on the strided sample of 64 of its 2 048 sets
    (first and last included) that the in-HBM test checks."""
    torch = torch_gpu
    r = large1m_ref
    pr, idx = r["p"], r["idx"]
    V, S, _ = host_tensors(torch, pr.X, pr.sets[idx], "fp16")
    say(f"streamed large1m: {len(idx)} sets")
    got = streamed(V, S, 131072)
    check(got, r["want"], r["le0"], "fp16", "large1m streamed")
    exact(got, r["want"], "large1m streamed vs rounded-input oracle")
