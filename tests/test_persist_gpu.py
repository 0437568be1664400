"""Persistent and plain-grid launches of the MFMA evaluation kernel give the
same bits, and so does any grouping of set groups into chunks.

Every (row block, set group) unit is computed by exactly one workgroup, in
the same order, whichever launch runs it, and each wavefront writes its own
partial-sum row; so the two launches must agree bit for bit.
EXEMCL_PERSIST=0 forces the plain grid, 2 the persistent one (read on every
launch).  The larger cases have more row blocks than the chip holds
workgroups at once, so the persistent launch runs both of its phases (whole
row blocks in step, then the even split of the rest); the small ones leave
most persistent workgroups without work.
"""
import numpy as np
import pytest

from paper_2101_08763_amd import api, synth
from test_parity_gpu import check, gpu_eval, say, to_gpu

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


@pytest.fixture(autouse=True)
def _plain_env(monkeypatch):
    monkeypatch.delenv("EXEMCL_PATH", raising=False)
    monkeypatch.delenv("EXEMCL_WG_TARGET", raising=False)


def both_launches(monkeypatch, fn):
    monkeypatch.setenv("EXEMCL_PERSIST", "0")
    plain = fn()
    monkeypatch.setenv("EXEMCL_PERSIST", "2")
    pers = fn()
    monkeypatch.delenv("EXEMCL_PERSIST")
    return plain, pers


CASES = [
    ("fp32", 32, 300_001, 70, 7),
    ("fp32", 100, 300_001, 40, 5),
    ("fp32", 128, 5_003, 70, 7),
    ("fp16", 100, 300_001, 40, 5),   # half last k-block
    ("fp16", 256, 300_001, 40, 5),
    ("bf16", 512, 5_003, 33, 3),
    ("bf16", 64, 300_001, 1, 1),      # one set group of one member
]


@pytest.mark.parametrize("prec,d,n,l,k", CASES)
def test_eval_persistent_equals_plain(torch_gpu, orc, monkeypatch, prec, d, n, l, k):
    torch = torch_gpu
    p = synth.random_problem(n, d, l, k, seed=500 + d, clusters=5)
    Vg, X64 = to_gpu(torch, p.X, prec)
    say(f"persistent vs plain: prec={prec} n={n} d={d} l={l} k={k}")
    plain, pers = both_launches(monkeypatch, lambda: gpu_eval(torch, Vg, p.sets))
    assert np.array_equal(plain, pers)
    # and both are right: a few sets against the oracle
    idx = np.unique(np.linspace(0, l - 1, 3).astype(int))
    check(pers[idx], orc.eval(X64, p.sets[idx], 8), orc.loss_e0(X64), prec, "persistent vs oracle")


def test_gain_persistent_equals_plain(torch_gpu, orc, monkeypatch):
    """The scoring kernel with a per-point initial maximum (f(S u {c}))."""
    torch = torch_gpu
    n, d = 300_001, 100
    p = synth.random_problem(n, d, 1, 1, seed=77, clusters=8)
    rng = np.random.default_rng(77)
    S = rng.choice(n, 9, replace=False).astype(np.int32)
    cands = rng.choice(n, 500, replace=False).astype(np.int32)
    Vg, X64 = to_gpu(torch, p.X, "fp32")
    Sg, cg = torch.from_numpy(S).cuda(), torch.from_numpy(cands).cuda()

    def run():
        out = api.exemplar_gain(Vg, Sg, cg)
        torch.cuda.synchronize()
        return out.cpu().numpy().astype(np.float64)

    say(f"persistent vs plain gain: n={n} d={d} |S|=9 candidates=500")
    plain, pers = both_launches(monkeypatch, run)
    assert np.array_equal(plain, pers)
    check(pers[:4], orc.gain(X64, S, cands[:4], 8), orc.loss_e0(X64), "fp32", "persistent gain vs oracle")


@pytest.mark.parametrize("prec,d,n,l,k", [("fp32", 32, 50_000, 256, 10), ("fp16", 128, 20_011, 300, 6)])
def test_chunking_target_keeps_the_bits(torch_gpu, monkeypatch, prec, d, n, l, k):
    """EXEMCL_WG_TARGET only changes how set groups are grouped into chunks
    (one workgroup walks a chunk over its rows): every set's partial sums
    come out the same, from one chunk of all groups to one chunk per group."""
    torch = torch_gpu
    p = synth.random_problem(n, d, l, k, seed=900 + d, clusters=5)
    Vg, _ = to_gpu(torch, p.X, prec)
    base = gpu_eval(torch, Vg, p.sets)
    for target in ("1", "300", "1000000"):
        monkeypatch.setenv("EXEMCL_WG_TARGET", target)
        say(f"chunking target {target}: prec={prec} n={n} d={d} l={l} k={k}")
        assert np.array_equal(gpu_eval(torch, Vg, p.sets), base)
