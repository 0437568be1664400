"""The pair loop of the fp16/bf16 kernel for d <= 16 (32x32x16 tiles of one
k-block and one member each; two tiles of a set group folded with one max3
per element, a lone tile with one max).

Stages hold an even number of tiles (20 here), so only a set group of odd
k ends with a lone tile; k = 2 fits a single pair, k = 32 spans two stages,
and with EXEMCL_WG_TARGET=1 a workgroup walks every set group, so groups end
inside stages and, for odd k, pairs restart mid-stage.  Every result is compared with the oracle on the rounded
inputs at EXACT_RTOL.

The clamp-form value is a maximum over a set's members, so repeating a
member changes nothing: a set of odd k and the same set with one member
repeated (k + 1, folded as pairs only) give the same bits, on the same row
blocks and partial-sum order.
"""
import numpy as np
import pytest

from paper_2101_08763_amd import api, synth
from test_parity_gpu import check, exact, gpu_eval, say, to_gpu

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
    for v in ("EXEMCL_PATH", "EXEMCL_WG_TARGET", "EXEMCL_PERSIST"):
        monkeypatch.delenv(v, raising=False)


@pytest.mark.parametrize("target", ["default", "1"])
@pytest.mark.parametrize("k", [2, 4, 6, 16, 32])
@pytest.mark.parametrize("d", [2, 13, 16])
@pytest.mark.parametrize("prec", ["fp16", "bf16"])
def test_pairs_exact(torch_gpu, orc, monkeypatch, prec, d, k, target):
    torch = torch_gpu
    if target != "default":
        monkeypatch.setenv("EXEMCL_WG_TARGET", target)
    n, l = 2003, 75
    p = synth.random_problem(n, d, l, k, seed=7100 + 37 * d + k, clusters=4)
    say(f"pair loop: prec={prec} n={n} d={d} l={l} k={k} wg_target={target}")
    Vg, X64 = to_gpu(torch, p.X, prec)
    got = gpu_eval(torch, Vg, p.sets)
    want = orc.eval(X64, p.sets, 8)
    check(got, want, orc.loss_e0(X64), prec, f"d={d} k={k}")
    exact(got, want, f"{prec} d={d} k={k}")


@pytest.mark.parametrize("target", ["default", "1"])
@pytest.mark.parametrize("k", [1, 5, 15, 31])
@pytest.mark.parametrize("prec", ["fp16", "bf16"])
def test_repeated_member_keeps_the_bits(torch_gpu, monkeypatch, prec, k, target):
    torch = torch_gpu
    if target != "default":
        monkeypatch.setenv("EXEMCL_WG_TARGET", target)
    n, d, l = 40_009, 16, 200
    p = synth.random_problem(n, d, l, k, seed=7300 + k, clusters=6)
    dup = np.concatenate([p.sets, p.sets[:, -1:]], axis=1)  # one member twice: k + 1
    say(f"repeated member: prec={prec} n={n} l={l} k={k} / {k + 1} wg_target={target}")
    Vg, _ = to_gpu(torch, p.X, prec)
    assert np.array_equal(gpu_eval(torch, Vg, p.sets), gpu_eval(torch, Vg, dup))


def test_pairs_persistent_equals_plain(torch_gpu, orc, monkeypatch):
    torch = torch_gpu
    n, d, l, k = 300_001, 16, 100, 16
    p = synth.random_problem(n, d, l, k, seed=7500, clusters=8)
    Vg, X64 = to_gpu(torch, p.X, "fp16")
    say(f"pair loop, persistent vs plain: n={n} d={d} l={l} k={k}")
    monkeypatch.setenv("EXEMCL_PERSIST", "0")
    plain = gpu_eval(torch, Vg, p.sets)
    monkeypatch.setenv("EXEMCL_PERSIST", "2")
    pers = gpu_eval(torch, Vg, p.sets)
    assert np.array_equal(plain, pers)
    idx = np.array([0, l // 2, l - 1])
    exact(pers[idx], orc.eval(X64, p.sets[idx], 8), "persistent, sampled sets vs oracle")
