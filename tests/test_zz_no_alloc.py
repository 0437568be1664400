"""exemplar_eval_noalloc through the C ABI: the entry point for callers that
cannot allocate device memory, whose temporaries live in the library's fixed
scratch buffer.  Its results must equal exemplar_eval's bit for bit (same
kernels, same per-set arithmetic), on consecutive calls whose sizes shrink
(the buffer keeps the previous call's contents), and match the oracle."""
import numpy as np
import pytest

from paper_2101_08763_amd import api, synth
from test_parity_gpu import check, exact, say, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.load()
    return torch


@pytest.fixture(autouse=True)
def _defaults(monkeypatch):
    for v in ("EXEMCL_PATH", "EXEMCL_WORKSPACE_LIMIT", "EXEMCL_PERSIST"):
        monkeypatch.delenv(v, raising=False)


def both(torch, V, sets_np):
    s = torch.from_numpy(np.ascontiguousarray(sets_np, dtype=np.int32)).cuda()
    ref = api.exemplar_eval(V, s)
    out = torch.full((s.shape[0],), -123.0, dtype=torch.float32, device="cuda")
    api.exemplar_eval_noalloc(V, s, out)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64)


# (n, d, l, k, precision): a batch whose workspace exceeds the 64 MiB buffer
# (processed in chunks of set groups), then smaller calls; padded rows
# (fp16 d = 100, fp32 d = 13) and rows read in place.
CALLS = [
    (200_000, 64, 4096, 16, "fp32"),
    (60_001, 100, 300, 9, "fp16"),
    (5_003, 13, 70, 7, "fp32"),
    (1_000, 256, 33, 5, "bf16"),
]


def test_noalloc_matches_eval_on_consecutive_calls(torch_gpu):
    import oracle
    torch = torch_gpu
    o = oracle.load()
    for i, (n, d, l, k, prec) in enumerate(CALLS):
        p = synth.random_problem(n, d, l, k, seed=700 + i, clusters=4)
        _, ws = api.exemplar_plan(n, d, l, k, {"fp32": 0, "fp16": 1, "bf16": 2}[prec])
        say(f"noalloc call {i}: n={n} d={d} l={l} k={k} {prec}, exemplar_eval workspace {ws / 2**20:.1f} MiB")
        Vg, X64 = to_gpu(torch, p.X, prec)
        got, ref = both(torch, Vg, p.sets)
        assert np.array_equal(got, ref), f"call {i}: differs from exemplar_eval"
        idx = np.unique((np.arange(24) * (l - 1)) // 23)
        want = o.eval(X64, p.sets[idx], 0)
        check(got[idx], want, o.loss_e0(X64), prec, f"call {i} vs oracle")
        exact(got[idx], want, f"call {i} vs oracle")
        if i == 0:
            assert ws > api.EXEMCL_SCRATCH_BYTES  # the first call runs in chunks


def test_noalloc_edge_cases(torch_gpu):
    torch = torch_gpu
    p = synth.random_problem(3001, 24, 6, 5, seed=71)
    sets = p.sets.copy()
    sets[1, 2:] = -1        # shorter set
    sets[2, :] = -1         # all empty: 0
    sets[3, 1] = 3001       # invalid: NaN
    Vg, _ = to_gpu(torch, p.X, "fp32")
    got, ref = both(torch, Vg, sets)
    assert np.array_equal(np.isnan(got), np.isnan(ref)) and np.isnan(got[3])
    assert np.array_equal(got[~np.isnan(got)], ref[~np.isnan(ref)])
    assert got[2] == 0.0
    # k = 0 and l = 0
    got0, _ = both(torch, Vg, np.zeros((4, 0), np.int32))
    assert np.array_equal(got0, np.zeros(4))
    empty = torch.empty(0, dtype=torch.float32, device="cuda")
    api.exemplar_eval_noalloc(Vg, torch.zeros((0, 3), dtype=torch.int32, device="cuda"), empty)


def test_noalloc_rejects_what_does_not_fit(torch_gpu):
    """One set group of 40 million points needs 80 MiB of partial sums: more
    than the buffer, so the call is refused with EXEMCL_ESCRATCH and queues
    nothing (out keeps its contents), while exemplar_eval takes it."""
    torch = torch_gpu
    n = 40_000_000
    V = torch.zeros((n, 1), dtype=torch.float32, device="cuda")
    s = torch.tensor([[0, 1]], dtype=torch.int32, device="cuda")
    out = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(api.ExemclError) as ei:
        api.exemplar_eval_noalloc(V, s, out)
    assert ei.value.status == api.EXEMCL_ESCRATCH
    torch.cuda.synchronize()
    assert out.item() == 7.0
    assert api.exemplar_eval(V, s).item() == 0.0
