"""Temporary blocks kept per stream between calls: reuse, growth, many
streams (eviction of the least recently used stream's blocks) and host
threads sharing one stream.  Every result must equal the one computed alone
(bit for bit: the kernels and their order do not depend on where the
temporary memory came from)."""
import threading

import numpy as np
import pytest

from paper_2101_08763_amd import api, synth
from test_parity_gpu import gpu_eval, say, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.load()
    return torch


def problems(torch, count, seed):
    out = []
    for i in range(count):
        n, d, l, k = 3000 + 700 * i, 24 + 8 * (i % 3), 40 + 30 * i, 3 + i % 5
        p = synth.random_problem(n, d, l, k, seed=seed + i, clusters=3)
        Vg, _ = to_gpu(torch, p.X, "fp32" if i % 2 == 0 else "fp16")
        out.append((Vg, torch.from_numpy(p.sets).cuda()))
    return out


def alone(torch, probs):
    res = []
    for Vg, s in probs:
        o = api.exemplar_eval(Vg, s)
        torch.cuda.synchronize()
        res.append(o.cpu().numpy())
    return res


def test_reuse_and_growth(torch_gpu):
    """Small, large, small again on one stream: kept blocks are reused and
    replaced by larger ones."""
    torch = torch_gpu
    probs = problems(torch, 4, 900)
    want = alone(torch, probs)
    order = [0, 3, 1, 3, 0, 2, 2, 3]
    outs = [api.exemplar_eval(*probs[i]) for i in order]
    torch.cuda.synchronize()
    for i, o in zip(order, outs):
        assert np.array_equal(o.cpu().numpy(), want[i])


def test_many_streams(torch_gpu):
    """More streams than are kept: the least recently used stream's blocks
    are released while the others keep working."""
    torch = torch_gpu
    probs = problems(torch, 3, 950)
    want = alone(torch, probs)
    streams = [torch.cuda.Stream() for _ in range(12)]
    say(f"{len(streams)} streams x {len(probs)} problems")
    outs = []
    for rep in range(2):
        for si, st in enumerate(streams):
            i = (si + rep) % len(probs)
            Vg, s = probs[i]
            with torch.cuda.stream(st):
                outs.append((i, api.exemplar_eval(Vg, s, stream=st)))
    torch.cuda.synchronize()
    for i, o in outs:
        assert np.array_equal(o.cpu().numpy(), want[i])


def test_threads_share_a_stream(torch_gpu):
    """Host threads queueing on the same stream never share a block."""
    torch = torch_gpu
    probs = problems(torch, 4, 990)
    want = alone(torch, probs)
    st = torch.cuda.Stream()
    results = [[] for _ in probs]
    errors = []

    def worker(t):
        try:
            Vg, s = probs[t]
            for _ in range(12):
                results[t].append(api.exemplar_eval(Vg, s, stream=st))
        except Exception as e:  # noqa: BLE001 -- reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(len(probs))]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for t, outs in enumerate(results):
        assert len(outs) == 12
        for o in outs:
            assert np.array_equal(o.cpu().numpy(), want[t])


def test_gain_after_eval_on_one_stream(torch_gpu):
    """Gain needs several temporary blocks at once (cache, tiles, scoring
    workspace): they must be distinct blocks of the same stream's set."""
    torch = torch_gpu
    p = synth.random_problem(5000, 40, 30, 6, seed=1010, clusters=4)
    Vg, _ = to_gpu(torch, p.X, "fp32")
    rng = np.random.default_rng(1010)
    S = torch.from_numpy(rng.choice(5000, 7, replace=False).astype(np.int32)).cuda()
    C = torch.from_numpy(rng.choice(5000, 300, replace=False).astype(np.int32)).cuda()
    g0 = api.exemplar_gain(Vg, S, C).cpu().numpy()
    e0 = gpu_eval(torch, Vg, p.sets)
    for _ in range(3):
        assert np.array_equal(api.exemplar_gain(Vg, S, C).cpu().numpy(), g0)
        assert np.array_equal(gpu_eval(torch, Vg, p.sets), e0)


def test_default_stream_is_the_current_one(torch_gpu):
    """Without `stream=`, calls queue on PyTorch's current stream."""
    torch = torch_gpu
    st = torch.cuda.Stream()
    assert (api._stream(None).value or 0) == torch.cuda.current_stream().cuda_stream
    with torch.cuda.stream(st):
        assert (api._stream(None).value or 0) == st.cuda_stream
        probs = problems(torch, 1, 1100)
        Vg, s = probs[0]
        o = api.exemplar_eval(Vg, s)
    st.synchronize()
    assert np.array_equal(o.cpu().numpy(), alone(torch, probs)[0])
