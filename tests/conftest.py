import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large workload, run on the GPU box")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    return oracle.load()


def strided_sample(l: int, m: int):
    """m strided positions of [0, l), the first and the last included."""
    import numpy as np
    if l <= m:
        return np.arange(l)
    return np.unique((np.arange(m) * (l - 1)) // (m - 1))


_LARGE1M = {}


@pytest.fixture(scope="session")
def large1m_ref():
    """The 1 000 000 x 256 fp16 workload (seed 4) with the oracle's values on
    a strided sample of 64 of its 2 048 sets, computed once per session on the
    rounded (fp16) values the GPU sees.  The fp32-data values of the same sets
    are computed on first use of ``fp32_values()``."""
    import oracle
    from paper_2101_08763_amd import synth
    if not _LARGE1M:
        o = oracle.load()
        p = synth.make("large1m")
        idx = strided_sample(p.workload.l, 64)
        _, X64 = synth.rounded(p.X, "fp16")
        _LARGE1M.update(p=p, idx=idx, X64=X64, want=o.eval(X64, p.sets[idx], 0), le0=o.loss_e0(X64))

        def fp32_values():
            if "want32" not in _LARGE1M:
                _LARGE1M["want32"] = o.eval(p.X.astype("float64"), p.sets[idx], 0)
            return _LARGE1M["want32"]

        _LARGE1M["fp32_values"] = fp32_values
    return _LARGE1M
