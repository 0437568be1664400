"""CPU fp64 oracle for exemplar-based clustering -- TEST INFRASTRUCTURE ONLY.

This package wraps ``exemcl_oracle.c``, a plain C implementation of the
definitions in the paper (k-medoids loss, Eq. (3); exemplar-based clustering
f(S) = L({e0}) - L(S u {e0}), Eq. (4); evaluated as in Algorithm 2 with the
squared Euclidean distance of Section V).  Only the tests, the smoke check and
the benchmark's CPU-baseline leg may import it.  The GPU library never does:
the two share no code.

Inputs are converted to float64 exactly (fp32/fp16/bf16 values upcast without
rounding); callers that test a reduced-precision GPU run pass the *rounded*
values the GPU saw.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "exemcl_oracle.c")
_BUILD = os.path.join(_HERE, "_build")

OK, EINVAL, ENOMEM = 0, 1, 2


def build(mutant: int = 0, out_dir: str | None = None) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math); return the .so path.

    ``mutant`` > 0 plants the numbered deliberate mistake (tests only).
    """
    out_dir = out_dir or _BUILD
    os.makedirs(out_dir, exist_ok=True)
    name = "liboracle.so" if mutant == 0 else f"liboracle_m{mutant}.so"
    path = os.path.join(out_dir, name)
    tmp = f"{path}.tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", f"-DORACLE_MUTANT={int(mutant)}", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)
    return path


class Oracle:
    """ctypes handle on one build of the oracle library."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        i64 = ctypes.c_int64
        lib.oracle_eval.argtypes = [dp, i64, i64, ip, i64, i64, dp, ctypes.c_int]
        lib.oracle_eval.restype = ctypes.c_int
        lib.oracle_gain.argtypes = [dp, i64, i64, ip, i64, ip, i64, dp, ctypes.c_int]
        lib.oracle_gain.restype = ctypes.c_int
        lib.oracle_sqnorm.argtypes = [dp, i64, i64, dp]
        lib.oracle_sqnorm.restype = ctypes.c_int
        lib.oracle_loss_e0.argtypes = [dp, i64, i64]
        lib.oracle_loss_e0.restype = ctypes.c_double
        lib.oracle_greedy.argtypes = [dp, i64, i64, i64, ip, dp, ctypes.c_int]
        lib.oracle_greedy.restype = ctypes.c_int
        lib.oracle_threads.argtypes = [ctypes.c_int]
        lib.oracle_threads.restype = ctypes.c_int
        self._lib = lib
        self.path = path

    @staticmethod
    def _mat(V) -> np.ndarray:
        V = np.ascontiguousarray(np.asarray(V, dtype=np.float64))
        if V.ndim == 1:
            V = V.reshape(-1, 1)
        if V.ndim != 2:
            raise ValueError("V must be n x d")
        return V

    @staticmethod
    def _p(a, t):
        return a.ctypes.data_as(ctypes.POINTER(t))

    def threads(self, nthreads: int = 0) -> int:
        return int(self._lib.oracle_threads(int(nthreads)))

    def eval(self, V, sets, nthreads: int = 0) -> np.ndarray:
        """f(S_j) for every row of ``sets`` (l x k int indices into V)."""
        V = self._mat(V)
        sets = np.ascontiguousarray(np.asarray(sets, dtype=np.int32))
        if sets.ndim != 2:
            raise ValueError("sets must be l x k")
        l, k = sets.shape
        out = np.full(l, np.nan, dtype=np.float64)
        rc = self._lib.oracle_eval(self._p(V, ctypes.c_double), V.shape[0], V.shape[1],
                                   self._p(sets, ctypes.c_int32), l, k,
                                   self._p(out, ctypes.c_double), int(nthreads))
        if rc != OK:
            raise RuntimeError(f"oracle_eval failed with status {rc}")
        return out

    def gain(self, V, S, cands, nthreads: int = 0) -> np.ndarray:
        """f(S u {c}) for every candidate index c."""
        V = self._mat(V)
        S = np.ascontiguousarray(np.asarray(S, dtype=np.int32).reshape(-1))
        cands = np.ascontiguousarray(np.asarray(cands, dtype=np.int32).reshape(-1))
        out = np.full(cands.shape[0], np.nan, dtype=np.float64)
        rc = self._lib.oracle_gain(self._p(V, ctypes.c_double), V.shape[0], V.shape[1],
                                   self._p(S, ctypes.c_int32), S.shape[0],
                                   self._p(cands, ctypes.c_int32), cands.shape[0],
                                   self._p(out, ctypes.c_double), int(nthreads))
        if rc != OK:
            raise RuntimeError(f"oracle_gain failed with status {rc}")
        return out

    def greedy(self, V, K: int, nthreads: int = 0):
        """Algorithm 1: (indices added per round, f(S_i) after each round)."""
        V = self._mat(V)
        S = np.zeros(K, dtype=np.int32)
        f = np.zeros(K, dtype=np.float64)
        rc = self._lib.oracle_greedy(self._p(V, ctypes.c_double), V.shape[0], V.shape[1], int(K),
                                     self._p(S, ctypes.c_int32), self._p(f, ctypes.c_double), int(nthreads))
        if rc != OK:
            raise RuntimeError(f"oracle_greedy failed with status {rc}")
        return S, f

    def sqnorm(self, V) -> np.ndarray:
        V = self._mat(V)
        q = np.empty(V.shape[0], dtype=np.float64)
        rc = self._lib.oracle_sqnorm(self._p(V, ctypes.c_double), V.shape[0], V.shape[1],
                                     self._p(q, ctypes.c_double))
        if rc != OK:
            raise RuntimeError(f"oracle_sqnorm failed with status {rc}")
        return q

    def loss_e0(self, V) -> float:
        V = self._mat(V)
        return float(self._lib.oracle_loss_e0(self._p(V, ctypes.c_double), V.shape[0], V.shape[1]))

    def timed_eval(self, V, sets, nthreads: int = 0):
        """(values, seconds) with the clock around the evaluation call only."""
        V = self._mat(V)
        sets = np.ascontiguousarray(np.asarray(sets, dtype=np.int32))
        t0 = time.perf_counter()
        out = self.eval(V, sets, nthreads)
        return out, time.perf_counter() - t0


_DEFAULT: Oracle | None = None


def load(rebuild: bool = False) -> Oracle:
    """The unmutated oracle, built on first use (or when ``rebuild``)."""
    global _DEFAULT
    if _DEFAULT is None or rebuild:
        path = os.path.join(_BUILD, "liboracle.so")
        if rebuild or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            path = build()
        _DEFAULT = Oracle(path)
    return _DEFAULT


def load_mutant(mutant: int, out_dir: str) -> Oracle:
    return Oracle(build(mutant, out_dir))
