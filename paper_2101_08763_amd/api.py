"""Python binding of the C ABI in include/exemcl.h (argument marshalling only).

Every function takes torch tensors that already live on the current HIP
device, passes their device pointers and the current torch stream to
libexemcl.so, and returns without synchronising.  No computation happens
here; when the library is missing every call raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libexemcl.so")

EXEMCL_FP32, EXEMCL_FP16, EXEMCL_BF16 = 0, 1, 2
EXEMCL_OK, EXEMCL_EINVAL, EXEMCL_ENOMEM, EXEMCL_EDEVICE, EXEMCL_ESCRATCH = 0, 1, 2, 3, 4
EXEMCL_SCRATCH_BYTES = 64 << 20   # fixed scratch buffer of exemplar_eval_noalloc
PATH_NONE, PATH_VALU, PATH_MFMA = 0, 1, 2
PATH_NAMES = {PATH_NONE: "none", PATH_VALU: "valu", PATH_MFMA: "mfma"}

EXPORTED = ("exemplar_eval", "exemplar_eval_noalloc", "exemplar_eval_streamed", "exemplar_gain", "exemplar_greedy", "exemplar_sqnorm",
            "exemplar_plan",
            "exemplar_prof_enable", "exemplar_prof_read", "exemplar_strerror", "exemplar_version")


class ExemclError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} (status {status})")


_LIB = None


def load(path: str | None = None) -> ctypes.CDLL:
    """Open libexemcl.so (once; EXEMCL_LIB overrides the path).  Raises if it
    has not been built."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    p = path or os.environ.get("EXEMCL_LIB") or LIB_PATH
    if not os.path.exists(p):
        raise ImportError(f"{p} is missing: build it with `python -m paper_2101_08763_amd.build` "
                          "(or __graft_entry__.build()); there is no fallback implementation")
    lib = ctypes.CDLL(p)
    vp, i64, ip = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.exemplar_eval.argtypes = [vp, i64, i64, vp, i64, i64, ip, vp, vp]
    lib.exemplar_eval.restype = ip
    lib.exemplar_eval_noalloc.argtypes = [vp, i64, i64, vp, i64, i64, ip, vp, vp]
    lib.exemplar_eval_noalloc.restype = ip
    lib.exemplar_eval_streamed.argtypes = [vp, i64, i64, vp, i64, i64, ip, i64, vp, vp]
    lib.exemplar_eval_streamed.restype = ip
    lib.exemplar_gain.argtypes = [vp, i64, i64, vp, i64, vp, i64, vp, vp]
    lib.exemplar_gain.restype = ip
    lib.exemplar_greedy.argtypes = [vp, i64, i64, i64, vp, vp, vp]
    lib.exemplar_greedy.restype = ip
    lib.exemplar_sqnorm.argtypes = [vp, i64, i64, ip, vp, vp]
    lib.exemplar_sqnorm.restype = ip
    lib.exemplar_plan.argtypes = [i64, i64, i64, i64, ip, ctypes.POINTER(ctypes.c_int),
                                  ctypes.POINTER(ctypes.c_int64)]
    lib.exemplar_plan.restype = ip
    lib.exemplar_strerror.argtypes = [ip]
    lib.exemplar_strerror.restype = ctypes.c_char_p
    lib.exemplar_prof_enable.argtypes = [ip]
    lib.exemplar_prof_enable.restype = ip
    lib.exemplar_prof_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    lib.exemplar_prof_read.restype = ip
    lib.exemplar_version.argtypes = []
    lib.exemplar_version.restype = ip
    if path is None:
        _LIB = lib
    return lib


def strerror(status: int) -> str:
    try:
        return load().exemplar_strerror(int(status)).decode()
    except ImportError:
        return {0: "success", 1: "invalid argument", 2: "temporary device memory unavailable",
                3: "HIP runtime or kernel launch failure",
                4: "workspace needed exceeds the fixed no-allocation scratch buffer"}.get(int(status), "unknown status")


def precision_of(dtype) -> int:
    import torch
    table = {torch.float32: EXEMCL_FP32, torch.float16: EXEMCL_FP16, torch.bfloat16: EXEMCL_BF16}
    if dtype not in table:
        raise TypeError(f"V must be float32, float16 or bfloat16, not {dtype}")
    return table[dtype]


def _stream(stream):
    """The HIP stream handle of `stream`, or of the current stream of the
    current device (PyTorch's raw-stream query when it has one: it skips
    building a Stream object, a few microseconds per call)."""
    import torch
    if stream is not None:
        return ctypes.c_void_p(stream.cuda_stream)
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return ctypes.c_void_p(raw(torch.cuda.current_device()))
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check_device(*tensors):
    dev = None
    for t in tensors:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("all tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("tensors are on different devices")
    return dev


def _device_scope(dev):
    """Make `dev` current for the call; a no-op (no device switch) when it
    already is, which saves the switch and restore on every call."""
    import contextlib
    import torch
    if dev is None or dev.index == torch.cuda.current_device():
        return contextlib.nullcontext()
    return torch.cuda.device(dev)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(0)


def exemplar_eval(V, sets, out=None, stream=None):
    """out[j] = f(S_j) for the l x k int32 index matrix ``sets`` (see exemplar_eval in exemcl.h)."""
    import torch
    if V.dim() != 2 or sets.dim() != 2:
        raise ValueError("V must be n x d and sets l x k")
    if sets.dtype != torch.int32:
        raise TypeError("sets must be int32")
    prec = precision_of(V.dtype)
    n, d = V.shape
    l, k = sets.shape
    if out is None:
        out = torch.empty(l, dtype=torch.float32, device=V.device)
    elif out.dtype != torch.float32 or out.numel() != l:
        raise ValueError("out must be float32 with l elements")
    with _device_scope(_check_device(V, sets, out)):
        rc = load().exemplar_eval(_ptr(V), n, d, _ptr(sets), l, k, prec, _ptr(out), _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_eval")
    return out


def exemplar_eval_noalloc(V, sets, out, stream=None):
    """exemplar_eval with every temporary in the library's fixed scratch
    buffer (see exemplar_eval_noalloc in exemcl.h); ``out`` (float32, l
    elements, on V's device) is required, so nothing is allocated here
    either."""
    import torch
    if V.dim() != 2 or sets.dim() != 2:
        raise ValueError("V must be n x d and sets l x k")
    if sets.dtype != torch.int32:
        raise TypeError("sets must be int32")
    prec = precision_of(V.dtype)
    n, d = V.shape
    l, k = sets.shape
    if out is None or out.dtype != torch.float32 or out.numel() != l:
        raise ValueError("out must be float32 with l elements")
    with _device_scope(_check_device(V, sets, out)):
        rc = load().exemplar_eval_noalloc(_ptr(V), n, d, _ptr(sets), l, k, prec, _ptr(out), _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_eval_noalloc")
    return out


def exemplar_eval_streamed(V, sets, rows_per_block=0, out=None, device=None, stream=None):
    """out[j] = f(S_j) for V and ``sets`` in host memory (CPU tensors), with V
    streamed through the GPU in row blocks (see exemplar_eval_streamed in
    exemcl.h).  Synchronous; returns a CPU float32 tensor.  ``device`` is the
    GPU to use (default: the current one)."""
    import torch
    if V.dim() != 2 or sets.dim() != 2:
        raise ValueError("V must be n x d and sets l x k")
    if V.is_cuda or sets.is_cuda:
        raise ValueError("V and sets must be in host memory")
    if not V.is_contiguous() or not sets.is_contiguous():
        raise ValueError("tensors must be contiguous")
    if sets.dtype != torch.int32:
        raise TypeError("sets must be int32")
    prec = precision_of(V.dtype)
    n, d = V.shape
    l, k = sets.shape
    if out is None:
        out = torch.empty(l, dtype=torch.float32)
    elif out.is_cuda or out.dtype != torch.float32 or out.numel() != l or not out.is_contiguous():
        raise ValueError("out must be a contiguous host float32 tensor with l elements")
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    with torch.cuda.device(dev):
        rc = load().exemplar_eval_streamed(_ptr(V), n, d, _ptr(sets), l, k, prec, int(rows_per_block), _ptr(out),
                                           _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_eval_streamed")
    return out


def exemplar_gain(V, S, cands, out=None, stream=None):
    """out[j] = f(S u {cands[j]}) for fp32 V (see exemplar_gain in exemcl.h)."""
    import torch
    if V.dtype != torch.float32:
        raise TypeError("exemplar_gain takes float32 V")
    if S.dtype != torch.int32 or cands.dtype != torch.int32:
        raise TypeError("S and cands must be int32")
    if V.dim() != 2:
        raise ValueError("V must be n x d")
    n, d = V.shape
    l = cands.numel()
    if out is None:
        out = torch.empty(l, dtype=torch.float32, device=V.device)
    elif out.dtype != torch.float32 or out.numel() != l:
        raise ValueError("out must be float32 with one element per candidate")
    with _device_scope(_check_device(V, S if S.numel() else None, cands, out)):
        rc = load().exemplar_gain(_ptr(V), n, d, _ptr(S), S.numel(), _ptr(cands), l, _ptr(out),
                                  _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_gain")
    return out


def exemplar_greedy(V, K, S_out=None, f_out=None, stream=None):
    """Algorithm 1 for K rounds on fp32 V: returns (S_out, f_out), the point
    added in each round and f of the solution after it (see exemplar_greedy
    in exemcl.h)."""
    import torch
    if V.dtype != torch.float32:
        raise TypeError("exemplar_greedy takes float32 V")
    if V.dim() != 2:
        raise ValueError("V must be n x d")
    n, d = V.shape
    K = int(K)
    if S_out is None:
        S_out = torch.empty(max(K, 0), dtype=torch.int32, device=V.device)
    if f_out is None:
        f_out = torch.empty(max(K, 0), dtype=torch.float32, device=V.device)
    if S_out.dtype != torch.int32 or f_out.dtype != torch.float32 or S_out.numel() < K or f_out.numel() < K:
        raise ValueError("S_out must be int32 and f_out float32, with K elements each")
    with _device_scope(_check_device(V, S_out if K > 0 else None, f_out if K > 0 else None)):
        rc = load().exemplar_greedy(_ptr(V), n, d, K, _ptr(S_out), _ptr(f_out), _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_greedy")
    return S_out, f_out


def exemplar_sqnorm(V, out=None, stream=None):
    """q[i] = ||v_i||^2 in fp32."""
    import torch
    prec = precision_of(V.dtype)
    n, d = V.shape
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=V.device)
    elif out.dtype != torch.float32 or out.numel() != n:
        raise ValueError("out must be float32 with n elements")
    with _device_scope(_check_device(V, out)):
        rc = load().exemplar_sqnorm(_ptr(V), n, d, prec, _ptr(out), _stream(stream))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_sqnorm")
    return out


def exemplar_plan(n: int, d: int, l: int, k: int, precision: int = EXEMCL_FP32):
    """(path name, workspace bytes) exemplar_eval would use; host only."""
    path = ctypes.c_int(-1)
    ws = ctypes.c_int64(-1)
    rc = load().exemplar_plan(n, d, l, k, precision, ctypes.byref(path), ctypes.byref(ws))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_plan")
    return PATH_NAMES.get(path.value, str(path.value)), int(ws.value)


def exemplar_prof_enable(on=True) -> None:
    """Record HIP events around the dominant kernel of following calls:
    True or 1 = every call, an integer N > 1 = every N-th call (the first
    included), False or 0 = stop."""
    every = int(on) if not isinstance(on, bool) else (1 if on else 0)
    rc = load().exemplar_prof_enable(every)
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_prof_enable")


def exemplar_prof_read():
    """(summed kernel milliseconds, launches) recorded since the last read."""
    ms = ctypes.c_double(0.0)
    cnt = ctypes.c_int64(0)
    rc = load().exemplar_prof_read(ctypes.byref(ms), ctypes.byref(cnt))
    if rc != EXEMCL_OK:
        raise ExemclError(rc, "exemplar_prof_read")
    return float(ms.value), int(cnt.value)


def exemplar_version() -> int:
    return int(load().exemplar_version())
