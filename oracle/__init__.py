"""CPU oracle for C = A x B — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GEMM library never calls it, and it
shares no code with the library: its own fp16/bf16 codec, its own loops.

The arithmetic lives in ``oracle.c`` (plain C, binary64, k ascending; the
definition of Section 4.1).  This module only marshals numpy arrays into it.

Pins (tests/test_oracle_pins.py) tie it to facts outside itself: exact
rational brute force on tiny shapes, numpy's float64 matmul, identity and
permutation matrices, rank-1 closed forms, and exhaustive codec checks.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, F16, BF16 = 0, 1, 2
_NAMES = {"f32": F32, "fp32": F32, "float32": F32, "f16": F16, "fp16": F16,
          "float16": F16, "bf16": BF16, "bfloat16": BF16}

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = _build.LIB
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
        _build.build()
    lib = ctypes.CDLL(path)
    i64, vp, dp, ip = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int
    lib.oracle_gemm.argtypes = [ip, i64, i64, i64, i64, vp, i64, vp, i64, dp, dp, ip]
    lib.oracle_gemm.restype = ctypes.c_int
    lib.oracle_gemm_sampled.argtypes = [ip, i64, i64, i64, vp, i64, vp, i64, i64,
                                        vp, vp, vp, dp, dp]
    lib.oracle_gemm_sampled.restype = ctypes.c_int
    lib.oracle_encode.argtypes = [ip, dp, vp, i64]
    lib.oracle_encode.restype = None
    lib.oracle_decode.argtypes = [ip, vp, dp, i64]
    lib.oracle_decode.restype = None
    _lib = lib
    return lib


def dtype_code(dtype) -> int:
    if isinstance(dtype, int):
        return dtype
    return _NAMES[str(dtype).replace("torch.", "")]


def storage_np_dtype(code: int):
    return np.float32 if code == F32 else np.uint16


def _as_storage(x, code):
    x = np.ascontiguousarray(x)
    want = storage_np_dtype(code)
    if code == F16 and x.dtype == np.float16:
        x = x.view(np.uint16)
    if x.dtype == np.int16:
        x = x.view(np.uint16)
    if x.dtype != want:
        raise TypeError("oracle expects %s storage, got %s" % (want, x.dtype))
    return x


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return max(1, os.cpu_count() or 1)


def decode(bits, dtype) -> np.ndarray:
    """Stored values (fp32 array or fp16/bf16 bit patterns) -> float64."""
    code = dtype_code(dtype)
    x = _as_storage(bits, code)
    out = np.empty(x.shape, dtype=np.float64)
    _load().oracle_decode(code, x.ctypes.data, out.ctypes.data, x.size)
    return out


def encode(values, dtype) -> np.ndarray:
    """float64 -> stored values of `dtype`, round to nearest, ties to even."""
    code = dtype_code(dtype)
    v = np.ascontiguousarray(values, dtype=np.float64)
    out = np.empty(v.shape, dtype=storage_np_dtype(code))
    _load().oracle_encode(code, v.ctypes.data, out.ctypes.data, v.size)
    return out


def gemm(A, B, dtype, M=None, N=None, K=None, batch=1, sA=None, sB=None,
         threads=None, with_mag=True):
    """Reference C = A x B in float64 (plus Mag = |A| x |B|) for stored inputs.

    A, B: storage arrays (fp32, or uint16 bit patterns for fp16/bf16) holding
    `batch` matrices at element strides sA, sB (sB = 0 broadcasts B).
    Returns (Cref, Mag) shaped (batch, M, N), or (M, N) when batch == 1 and the
    inputs were 2-D.
    """
    code = dtype_code(dtype)
    a = _as_storage(A, code)
    b = _as_storage(B, code)
    squeeze = a.ndim == 2 and b.ndim == 2 and batch == 1
    if M is None:
        M, K = a.shape[-2], a.shape[-1]
    if N is None:
        N = b.shape[-1]
    if sA is None:
        sA = M * K
    if sB is None:
        sB = K * N
    need_a = (batch - 1) * sA + M * K if batch > 0 else 0
    need_b = (batch - 1) * sB + K * N if batch > 0 else 0
    if a.size < need_a or b.size < need_b:
        raise ValueError("operand storage too small for the given shape/strides")
    C = np.zeros((batch, M, N), dtype=np.float64)
    G = np.zeros((batch, M, N), dtype=np.float64) if with_mag else None
    rc = _load().oracle_gemm(code, batch, M, N, K, a.ctypes.data, sA, b.ctypes.data, sB,
                             C.ctypes.data, G.ctypes.data if with_mag else None,
                             threads or default_threads())
    if rc != 0:
        raise RuntimeError("oracle_gemm failed (rc=%d)" % rc)
    if squeeze:
        C = C[0]
        G = G[0] if with_mag else None
    return (C, G) if with_mag else C


def gemm_sampled(A, B, dtype, M, N, K, rows, cols, bats=None, sA=None, sB=None):
    """Reference values at the sampled positions only: (ref, mag) float64 vectors."""
    code = dtype_code(dtype)
    a = _as_storage(A, code)
    b = _as_storage(B, code)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    bats = np.zeros_like(rows) if bats is None else np.ascontiguousarray(bats, dtype=np.int64)
    if sA is None:
        sA = M * K
    if sB is None:
        sB = K * N
    n = rows.size
    if n:
        nb = int(bats.max()) + 1
        if a.size < (nb - 1) * sA + M * K or b.size < (nb - 1) * sB + K * N:
            raise ValueError("operand storage too small for the sampled batches")
    ref = np.empty(n, dtype=np.float64)
    mag = np.empty(n, dtype=np.float64)
    rc = _load().oracle_gemm_sampled(code, M, N, K, a.ctypes.data, sA, b.ctypes.data, sB, n,
                                     bats.ctypes.data, rows.ctypes.data, cols.ctypes.data,
                                     ref.ctypes.data, mag.ctypes.data)
    if rc != 0:
        raise RuntimeError("oracle_gemm_sampled failed (rc=%d)" % rc)
    return ref, mag
