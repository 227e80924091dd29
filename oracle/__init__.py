"""CPU oracle for C = A x B and the 2-D convolution — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GEMM library never calls it, and it
shares no code with the library: its own fp16/bf16 codec, its own loops.

The arithmetic lives in ``oracle.c`` (plain C, binary64, k ascending; the
definition of Section 4.1; the direct convolution of Section 7.1, Table 4).
This module only marshals numpy arrays into it.

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
    lib.oracle_gemm_sampled_mt.argtypes = [ip, i64, i64, i64, vp, i64, vp, i64, i64,
                                           vp, vp, vp, dp, dp, ip]
    lib.oracle_gemm_sampled_mt.restype = ctypes.c_int
    lib.oracle_conv2d.argtypes = [ip] + [i64] * 13 + [vp, vp, dp, dp, ip]
    lib.oracle_conv2d.restype = ctypes.c_int
    lib.oracle_conv_out_dim.argtypes = [i64] * 5
    lib.oracle_conv_out_dim.restype = i64
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


def gemm_sampled(A, B, dtype, M, N, K, rows, cols, bats=None, sA=None, sB=None, threads=1):
    """Reference values at the sampled positions only: (ref, mag) float64 vectors.

    threads > 1 shares the samples over that many threads (visited grouped by
    batch and column, so a strided column of B is decoded once per group);
    every value is the same binary64 sum either way."""
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
    if threads is None or threads > 1:
        order = np.lexsort((rows, cols, bats))
        r_ = np.ascontiguousarray(rows[order])
        c_ = np.ascontiguousarray(cols[order])
        b_ = np.ascontiguousarray(bats[order])
        ref_s = np.empty(n, dtype=np.float64)
        mag_s = np.empty(n, dtype=np.float64)
        rc = _load().oracle_gemm_sampled_mt(code, M, N, K, a.ctypes.data, sA, b.ctypes.data, sB, n,
                                            b_.ctypes.data, r_.ctypes.data, c_.ctypes.data,
                                            ref_s.ctypes.data, mag_s.ctypes.data, threads or default_threads())
        ref[order] = ref_s
        mag[order] = mag_s
    else:
        rc = _load().oracle_gemm_sampled(code, M, N, K, a.ctypes.data, sA, b.ctypes.data, sB, n,
                                         bats.ctypes.data, rows.ctypes.data, cols.ctypes.data,
                                         ref.ctypes.data, mag.ctypes.data)
    if rc != 0:
        raise RuntimeError("oracle_gemm_sampled failed (rc=%d)" % rc)
    return ref, mag


def conv_out_dim(size, k, stride, pad, dil):
    """Output extent of a convolution along one axis (0 if nothing fits)."""
    return int(_load().oracle_conv_out_dim(size, k, stride, pad, dil))


def conv2d(x, w, dtype, stride=(1, 1), pad=(0, 0), dil=(1, 1), threads=None, with_mag=True):
    """Reference 2-D convolution in float64 (plus Mag) for stored inputs.

    x: N x H x W x Cin storage; w: KH x KW x Cin x Cout storage.  Returns
    (out, Mag) shaped N x OH x OW x Cout (or out alone without Mag).
    """
    code = dtype_code(dtype)
    xs = _as_storage(x, code)
    ws = _as_storage(w, code)
    if xs.ndim != 4 or ws.ndim != 4 or xs.shape[3] != ws.shape[2]:
        raise ValueError("x must be N x H x W x Cin and w KH x KW x Cin x Cout")
    N, H, W, Cin = xs.shape
    KH, KW, _, Cout = ws.shape
    OH = conv_out_dim(H, KH, stride[0], pad[0], dil[0])
    OW = conv_out_dim(W, KW, stride[1], pad[1], dil[1])
    out = np.zeros((N, OH, OW, Cout), dtype=np.float64)
    mag = np.zeros((N, OH, OW, Cout), dtype=np.float64) if with_mag else None
    rc = _load().oracle_conv2d(code, N, H, W, Cin, Cout, KH, KW, stride[0], stride[1], pad[0], pad[1],
                               dil[0], dil[1], xs.ctypes.data, ws.ctypes.data, out.ctypes.data,
                               mag.ctypes.data if with_mag else None, threads or default_threads())
    if rc != 0:
        raise RuntimeError("oracle_conv2d failed (rc=%d)" % rc)
    return (out, mag) if with_mag else out
