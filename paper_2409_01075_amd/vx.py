"""Thin ctypes binding of libvx.so (argument marshalling only).

The names mirror the C ABI in include/vx.h.  Every GEMM runs in the library's
HIP kernels; there is no fallback: if libvx.so is missing or cannot be loaded
this module raises.  PyTorch is used only to hand over device pointers and the
current HIP stream.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvx.so")

VX_F32, VX_F16, VX_BF16 = 0, 1, 2
STATUS = {0: "VX_OK", 1: "VX_ERR_INVALID_ARG", 2: "VX_ERR_UNSUPPORTED_DTYPE",
          3: "VX_ERR_NO_CANDIDATE", 4: "VX_ERR_WORKSPACE", 5: "VX_ERR_HIP"}


class vx_hwinfo(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_char * 32)] + [
        (n, ctypes.c_int) for n in ("num_cu", "num_xcd", "simd_per_cu", "wave_size", "max_threads_per_wg",
                                    "lds_bytes_per_cu", "vgprs_per_lane", "max_waves_per_simd")] + [
        (n, ctypes.c_double) for n in ("clock_ghz", "hbm_gbps", "l2_bytes_per_xcd", "mall_bytes",
                                       "mfma_flop_clk_cu_f16", "mfma_flop_clk_cu_f32", "l2_bytes_clk_cu",
                                       "lds_bytes_clk_cu", "mem_latency_ns", "atomic_latency_ns",
                                       "launch_ns")]


class vx_kernel_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in (
        "id", "dtype", "mb", "nb", "kb", "wm", "wn", "mfma_m", "mfma_n", "mfma_k", "vec", "family", "stages",
        "threads",
        "lds_bytes", "vgprs", "agprs", "sgprs", "scratch_bytes", "enabled", "k_max", "op", "align", "schedule")]


class vx_conv2d_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("n", "h", "w", "c_in", "c_out", "kh", "kw", "stride_h", "stride_w",
                                              "pad_h", "pad_w", "dil_h", "dil_w")] + [("dtype", ctypes.c_int)]


class vx_plan(ctypes.Structure):
    _fields_ = [("kernel_id", ctypes.c_int), ("split_k", ctypes.c_int), ("k_per_split", ctypes.c_int),
                ("c_vec", ctypes.c_int), ("tiles_m", ctypes.c_int64), ("tiles_n", ctypes.c_int64),
                ("grid", ctypes.c_int64), ("dp_tiles", ctypes.c_int64), ("group_m", ctypes.c_int),
                ("workspace_bytes", ctypes.c_size_t),
                ("predicted_ns", ctypes.c_double), ("kernel", vx_kernel_info)]


class VxError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        super().__init__("%s%s" % (what + ": " if what else "", STATUS.get(status, status)))


_lib = None


def lib():
    """Loads libvx.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libvx.so not built: run `python -m paper_2409_01075_amd.build` "
                           "(or __graft_entry__.build())")
    # PyTorch bundles its own HIP runtime (soname libamdhip64.so.7, but its
    # libraries ask for it as libamdhip64.so).  Loaded first, it also
    # satisfies this library's libamdhip64.so.7; loaded after this library,
    # it would come in as a second HIP runtime beside the system one, and the
    # two would not share devices, streams or allocations.  So torch goes first.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    L.vx_gemm.argtypes = [i64, i64, i64, i32, vp, vp, vp, vp]
    L.vx_gemm.restype = i32
    L.vx_gemm_batched.argtypes = [i64, i64, i64, i64, i32, vp, i64, vp, i64, vp, i64, vp]
    L.vx_gemm_batched.restype = i32
    L.vx_gemm_batched_noalloc.argtypes = [i64, i64, i64, i64, i32, vp, i64, vp, i64, vp, i64, vp]
    L.vx_gemm_batched_noalloc.restype = i32
    L.vx_test_fail_workspace_alloc.argtypes = [i32]
    L.vx_test_fail_workspace_alloc.restype = i32
    L.vx_plan_query.argtypes = [i64, i64, i64, i64, i32, i64, i64, i64, ctypes.c_uint64, ctypes.POINTER(vx_plan)]
    L.vx_plan_query.restype = i32
    L.vx_plan_cost.argtypes = [i64, i64, i64, i64, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_double)]
    L.vx_plan_cost.restype = i32
    L.vx_cost_temporal.argtypes = [ctypes.c_double, i64, ctypes.c_double, ctypes.c_double]
    L.vx_cost_temporal.restype = ctypes.c_double
    L.vx_cost_parallel_factor.argtypes = [i64, i64]
    L.vx_cost_parallel_factor.restype = i64
    L.vx_get_hwinfo.argtypes = [ctypes.POINTER(vx_hwinfo)]
    L.vx_get_hwinfo.restype = i32
    L.vx_set_hwinfo_override.argtypes = [ctypes.POINTER(vx_hwinfo)]
    L.vx_set_hwinfo_override.restype = i32
    L.vx_registry_count.argtypes = []
    L.vx_registry_count.restype = i32
    L.vx_registry_get.argtypes = [i32, ctypes.POINTER(vx_kernel_info)]
    L.vx_registry_get.restype = i32
    L.vx_enable_hybrid_grid.argtypes = [i32]
    L.vx_enable_hybrid_grid.restype = i32
    L.vx_selector_exhaustive.argtypes = [i32]
    L.vx_selector_exhaustive.restype = i32
    L.vx_selector_last_evaluations.argtypes = []
    L.vx_selector_last_evaluations.restype = ctypes.c_int64
    L.vx_enable_k_rotation.argtypes = [i32]
    L.vx_enable_k_rotation.restype = i32
    L.vx_force_plan.argtypes = [i32, i32]
    L.vx_force_plan.restype = i32
    L.vx_fix_wavefront.argtypes = [i32, i32, i32]
    L.vx_fix_wavefront.restype = i32
    L.vx_restrict_backends.argtypes = [i32]
    L.vx_restrict_backends.restype = i32
    L.vx_conv2d.argtypes = [ctypes.POINTER(vx_conv2d_desc), vp, vp, vp, vp]
    L.vx_conv2d.restype = i32
    L.vx_conv2d_plan_query.argtypes = [ctypes.POINTER(vx_conv2d_desc), ctypes.POINTER(vx_plan)]
    L.vx_conv2d_plan_query.restype = i32
    L.vx_conv2d_output_dims.argtypes = [ctypes.POINTER(vx_conv2d_desc), ctypes.POINTER(i64), ctypes.POINTER(i64)]
    L.vx_conv2d_output_dims.restype = i32
    L.vx_set_workspace.argtypes = [vp, ctypes.c_size_t, vp]
    L.vx_set_workspace.restype = i32
    L.vx_calibration_load.argtypes = [ctypes.c_char_p, ctypes.POINTER(i32)]
    L.vx_calibration_load.restype = i32
    L.vx_calibration_enable.argtypes = [i32]
    L.vx_calibration_enable.restype = i32
    L.vx_calibration_active.argtypes = []
    L.vx_calibration_active.restype = i32
    L.vx_kernel_occupancy.argtypes = [i32, ctypes.POINTER(i32)]
    L.vx_kernel_occupancy.restype = i32
    L.vx_registry_hash.argtypes = []
    L.vx_registry_hash.restype = ctypes.c_char_p
    L.vx_status_string.argtypes = [i32]
    L.vx_status_string.restype = ctypes.c_char_p
    L.vx_version.argtypes = []
    L.vx_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _chk(st, what):
    if st != 0:
        raise VxError(st, what)


# ------------------------------------------------------------- raw ABI -----
def vx_gemm(M, N, K, dtype, A, B, C, stream=None):
    return lib().vx_gemm(M, N, K, dtype, A, B, C, stream)


def vx_gemm_batched(batch, M, N, K, dtype, A, sA, B, sB, C, sC, stream=None):
    return lib().vx_gemm_batched(batch, M, N, K, dtype, A, sA, B, sB, C, sC, stream)


def vx_gemm_batched_noalloc(batch, M, N, K, dtype, A, sA, B, sB, C, sC, stream=None):
    return lib().vx_gemm_batched_noalloc(batch, M, N, K, dtype, A, sA, B, sB, C, sC, stream)


def vx_test_fail_workspace_alloc(fail):
    return lib().vx_test_fail_workspace_alloc(1 if fail else 0)


def vx_plan_query(batch, M, N, K, dtype, sA=None, sB=None, sC=None, base_align=256):
    p = vx_plan()
    st = lib().vx_plan_query(batch, M, N, K, dtype, M * K if sA is None else sA, K * N if sB is None else sB,
                             M * N if sC is None else sC, base_align, ctypes.byref(p))
    _chk(st, "vx_plan_query")
    return p


def vx_plan_cost(batch, M, N, K, dtype, kernel_id, split_k, align=3):
    c = ctypes.c_double()
    st = lib().vx_plan_cost(batch, M, N, K, dtype, kernel_id, split_k, align, ctypes.byref(c))
    return st, c.value


def vx_cost_temporal(t_load, trips, cost_lower, t_store):
    return lib().vx_cost_temporal(t_load, trips, cost_lower, t_store)


def vx_cost_parallel_factor(parallel, units):
    return lib().vx_cost_parallel_factor(parallel, units)


def vx_get_hwinfo():
    h = vx_hwinfo()
    _chk(lib().vx_get_hwinfo(ctypes.byref(h)), "vx_get_hwinfo")
    return h


def vx_set_hwinfo_override(hw):
    return lib().vx_set_hwinfo_override(None if hw is None else ctypes.byref(hw))


def vx_registry_count():
    return lib().vx_registry_count()


def vx_registry_get(i):
    k = vx_kernel_info()
    _chk(lib().vx_registry_get(i, ctypes.byref(k)), "vx_registry_get")
    return k


def vx_force_plan(kernel_id, split_k=0):
    return lib().vx_force_plan(kernel_id, split_k)


def vx_fix_wavefront(wave_m=0, wave_n=0, mfma_m=0):
    return lib().vx_fix_wavefront(wave_m, wave_n, mfma_m)


def conv_desc(n, h, w, c_in, c_out, kh, kw, dtype, stride=(1, 1), pad=(0, 0), dil=(1, 1)):
    return vx_conv2d_desc(n, h, w, c_in, c_out, kh, kw, stride[0], stride[1], pad[0], pad[1], dil[0], dil[1],
                          dtype)


def vx_conv2d(desc, x, w, y, stream=None):
    return lib().vx_conv2d(ctypes.byref(desc), x, w, y, stream)


def vx_conv2d_plan_query(desc):
    p = vx_plan()
    _chk(lib().vx_conv2d_plan_query(ctypes.byref(desc), ctypes.byref(p)), "vx_conv2d_plan_query")
    return p


BACKEND_MFMA, BACKEND_VALU = 1, 2


def vx_restrict_backends(mask=0):
    return lib().vx_restrict_backends(mask)


def vx_enable_hybrid_grid(enable=1):
    return lib().vx_enable_hybrid_grid(enable)


def vx_selector_exhaustive(enable=1):
    return lib().vx_selector_exhaustive(enable)


def vx_selector_last_evaluations():
    return lib().vx_selector_last_evaluations()


def vx_enable_k_rotation(enable=1):
    return lib().vx_enable_k_rotation(enable)


def vx_set_workspace(ptr, nbytes, stream=None):
    return lib().vx_set_workspace(ptr, nbytes, stream)


def vx_calibration_load(path=None):
    n = ctypes.c_int(0)
    st = lib().vx_calibration_load(None if path is None else path.encode(), ctypes.byref(n))
    return st, n.value


def vx_calibration_enable(enable):
    return lib().vx_calibration_enable(1 if enable else 0)


def vx_calibration_active():
    return lib().vx_calibration_active()


def vx_kernel_occupancy(kernel_id):
    n = ctypes.c_int(0)
    _chk(lib().vx_kernel_occupancy(kernel_id, ctypes.byref(n)), "vx_kernel_occupancy")
    return n.value


def vx_registry_hash():
    return lib().vx_registry_hash().decode()


def vx_status_string(s):
    return lib().vx_status_string(s).decode()


def vx_version():
    return lib().vx_version().decode()


def mi355x_hwinfo():
    """The gfx950 description the library builds from the device, as a literal
    (for planning on a host without a GPU)."""
    h = vx_hwinfo()
    h.arch = b"gfx950"
    h.num_cu, h.num_xcd, h.simd_per_cu, h.wave_size = 256, 8, 4, 64
    h.max_threads_per_wg, h.lds_bytes_per_cu, h.vgprs_per_lane, h.max_waves_per_simd = 1024, 160 * 1024, 512, 8
    h.clock_ghz, h.hbm_gbps = 2.4, 8000.0
    h.l2_bytes_per_xcd, h.mall_bytes = 4.0 * 2 ** 20, 256.0 * 2 ** 20
    h.mfma_flop_clk_cu_f16, h.mfma_flop_clk_cu_f32 = 4096.0, 256.0
    h.l2_bytes_clk_cu, h.lds_bytes_clk_cu = 64.0, 128.0
    h.mem_latency_ns, h.atomic_latency_ns, h.launch_ns = 900.0, 1200.0, 2000.0
    return h


# ------------------------------------------------------ torch helpers -------
# The C ABI cannot see tensor extents, so the helpers below check everything
# the kernels will rely on before any library call: ranks, matching inner
# dimensions, one supported dtype, contiguity, the exact shape and dtype of a
# caller's `out`, and that every tensor lives on the current GPU (a host
# pointer or a short `out` handed to a kernel would be an out-of-bounds
# device access).  Violations raise ValueError.

def _torch_dtype_code(t):
    import torch
    codes = {torch.float32: VX_F32, torch.float16: VX_F16, torch.bfloat16: VX_BF16}
    if t.dtype not in codes:
        raise ValueError("unsupported dtype %s (float32, float16 or bfloat16)" % t.dtype)
    return codes[t.dtype]


def _stream_ptr(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check_operands(what, tensors, out, out_shape):
    """Validates operands (name -> tensor) and the optional `out` against the
    shape the call will write; returns the dtype code."""
    import torch
    first = next(iter(tensors.values()))
    code = _torch_dtype_code(first)
    for name, t in tensors.items():
        if t.dtype != first.dtype:
            raise ValueError("%s: %s has dtype %s, expected %s" % (what, name, t.dtype, first.dtype))
        if not t.is_contiguous():
            raise ValueError("%s: %s must be contiguous" % (what, name))
    if out is not None:
        if tuple(out.shape) != tuple(out_shape):
            raise ValueError("%s: out has shape %s, expected %s" % (what, tuple(out.shape), tuple(out_shape)))
        if out.dtype != first.dtype:
            raise ValueError("%s: out has dtype %s, expected %s" % (what, out.dtype, first.dtype))
        if not out.is_contiguous():
            raise ValueError("%s: out must be contiguous" % what)
    every = list(tensors.items()) + ([("out", out)] if out is not None else [])
    for name, t in every:
        if t.device.type != "cuda":
            raise ValueError("%s: %s is on %s; every tensor must be on the current GPU" % (what, name, t.device))
    dev = torch.cuda.current_device()
    for name, t in every:
        if t.device.index != dev:
            raise ValueError("%s: %s is on cuda:%s, the current device is cuda:%d" % (what, name, t.device.index, dev))
    return code


def gemm(A, B, out=None, stream=None):
    """C = A @ B for 2-D row-major tensors (contiguous, one dtype, current GPU)."""
    import torch
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError("gemm expects 2-D A (M x K) and B (K x N), got %d-D and %d-D" % (A.dim(), B.dim()))
    M, K = A.shape
    K2, N = B.shape
    if K2 != K:
        raise ValueError("gemm: inner dimensions differ (A is %d x %d, B is %d x %d)" % (M, K, K2, N))
    code = _check_operands("gemm", {"A": A, "B": B}, out, (M, N))
    C = torch.empty((M, N), dtype=A.dtype, device=A.device) if out is None else out
    _chk(vx_gemm(M, N, K, code, A.data_ptr(), B.data_ptr(), C.data_ptr(), _stream_ptr(stream)), "vx_gemm")
    return C


def bmm(A, B, out=None, stream=None):
    """C[b] = A[b] @ B[b] for a 3-D A (batch x M x K) and a 3-D B (batch x K x N),
    or a 2-D B (K x N) broadcast to every batch; contiguous, one dtype, current GPU."""
    import torch
    if A.dim() != 3 or B.dim() not in (2, 3):
        raise ValueError("bmm expects a 3-D A and a 2-D or 3-D B, got %d-D and %d-D" % (A.dim(), B.dim()))
    bt, M, K = A.shape
    if B.dim() == 2:
        K2, N = B.shape
        sB = 0
    else:
        bb, K2, N = B.shape
        if bb != bt:
            raise ValueError("bmm: batch sizes differ (%d and %d)" % (bt, bb))
        sB = K2 * N
    if K2 != K:
        raise ValueError("bmm: inner dimensions differ (A is .. x %d x %d, B is .. x %d x %d)" % (M, K, K2, N))
    code = _check_operands("bmm", {"A": A, "B": B}, out, (bt, M, N))
    C = torch.empty((bt, M, N), dtype=A.dtype, device=A.device) if out is None else out
    _chk(vx_gemm_batched(bt, M, N, K, code, A.data_ptr(), M * K, B.data_ptr(), sB,
                         C.data_ptr(), M * N, _stream_ptr(stream)), "vx_gemm_batched")
    return C


def conv2d_output_shape(x_shape, w_shape, stride=(1, 1), padding=(0, 0), dilation=(1, 1)):
    """(N, OH, OW, Cout) of conv2d(x, w) as the library computes it
    (vx_conv2d_output_dims)."""
    N, H, W, Cin = x_shape
    KH, KW, _, Cout = w_shape
    d = conv_desc(N, H, W, Cin, Cout, KH, KW, VX_F16, stride, padding, dilation)
    oh, ow = ctypes.c_int64(), ctypes.c_int64()
    _chk(lib().vx_conv2d_output_dims(ctypes.byref(d), ctypes.byref(oh), ctypes.byref(ow)), "vx_conv2d_output_dims")
    return (N, oh.value, ow.value, Cout)


def conv2d(x, w, stride=(1, 1), padding=(0, 0), dilation=(1, 1), out=None, stream=None):
    """y = conv2d(x, w) for torch tensors: x N x H x W x Cin, w KH x KW x Cin x Cout
    (both contiguous, same dtype, on the current GPU); returns y N x OH x OW x Cout."""
    import torch
    if x.dim() != 4 or w.dim() != 4:
        raise ValueError("conv2d: x must be N x H x W x Cin and w KH x KW x Cin x Cout")
    if x.shape[3] != w.shape[2]:
        raise ValueError("conv2d: x has %d channels, w expects %d" % (x.shape[3], w.shape[2]))
    _check_operands("conv2d", {"x": x, "w": w}, None, None)
    shape = conv2d_output_shape(tuple(x.shape), tuple(w.shape), stride, padding, dilation)
    code = _check_operands("conv2d", {"x": x, "w": w}, out, shape)
    if out is None:
        out = torch.empty(shape, dtype=x.dtype, device=x.device)
    d = conv_desc(*shape[:1], x.shape[1], x.shape[2], x.shape[3], shape[3], w.shape[0], w.shape[1], code,
                  stride, padding, dilation)
    _chk(vx_conv2d(d, x.data_ptr(), w.data_ptr(), out.data_ptr(), _stream_ptr(stream)), "vx_conv2d")
    return out
