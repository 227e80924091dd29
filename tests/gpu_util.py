"""Helpers for the GPU tests: move stored operands to the device and back,
and call the library through its C ABI."""
import numpy as np

from paper_2409_01075_amd import vx


def torch_dtype(code):
    import torch
    return {0: torch.float32, 1: torch.float16, 2: torch.bfloat16}[code]


def to_dev(x, code, device="cuda"):
    import torch
    x = np.ascontiguousarray(x)
    raw = x.view(np.float32) if code == 0 else x.view(np.int16)
    return torch.from_numpy(raw).to(device).view(torch_dtype(code))


def from_dev(t, code):
    import torch
    t = t.detach()
    if code == 0:
        return t.view(torch.int32).cpu().numpy().view(np.float32)
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def empty_out(shape, code, fill_bits=None, device="cuda"):
    import torch
    t = torch.empty(shape, dtype=torch_dtype(code), device=device)
    if fill_bits is not None:
        t.view(torch.int32 if code == 0 else torch.int16).fill_(fill_bits)
    return t


def run_gemm(A, B, code, C=None):
    """C = A x B through vx_gemm; returns C's stored bits (numpy)."""
    import torch
    M, K = A.shape
    N = B.shape[1]
    At, Bt = to_dev(A, code), to_dev(B, code)
    Ct = empty_out((M, N), code, fill_bits=0x7fc0 if code else 0x7fc00000) if C is None else C
    st = vx.vx_gemm(M, N, K, code, At.data_ptr(), Bt.data_ptr(), Ct.data_ptr(),
                    torch.cuda.current_stream().cuda_stream)
    assert st == 0, vx.STATUS.get(st, st)
    torch.cuda.synchronize()
    return from_dev(Ct, code)


def run_batched(A, sA, B, sB, code, batch, M, N, K, sC=None):
    import torch
    sC = M * N if sC is None else sC
    At, Bt = to_dev(A, code), to_dev(B, code)
    Ct = empty_out(((batch - 1) * sC + M * N,), code, fill_bits=0x7fc0 if code else 0x7fc00000)
    st = vx.vx_gemm_batched(batch, M, N, K, code, At.data_ptr(), sA, Bt.data_ptr(), sB, Ct.data_ptr(), sC,
                            torch.cuda.current_stream().cuda_stream)
    assert st == 0, vx.STATUS.get(st, st)
    torch.cuda.synchronize()
    return from_dev(Ct, code)
