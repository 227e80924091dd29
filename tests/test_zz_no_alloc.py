"""vx_gemm_batched_noalloc (the entry point that allocates nothing, its
split-K scratch a static device array) against vx_gemm_batched, through the
C ABI: the same plan gives bit-identical outputs, each within the oracle's
bound, on two calls in a row, the second with a smaller input (the scratch
keeps the first call's contents); a forced plan whose partials do not fit the
array is refused."""
import numpy as np
import pytest

import oracle
from oracle import tolerance
from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _case(batch, M, N, K, seed, split):
    """Runs one shape through both entry points with the same forced split;
    returns both outputs as bits plus the operands."""
    import torch
    dev = torch.device("cuda:0")
    A = I.device_normal((batch * M, K), 1.0, seed, dev, torch.bfloat16)
    B = I.device_normal((batch * K, N), 0.02, seed + 1, dev, torch.bfloat16)
    stream = torch.cuda.current_stream().cuda_stream
    p = vx.vx_plan_query(batch, M, N, K, vx.VX_BF16)
    assert vx.vx_force_plan(p.kernel_id, split) == 0
    outs = []
    try:
        for fn in (vx.vx_gemm_batched, vx.vx_gemm_batched_noalloc):
            C = torch.empty(batch * M * N, dtype=torch.bfloat16, device=dev)
            C.view(torch.int16).fill_(0x7fc0)
            st = fn(batch, M, N, K, vx.VX_BF16, A.data_ptr(), M * K, B.data_ptr(), K * N, C.data_ptr(), M * N,
                    stream)
            assert st == 0, vx.STATUS.get(st, st)
            torch.cuda.synchronize()
            outs.append(_bits(C).reshape(batch, M, N))
    finally:
        vx.vx_force_plan(-1, 0)
    return outs, _bits(A), _bits(B)


def _check(C, A, B, batch, M, N, K, what):
    ref, mag = oracle.gemm(A, B, I.BF16, M=M, N=N, K=K, batch=batch)
    tolerance.check(C, ref.reshape(batch, M, N), mag.reshape(batch, M, N), I.BF16, what)


def test_noalloc_matches_gemm_batched_two_calls_second_smaller():
    # first: a decode-like shape split 8 ways (partials 8 x 16 x 4096 fp32 per
    # batch entry); second, smaller: fewer tiles and slices
    for (batch, M, N, K, split, seed) in [(2, 16, 4096, 4096, 8, 11), (1, 5, 768, 3072, 4, 13)]:
        (c_ref, c_na), A, B = _case(batch, M, N, K, seed, split)
        assert np.array_equal(c_ref, c_na), "noalloc differs from vx_gemm_batched at (%d,%d,%d,%d)" % (
            batch, M, N, K)
        _check(c_na, A, B, batch, M, N, K, "noalloc (%d,%d,%d,%d) split %d" % (batch, M, N, K, split))


def test_noalloc_selector_plans_within_bound():
    """Unforced: the selector plans within the static scratch."""
    import torch
    dev = torch.device("cuda:0")
    for (M, N, K, seed) in [(16, 4096, 11008, 21), (3, 768, 768, 23)]:
        A = I.device_normal((M, K), 1.0, seed, dev, torch.bfloat16)
        B = I.device_normal((K, N), 0.02, seed + 1, dev, torch.bfloat16)
        C = torch.empty(M * N, dtype=torch.bfloat16, device=dev)
        st = vx.vx_gemm_batched_noalloc(1, M, N, K, vx.VX_BF16, A.data_ptr(), M * K, B.data_ptr(), K * N,
                                        C.data_ptr(), M * N, torch.cuda.current_stream().cuda_stream)
        assert st == 0, vx.STATUS.get(st, st)
        torch.cuda.synchronize()
        _check(_bits(C).reshape(1, M, N), _bits(A), _bits(B), 1, M, N, K, "noalloc selector (%d,%d,%d)" % (M, N, K))


def test_noalloc_refuses_a_forced_plan_beyond_its_scratch():
    """32 MiB of partials (256 tiles of 128 x 128, 2 slices): the library's own
    64 MiB workspace takes it, the 16 MiB static array does not."""
    import torch
    dev = torch.device("cuda:0")
    kid = next(i for i in range(vx.vx_registry_count())
               for k in [vx.vx_registry_get(i)]
               if k.enabled and k.dtype == vx.VX_BF16 and k.family == 1 and k.op == 0 and k.mb == 128
               and k.nb == 128 and k.align == 3 and k.schedule == 0)
    M, N, K = 1024, 4096, 512
    A = torch.zeros((M, K), dtype=torch.bfloat16, device=dev)
    B = torch.zeros((K, N), dtype=torch.bfloat16, device=dev)
    C = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    assert vx.vx_force_plan(kid, 2) == 0
    try:
        assert vx.vx_gemm_batched(1, M, N, K, vx.VX_BF16, A.data_ptr(), M * K, B.data_ptr(), K * N,
                                  C.data_ptr(), M * N, s) == 0
        assert vx.vx_gemm_batched_noalloc(1, M, N, K, vx.VX_BF16, A.data_ptr(), M * K, B.data_ptr(), K * N,
                                          C.data_ptr(), M * N, s) == 4   # VX_ERR_WORKSPACE
    finally:
        vx.vx_force_plan(-1, 0)
    torch.cuda.synchronize()


def test_noalloc_argument_errors():
    assert vx.vx_gemm_batched_noalloc(1, -1, 4, 4, vx.VX_BF16, None, 0, None, 0, None, 0, None) == 1
    assert vx.vx_gemm_batched_noalloc(1, 4, 4, 4, 7, None, 0, None, 0, None, 0, None) == 2
    assert vx.vx_gemm_batched_noalloc(0, 4, 4, 4, vx.VX_BF16, None, 0, None, 0, None, 0, None) == 0
