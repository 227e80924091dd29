"""The split-K workspace fallback on the device: when the library cannot get
a workspace for a stream, a call whose plan would split K runs without
split-K instead, with correct results (test hook vx_test_fail_workspace_alloc)."""
import numpy as np
import pytest

import oracle
from oracle import tolerance
from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

pytestmark = pytest.mark.gpu


def test_workspace_allocation_failure_falls_back_to_unsplit_plans():
    import torch
    dev = torch.device("cuda:0")
    # a long K over few output tiles: split-K under the calibrated and the analytical model alike
    M, N, K = 16, 256, 32768
    assert vx.vx_plan_query(1, M, N, K, vx.VX_BF16).split_k > 1
    A = I.device_normal((M, K), 1.0, 31, dev, torch.bfloat16)
    B = I.device_normal((K, N), 0.02, 32, dev, torch.bfloat16)
    C = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    C.view(torch.int16).fill_(0x7fc0)
    s = torch.cuda.Stream()          # a stream with no workspace yet
    assert vx.vx_test_fail_workspace_alloc(1) == 0
    try:
        assert vx.vx_plan_query(1, M, N, K, vx.VX_BF16).split_k == 1
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            st = vx.vx_gemm(M, N, K, vx.VX_BF16, A.data_ptr(), B.data_ptr(), C.data_ptr(), s.cuda_stream)
        assert st == 0, vx.STATUS.get(st, st)
        s.synchronize()
    finally:
        vx.vx_test_fail_workspace_alloc(0)
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    ref, mag = oracle.gemm(bits(A), bits(B), I.BF16)
    tolerance.check(bits(C), ref, mag, I.BF16, "fallback (16,256,32768)")
