"""The bench's untimed check of the sweep outputs (CPU): it accepts C equal to
the oracle's rounded result and reports a single element moved just beyond
the fp16 bound, with the whole last row, the last column and random entries
sampled."""
import numpy as np

import oracle
from paper_2409_01075_amd import inputs as I

import bench


def _rounded(ms):
    out = {}
    for M in ms:
        A, B = I.sweep_f16(M, bench.K_SWEEP, bench.N_SWEEP)
        ref, _ = oracle.gemm(A, B, I.F16, threads=4)
        out[M] = oracle.encode(ref, I.F16)
    return out


def test_check_accepts_the_rounded_oracle_result():
    ms = [1, 7, 33]
    res = bench._check_outputs(ms, _rounded(ms), threads=4)
    assert res["within_bound"] and res["shapes"] == 3
    assert res["max_err_over_bound"] <= 1.0
    assert res["entries"] == sum(bench.N_SWEEP + M + 512 for M in ms)


def test_check_reports_one_element_beyond_the_bound():
    ms = [5, 9]
    outs = _rounded(ms)
    M = 9
    A, B = I.sweep_f16(M, bench.K_SWEEP, bench.N_SWEEP)
    ref, mag = oracle.gemm(A, B, I.F16, threads=4)
    # the last row is always sampled: move one of its elements to 1.5x the bound
    j = 100
    bound = 4e-3 * mag[M - 1, j] + 1e-6
    outs[M] = outs[M].copy()
    outs[M][M - 1, j] = oracle.encode(np.array([ref[M - 1, j] + 1.5 * bound]), I.F16)[0]
    res = bench._check_outputs(ms, outs, threads=4)
    assert not res["within_bound"]
    assert "M=9" in res["first_failure"]
