"""Parity at the full workload sizes, in the launch configuration the
benchmark uses (the selector's own plans), on sampled outputs.

Sampled outputs: every element of the last row and last column (the ragged
edge tiles) plus random positions, each a full-K binary64 dot product from
the oracle.  Bounds as in the element-wise parity tests.
"""
import numpy as np
import pytest

import oracle
from oracle import tolerance
from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

from .gpu_util import run_gemm, run_batched

pytestmark = pytest.mark.gpu


def _sample(g, M, N, n_rand):
    rows = np.concatenate([np.full(N, M - 1), np.arange(M), g.integers(0, M, n_rand)])
    cols = np.concatenate([np.arange(N), np.full(M, N - 1), g.integers(0, N, n_rand)])
    return rows.astype(np.int64), cols.astype(np.int64)


def _check_sampled(C, A, B, code, M, N, K, g, n_rand, what, batch=1, sA=None, sB=None):
    rows, cols = _sample(g, M, N, n_rand)
    bats = g.integers(0, batch, rows.size) if batch > 1 else np.zeros(rows.size, np.int64)
    ref, mag = oracle.gemm_sampled(A, B, code, M, N, K, rows, cols, bats, sA=sA, sB=sB)
    C = C.reshape(batch, M, N)
    return tolerance.check(C[bats, rows, cols], ref, mag, code, what)


def test_sweep_f16_every_M():
    g = I.rng(1000)
    worst = 0.0
    for M in range(1, 513):
        A, B = I.sweep_f16(M)
        C = run_gemm(A, B, I.F16)
        worst = max(worst, _check_sampled(C, A, B, I.F16, M, 768, 768, g, 256, "sweep M=%d" % M))
    assert worst <= 1.0


@pytest.mark.parametrize("trial", [0, 1, 2, 3])
def test_encoder_trial(trial):
    g = I.rng(2000 + trial)
    M, gemms = I.encoder_trial(trial)
    for (A, B) in gemms:
        K, N = B.shape
        C = run_gemm(A, B, I.BF16)
        _check_sampled(C, A, B, I.BF16, M, N, K, g, 4096, "encoder t=%d M=%d %dx%d" % (trial, M, K, N))


@pytest.mark.parametrize("trial", [0, 1])
def test_attention_trial(trial):
    g = I.rng(3000 + trial)
    L, Q, Kt, P, V = I.attention_trial(trial)
    b, d = Q.shape[0], Q.shape[2]
    S = run_batched(Q, L * d, Kt, d * L, I.BF16, b, L, L, d)
    _check_sampled(S, Q, Kt, I.BF16, L, L, d, g, 4096, "S L=%d" % L, batch=b, sA=L * d, sB=d * L)
    O = run_batched(P, L * L, V, L * d, I.BF16, b, L, d, L)
    _check_sampled(O, P, V, I.BF16, L, d, L, g, 4096, "O L=%d" % L, batch=b, sA=L * L, sB=L * d)


@pytest.mark.parametrize("trial", [0, 1, 2, 3, 4, 5])
def test_llm_trial(trial):
    g = I.rng(4000 + trial)
    M, gemms = I.llm_trial(trial)
    for (A, B) in gemms:
        K, N = B.shape
        C = run_gemm(A, B, I.BF16)
        _check_sampled(C, A, B, I.BF16, M, N, K, g, 2048, "llm t=%d M=%d %dx%d" % (trial, M, K, N))


def test_attention_unaligned_lengths():
    """L values that break every vector alignment (odd, prime) use the
    element-aligned register-staged kernels; checked in full at a reduced batch."""
    g = I.rng(3100)
    for L in (1, 7, 37, 129, 255):
        b, d = 6, 64
        Q = I.normal(g, (b, L, d), I.BF16)
        Kt = I.normal(g, (b, d, L), I.BF16)
        S = run_batched(Q, L * d, Kt, d * L, I.BF16, b, L, L, d).reshape(b, L, L)
        ref, mag = oracle.gemm(Q, Kt, I.BF16, M=L, N=L, K=d, batch=b)
        tolerance.check(S, ref, mag, I.BF16, "S L=%d" % L)
        P = I.uniform(g, (b, L, L), I.BF16, 0.0, 2.0 / L)
        V = I.normal(g, (b, L, d), I.BF16)
        O = run_batched(P, L * L, V, L * d, I.BF16, b, L, d, L).reshape(b, L, d)
        ref, mag = oracle.gemm(P, V, I.BF16, M=L, N=d, K=L, batch=b)
        tolerance.check(O, ref, mag, I.BF16, "O L=%d" % L)
