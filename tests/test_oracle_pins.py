"""Pins for the CPU oracle: facts from outside the oracle that it must reproduce.

Each pin is chosen so that a plausible slip in the oracle (a dropped k term, a
wrong sign, a transposed operand, a wrong index or stride, a codec error)
fails at least one of them.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import F32, F16, BF16
from paper_2409_01075_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- codecs ----

def test_f16_decode_exhaustive_vs_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(bits, F16)
    want = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


def test_bf16_decode_exhaustive_vs_torch():
    torch = pytest.importorskip("torch")
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(bits, BF16)
    want = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def _probe_values(g, n):
    """Doubles spread over the fp16/bf16 ranges, plus exact midpoints (ties)."""
    e = g.integers(-30, 18, size=n)
    m = g.uniform(1.0, 2.0, size=n)
    s = np.where(g.integers(0, 2, size=n) == 0, 1.0, -1.0)
    return s * np.ldexp(m, e)


def test_f16_encode_vs_numpy():
    g = I.rng(1)
    x = _probe_values(g, 1_000_000)
    # exact midpoints between adjacent fp16 values, incl. subnormals
    b = g.integers(0, 0x7bff, size=200_000).astype(np.uint16)
    lo = b.view(np.float16).astype(np.float64)
    hi = (b + 1).astype(np.uint16).view(np.float16).astype(np.float64)
    x = np.concatenate([x, (lo + hi) / 2, -(lo + hi) / 2, [0.0, -0.0, 65519.0, 65520.0, 1e6]])
    got = oracle.encode(x, F16)
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want)


def _nearest_even_bruteforce(x, table_vals, table_bits):
    """Round by search in the sorted table of finite values; ties to even bits."""
    idx = np.searchsorted(table_vals, x)
    idx = np.clip(idx, 1, len(table_vals) - 1)
    lo, hi = table_vals[idx - 1], table_vals[idx]
    blo, bhi = table_bits[idx - 1], table_bits[idx]
    dlo, dhi = x - lo, hi - x
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (bhi % 2 == 0))
    return np.where(pick_hi, bhi, blo)


def test_bf16_encode_vs_bruteforce_nearest_even():
    bits = np.arange(0, 0x7f80, dtype=np.uint32).astype(np.uint16)   # +0 .. max finite
    vals = oracle.decode(bits, BF16)        # decode is pinned exhaustively above
    g = I.rng(2)
    e = g.integers(-130, 127, size=300_000)
    m = g.uniform(1.0, 2.0, size=300_000)
    x = np.ldexp(m, e)
    mid_b = g.integers(0, 0x7f7f, size=100_000).astype(np.uint16)
    mid = (oracle.decode(mid_b, BF16) + oracle.decode((mid_b + 1).astype(np.uint16), BF16)) / 2
    x = np.concatenate([x, mid])
    x = x[x <= vals[-1]]
    want = _nearest_even_bruteforce(x, vals, bits)
    got = oracle.encode(x, BF16)
    assert np.array_equal(got, want.astype(np.uint16))
    assert np.array_equal(oracle.encode(-x, BF16), (want | 0x8000).astype(np.uint16))


def test_bf16_encode_vs_torch_on_fp32_values():
    torch = pytest.importorskip("torch")
    g = I.rng(3)
    x = _probe_values(g, 500_000).astype(np.float32).astype(np.float64)  # exact in fp32
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.encode(x, BF16), want)


def test_rne_tie_table():
    with open(os.path.join(GOLDEN, "rne_ties.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    for dt, val, hexbits, expect in rows:
        code = {"f16": F16, "bf16": BF16}[dt]
        got = int(oracle.encode([float(val)], code)[0])
        assert got == int(hexbits, 16), (dt, val, hex(got))
        assert oracle.decode(np.array([got], dtype=np.uint16), code)[0] == float(expect)


# ------------------------------------------------------------ the GEMM ------

def test_textbook_worked_example():
    with open(os.path.join(GOLDEN, "gemm_textbook_2x3x4.txt")) as f:
        kv = {}
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                k, *v = ln.split()
                kv[k] = [float(t) for t in v]
    M, K, N = int(kv["M"][0]), int(kv["K"][0]), int(kv["N"][0])
    for code in (F32, F16, BF16):
        A = I.to_storage(np.array(kv["A"]).reshape(M, K), code)
        B = I.to_storage(np.array(kv["B"]).reshape(K, N), code)
        C, Mag = oracle.gemm(A, B, code)
        assert np.array_equal(C, np.array(kv["C"]).reshape(M, N))
        assert np.array_equal(Mag, C)       # all entries positive


def _exact(Av, Bv):
    M, K = Av.shape
    N = Bv.shape[1]
    Af = [[Fraction(float(v)) for v in r] for r in Av]
    Bf = [[Fraction(float(v)) for v in r] for r in Bv]
    return [[sum((Af[i][k] * Bf[k][j] for k in range(K)), Fraction(0)) for j in range(N)]
            for i in range(M)]


@pytest.mark.parametrize("code", [F32, F16, BF16])
def test_exact_rational_bruteforce_tiny(code):
    g = I.rng(10 + code)
    u = 2.0 ** -53
    for M in range(1, 7):
        for N in range(1, 7):
            for K in (1, 2, 3, 5, 6):
                A = I.uniform(g, (M, K), code)
                B = I.uniform(g, (K, N), code)
                C, Mag = oracle.gemm(A, B, code)
                ex = _exact(oracle.decode(A, code), oracle.decode(B, code))
                for i in range(M):
                    for j in range(N):
                        err = abs(Fraction(C[i, j]) - ex[i][j])
                        assert err <= Fraction(K * u * 1.0001) * Fraction(Mag[i, j]), (M, N, K, i, j)


@pytest.mark.parametrize("code", [F32, F16, BF16])
def test_vs_numpy_float64_matmul(code):
    g = I.rng(20 + code)
    M, K, N = 70, 131, 90
    A = I.uniform(g, (M, K), code)
    B = I.uniform(g, (K, N), code)
    C, Mag = oracle.gemm(A, B, code)
    Ad, Bd = oracle.decode(A, code), oracle.decode(B, code)
    assert np.all(np.abs(C - Ad @ Bd) <= 1e-12 * Mag)
    assert np.allclose(Mag, np.abs(Ad) @ np.abs(Bd), rtol=1e-13, atol=0)


@pytest.mark.parametrize("code", [F32, F16, BF16])
def test_identity_and_permutation(code):
    g = I.rng(30 + code)
    for M, K, N in [(77, 77, 96), (17, 17, 5), (1, 1, 9), (33, 33, 40)]:
        B = I.uniform(g, (K, N), code)
        Bd = oracle.decode(B, code)
        eye = I.to_storage(np.eye(M, K), code)
        C, _ = oracle.gemm(eye, B, code)
        assert np.array_equal(C, Bd)
        perm = g.permutation(M)
        P = I.to_storage(np.eye(M, K)[perm], code)
        C, _ = oracle.gemm(P, B, code)
        assert np.array_equal(C, Bd[perm])
        A = I.uniform(g, (M, K), code)
        C, _ = oracle.gemm(A, I.to_storage(np.eye(K, K), code), code)
        assert np.array_equal(C, oracle.decode(A, code))
        # rectangular [I; 0] picks the first K rows of B
        R = I.to_storage(np.vstack([np.eye(K), np.zeros((3, K))]), code)
        C, _ = oracle.gemm(R, B, code)
        assert np.array_equal(C[:K], Bd) and not C[K:].any()


@pytest.mark.parametrize("K", [1, 2, 5, 7, 64, 77, 768])
def test_rank1_closed_forms(K):
    M, N = 9, 11
    ones_a = I.to_storage(np.ones((M, K)), F32)
    ones_b = I.to_storage(np.ones((K, N)), F32)
    C, _ = oracle.gemm(ones_a, ones_b, F32)
    assert np.all(C == K)
    # B[k][j] = (k mod 5) - 2: the row sum has the closed form q*0 + r(r-1)/2 - 2r
    Bk = np.tile(((np.arange(K) % 5) - 2.0)[:, None], (1, N))
    C, Mag = oracle.gemm(ones_a, I.to_storage(Bk, F32), F32)
    q, r = divmod(K, 5)
    assert np.all(C == r * (r - 1) / 2 - 2 * r)
    assert np.all(Mag == q * 6 + sum(abs((k % 5) - 2) for k in range(r)))
    # A = u 1^T, B = 1 v^T  =>  C = K u v^T
    u = np.arange(1, M + 1, dtype=np.float64) - 4
    v = np.arange(1, N + 1, dtype=np.float64) - 6
    C, _ = oracle.gemm(I.to_storage(np.tile(u[:, None], (1, K)), F16),
                       I.to_storage(np.tile(v[None, :], (K, 1)), F16), F16)
    assert np.array_equal(C, K * np.outer(u, v))


def test_k_zero_and_empty():
    A = np.zeros((4, 0), dtype=np.float32)
    B = np.zeros((0, 3), dtype=np.float32)
    C, Mag = oracle.gemm(A, B, F32, M=4, N=3, K=0)
    assert C.shape == (4, 3) and not C.any() and not Mag.any()
    C, Mag = oracle.gemm(np.zeros((0, 5), np.float32), np.zeros((5, 3), np.float32), F32,
                         M=0, N=3, K=5)
    assert C.shape == (0, 3)


def test_batched_strides_and_broadcast():
    g = I.rng(40)
    bt, M, K, N = 3, 5, 7, 6
    A = I.uniform(g, (bt, M, K), BF16)
    B = I.uniform(g, (bt, K, N), BF16)
    C, Mag = oracle.gemm(A, B, BF16, M=M, N=N, K=K, batch=bt)
    for b in range(bt):
        Cb, Mb = oracle.gemm(A[b], B[b], BF16)
        assert np.array_equal(C[b], Cb) and np.array_equal(Mag[b], Mb)
    Cbc, _ = oracle.gemm(A, B[0], BF16, M=M, N=N, K=K, batch=bt, sB=0)
    for b in range(bt):
        assert np.array_equal(Cbc[b], oracle.gemm(A[b], B[0], BF16)[0])


def test_sampled_matches_full():
    g = I.rng(50)
    bt, M, K, N = 2, 33, 40, 29
    A = I.uniform(g, (bt, M, K), F16)
    B = I.uniform(g, (bt, K, N), F16)
    C, Mag = oracle.gemm(A, B, F16, M=M, N=N, K=K, batch=bt)
    rows = g.integers(0, M, 200)
    cols = g.integers(0, N, 200)
    bats = g.integers(0, bt, 200)
    ref, mag = oracle.gemm_sampled(A, B, F16, M, N, K, rows, cols, bats)
    assert np.array_equal(ref, C[bats, rows, cols])
    assert np.array_equal(mag, Mag[bats, rows, cols])
    # the threaded form (samples grouped by column, columns decoded once per
    # group) gives the same binary64 values, for any thread count
    for threads in (2, 3, 8, 500):
        ref_t, mag_t = oracle.gemm_sampled(A, B, F16, M, N, K, rows, cols, bats, threads=threads)
        assert np.array_equal(ref_t, ref) and np.array_equal(mag_t, mag)


@pytest.mark.parametrize("code", [F32, F16, BF16])
def test_sampled_threaded_matches_full_bf16_f32_broadcast(code):
    """Threaded sampling with a broadcast B (sB = 0) and repeated columns."""
    g = I.rng(51 + code)
    bt, M, K, N = 3, 17, 65, 23
    A = I.normal(g, (bt, M, K), code)
    B = I.normal(g, (K, N), code)
    C, Mag = oracle.gemm(A, B, code, M=M, N=N, K=K, batch=bt, sB=0)
    rows = np.concatenate([np.full(N, M - 1), np.arange(M), g.integers(0, M, 300)])
    cols = np.concatenate([np.arange(N), np.full(M, N - 1), g.integers(0, N, 300)])
    bats = g.integers(0, bt, rows.size)
    ref, mag = oracle.gemm_sampled(A, B, code, M, N, K, rows, cols, bats, sB=0, threads=4)
    assert np.array_equal(ref, C[bats, rows, cols])
    assert np.array_equal(mag, Mag[bats, rows, cols])


def test_threads_do_not_change_results():
    g = I.rng(60)
    A = I.uniform(g, (37, 300), F32)
    B = I.uniform(g, (300, 41), F32)
    C1, _ = oracle.gemm(A, B, F32, threads=1)
    C8, _ = oracle.gemm(A, B, F32, threads=8)
    assert np.array_equal(C1, C8)


def test_exact_range_helper():
    # K * r^2 <= 2^p keeps every partial sum exact in the output type
    for code, p in ((F16, 11), (BF16, 8), (F32, 24)):
        for K in (1, 5, 80, 768, 4096):
            r = I.exact_range(K, code)
            assert K * r * r <= 2 ** p
            assert K * (r + 1) * (r + 1) > 2 ** p


# ------------------------------------------------------------ convolution ----
# The direct convolution (N x H x W x Cin input, KH x KW x Cin x Cout filter,
# zero padding, stride, dilation) pinned to outside facts.

def _conv_cases(g, n):
    for _ in range(n):
        N, H, W = int(g.integers(1, 3)), int(g.integers(1, 6)), int(g.integers(1, 6))
        Cin, Cout, KH, KW = int(g.integers(1, 4)), int(g.integers(1, 4)), int(g.integers(1, 4)), int(g.integers(1, 4))
        st = (int(g.integers(1, 3)), int(g.integers(1, 3)))
        pd = (int(g.integers(0, 3)), int(g.integers(0, 3)))
        dl = (int(g.integers(1, 3)), int(g.integers(1, 3)))
        yield N, H, W, Cin, Cout, KH, KW, st, pd, dl


@pytest.mark.parametrize("code", [F32, F16, BF16])
def test_conv_bruteforce_exact_rational(code):
    """Every tap enumerated in exact rational arithmetic from the layer's
    definition; the oracle is within its own binary64 rounding of it."""
    g = I.rng(900 + code)
    for (N, H, W, Cin, Cout, KH, KW, st, pd, dl) in _conv_cases(g, 40):
        x = I.uniform(g, (N, H, W, Cin), code)
        w = I.uniform(g, (KH, KW, Cin, Cout), code)
        xd, wd = oracle.decode(x, code), oracle.decode(w, code)
        ref, mag = oracle.conv2d(x, w, code, st, pd, dl)
        OH, OW = ref.shape[1], ref.shape[2]
        assert OH == max(0, (H + 2 * pd[0] - dl[0] * (KH - 1) - 1) // st[0] + 1)
        assert OW == max(0, (W + 2 * pd[1] - dl[1] * (KW - 1) - 1) // st[1] + 1)
        K = KH * KW * Cin
        for n in range(N):
            for oh in range(OH):
                for ow in range(OW):
                    for co in range(Cout):
                        exact = Fraction(0)
                        for kh in range(KH):
                            for kw in range(KW):
                                ih = oh * st[0] - pd[0] + kh * dl[0]
                                iw = ow * st[1] - pd[1] + kw * dl[1]
                                if 0 <= ih < H and 0 <= iw < W:
                                    for ci in range(Cin):
                                        exact += Fraction(xd[n, ih, iw, ci]) * Fraction(wd[kh, kw, ci, co])
                        err = abs(Fraction(ref[n, oh, ow, co]) - exact)
                        assert err <= Fraction(K) * Fraction(2) ** -53 * Fraction(mag[n, oh, ow, co])


def test_conv_matches_torch_float64():
    """PyTorch's CPU convolution in binary64 (NCHW, so the test permutes)."""
    torch = pytest.importorskip("torch")
    g = I.rng(910)
    for (N, H, W, Cin, Cout, KH, KW, st, pd, dl) in list(_conv_cases(g, 25)) + [(2, 17, 13, 5, 7, 3, 3, (2, 1), (1, 2), (1, 1))]:
        x = I.uniform(g, (N, H, W, Cin), F32)
        w = I.uniform(g, (KH, KW, Cin, Cout), F32)
        ref, mag = oracle.conv2d(x, w, F32, st, pd, dl)
        if ref.size == 0:
            continue
        xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
        wt = torch.from_numpy(w.astype(np.float64)).permute(3, 2, 0, 1)
        want = torch.nn.functional.conv2d(xt, wt, stride=st, padding=pd, dilation=dl).permute(0, 2, 3, 1).numpy()
        assert want.shape == ref.shape
        assert np.all(np.abs(ref - want) <= 1e-12 * mag + 1e-300)


def test_conv_1x1_is_matmul():
    """A 1 x 1, stride-1, unpadded convolution is the GEMM of the pixels by the filter."""
    g = I.rng(920)
    x = I.uniform(g, (3, 7, 5, 11), F32)
    w = I.uniform(g, (1, 1, 11, 6), F32)
    ref, mag = oracle.conv2d(x, w, F32)
    want = x.astype(np.float64).reshape(-1, 11) @ w.astype(np.float64).reshape(11, 6)
    assert np.all(np.abs(ref.reshape(-1, 6) - want) <= 1e-12 * mag.reshape(-1, 6))


def test_conv_matches_scipy_correlate2d():
    """Single channel, stride 1: scipy's 2-D cross-correlation (zero-padded input)."""
    signal = pytest.importorskip("scipy.signal")
    g = I.rng(930)
    for (H, W, KH, KW, ph, pw) in ((6, 5, 3, 2, 0, 0), (4, 7, 2, 3, 1, 2), (5, 5, 5, 5, 2, 2), (3, 8, 1, 4, 0, 3)):
        x = I.uniform(g, (1, H, W, 1), F32)
        w = I.uniform(g, (KH, KW, 1, 1), F32)
        ref = oracle.conv2d(x, w, F32, (1, 1), (ph, pw), (1, 1), with_mag=False)
        xp = np.pad(x[0, :, :, 0].astype(np.float64), ((ph, ph), (pw, pw)))
        want = signal.correlate2d(xp, w[:, :, 0, 0].astype(np.float64), mode="valid")
        assert np.allclose(ref[0, :, :, 0], want, rtol=0, atol=1e-12)


def test_conv_delta_filter_moves_the_input():
    """A filter that is the identity channel map at one tap (kh0, kw0) copies
    the input pixel that tap reads: exact, zeros where it falls in the padding."""
    g = I.rng(940)
    for code in (F32, F16, BF16):
        N, H, W, C, KH, KW = 2, 7, 6, 3, 3, 2
        st, pd, dl = (2, 1), (2, 1), (1, 2)
        x = I.uniform(g, (N, H, W, C), code)
        for kh0 in range(KH):
            for kw0 in range(KW):
                wd = np.zeros((KH, KW, C, C))
                wd[kh0, kw0] = np.eye(C)
                ref = oracle.conv2d(x, oracle.encode(wd, code), code, st, pd, dl, with_mag=False)
                xd = oracle.decode(x, code)
                for oh in range(ref.shape[1]):
                    for ow in range(ref.shape[2]):
                        ih, iw = oh * st[0] - pd[0] + kh0 * dl[0], ow * st[1] - pd[1] + kw0 * dl[1]
                        want = xd[:, ih, iw, :] if (0 <= ih < H and 0 <= iw < W) else 0.0
                        assert np.array_equal(ref[:, oh, ow, :], np.broadcast_to(want, ref[:, oh, ow, :].shape))


def test_conv_ones_count_the_taps_inside_the_image():
    """All-ones input and filter: every output is Cin times the number of taps
    whose (ih, iw) falls inside the image -- counted here independently."""
    for (H, W, KH, KW, st, pd, dl) in ((5, 4, 3, 3, (1, 1), (1, 1), (1, 1)), (9, 7, 3, 2, (2, 3), (2, 1), (2, 1)),
                                       (4, 4, 5, 5, (1, 1), (2, 2), (1, 1))):
        C = 3
        x = np.ones((1, H, W, C), dtype=np.float32)
        w = np.ones((KH, KW, C, 2), dtype=np.float32)
        ref = oracle.conv2d(x, w, F32, st, pd, dl, with_mag=False)
        for oh in range(ref.shape[1]):
            rows = sum(1 for kh in range(KH) if 0 <= oh * st[0] - pd[0] + kh * dl[0] < H)
            for ow in range(ref.shape[2]):
                cols = sum(1 for kw in range(KW) if 0 <= ow * st[1] - pd[1] + kw * dl[1] < W)
                assert np.all(ref[0, oh, ow] == C * rows * cols)


def test_conv_stride_subsamples_and_dilation_spreads_the_filter():
    g = I.rng(950)
    x = I.uniform(g, (2, 11, 10, 3), F32)
    w = I.uniform(g, (3, 3, 3, 4), F32)
    full = oracle.conv2d(x, w, F32, (1, 1), (1, 1), (1, 1), with_mag=False)
    strided = oracle.conv2d(x, w, F32, (2, 3), (1, 1), (1, 1), with_mag=False)
    assert np.array_equal(strided, full[:, ::2, ::3, :])
    # dilation 2 == the filter with a zero between taps, undilated
    wd = np.zeros((5, 5, 3, 4), dtype=np.float32)
    wd[::2, ::2] = w
    assert np.array_equal(oracle.conv2d(x, w, F32, (1, 1), (2, 2), (2, 2), with_mag=False),
                          oracle.conv2d(x, wd, F32, (1, 1), (2, 2), (1, 1), with_mag=False))
