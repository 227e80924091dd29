"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bounds (see oracle/tolerance.py): fp16/bf16 |C-Cref| <= 4e-3*Mag + 1e-6,
fp32 1e-5*Mag elementwise and normwise; integer-valued inputs bit-exact.
"""
import numpy as np
import pytest

import oracle
from oracle import tolerance
from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

from .gpu_util import from_dev, run_gemm, run_batched

pytestmark = pytest.mark.gpu

DTS = [I.F32, I.F16, I.BF16]


@pytest.fixture(autouse=True)
def _unforce():
    vx.vx_force_plan(-1, 0)
    yield
    vx.vx_force_plan(-1, 0)


def test_single_f32_77x96x80():
    A, B = I.single_f32(0)
    C = run_gemm(A, B, I.F32)
    ref, mag = oracle.gemm(A, B, I.F32)
    tolerance.check(C, ref, mag, I.F32, "fp32 77x96x80")


@pytest.mark.parametrize("M", [1, 2, 3, 7, 8, 15, 16, 17, 31, 33, 63, 64, 65, 100, 127, 129, 200, 255,
                               256, 257, 300, 383, 384, 385, 448, 511, 512])
def test_sweep_f16(M):
    A, B = I.sweep_f16(M)
    C = run_gemm(A, B, I.F16)
    ref, mag = oracle.gemm(A, B, I.F16)
    tolerance.check(C, ref, mag, I.F16, "fp16 M=%d" % M)


@pytest.mark.parametrize("code", DTS)
def test_identity_permutation_exact(code):
    g = I.rng(100 + code)
    for M, N in [(77, 96), (17, 40), (1, 9), (130, 264)]:
        K = M
        B = I.small_int(g, (K, N), code, -8, 8)
        P = I.to_storage(np.eye(M)[g.permutation(M)], code)
        tolerance.check_exact(run_gemm(P, B, code), oracle.gemm(P, B, code)[0], code, "perm %d" % M)
        A = I.small_int(g, (M, N), code, -8, 8)
        E = I.to_storage(np.eye(N), code)
        tolerance.check_exact(run_gemm(A, E, code), oracle.gemm(A, E, code)[0], code, "B=I %d" % M)


@pytest.mark.parametrize("code", DTS)
def test_random_shapes_integer_exact(code):
    g = I.rng(200 + code)
    for _ in range(25):
        M, N, K = (int(v) for v in g.integers(1, 301, size=3))
        r = max(1, min(8, I.exact_range(K, code)))
        lo = -r
        A = I.small_int(g, (M, K), code, lo, r)
        B = I.small_int(g, (K, N), code, lo, r)
        ref = oracle.gemm(A, B, code, with_mag=False)
        # inputs with K*r*r beyond the exact range still must be within bounds
        if K * r * r <= 2 ** {0: 24, 1: 11, 2: 8}[code]:
            tolerance.check_exact(run_gemm(A, B, code), ref, code, "int %dx%dx%d" % (M, N, K))
        else:
            ref, mag = oracle.gemm(A, B, code)
            tolerance.check(run_gemm(A, B, code), ref, mag, code, "int %dx%dx%d" % (M, N, K))


@pytest.mark.parametrize("code", DTS)
def test_rank1_closed_form(code):
    for K in (1, 5, 77, 300):
        M, N = 35, 70
        A = I.to_storage(np.ones((M, K)), code)
        Bk = np.tile(((np.arange(K) % 5) - 2.0)[:, None], (1, N))
        C = run_gemm(A, I.to_storage(Bk, code), code)
        q, r = divmod(K, 5)
        want = I.to_storage(np.full((M, N), r * (r - 1) / 2 - 2 * r), code)
        assert np.array_equal(C, want)


def test_rne_ties_on_device():
    # fp16: 2048 + 1 = 2049 -> 2048; 2048 + 3 = 2051 -> 2052 (ties to even)
    A = I.to_storage(np.ones((1, 2)), I.F16)
    B = I.to_storage(np.array([[2048.0, 2048.0], [1.0, 3.0]]), I.F16)
    C = run_gemm(A, B, I.F16)
    assert [int(v) for v in C[0]] == [0x6800, 0x6802]
    A = I.to_storage(np.ones((1, 2)), I.BF16)
    B = I.to_storage(np.array([[256.0, 256.0], [1.0, 3.0]]), I.BF16)
    C = run_gemm(A, B, I.BF16)
    assert [int(v) for v in C[0]] == [0x4380, 0x4382]


def test_fp16_subnormal_output():
    A = I.to_storage(np.full((3, 1), 2.0 ** -12), I.F16)
    B = I.to_storage(np.full((1, 5), 2.0 ** -12), I.F16)
    C = run_gemm(A, B, I.F16)
    assert np.all(C == 0x0001), C   # 2^-24, the smallest fp16 subnormal


def test_k_zero_writes_zeros_and_empty_is_noop():
    import torch
    from .gpu_util import empty_out
    for code in DTS:
        C = empty_out((5, 7), code, fill_bits=0x1234)
        A = empty_out((5, 0), code)
        B = empty_out((0, 7), code)
        st = vx.vx_gemm(5, 7, 0, code, A.data_ptr() or 0, B.data_ptr() or 0, C.data_ptr(),
                        torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
        assert not C.float().abs().sum().item()
        C2 = empty_out((3, 4), code, fill_bits=0x1234)
        st = vx.vx_gemm(0, 4, 6, code, 0, C.data_ptr(), C2.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
        bits = from_dev(C2, code)
        assert np.all((bits.view(np.uint32) if code == 0 else bits) == 0x1234)


@pytest.mark.parametrize("code", DTS)
def test_batched_and_broadcast(code):
    g = I.rng(300 + code)
    bt, M, N, K = 5, 37, 45, 29
    A = I.normal(g, (bt, M, K), code)
    B = I.normal(g, (bt, K, N), code)
    C = run_batched(A, M * K, B, K * N, code, bt, M, N, K).reshape(bt, M, N)
    ref, mag = oracle.gemm(A, B, code, M=M, N=N, K=K, batch=bt)
    tolerance.check(C, ref, mag, code, "batched")
    C = run_batched(A, M * K, B[0], 0, code, bt, M, N, K).reshape(bt, M, N)
    ref, mag = oracle.gemm(A, B[0], code, M=M, N=N, K=K, batch=bt, sB=0)
    tolerance.check(C, ref, mag, code, "broadcast B")


def _kernel_cases():
    """Every GEMM kernel of the registry (the convolution kernels have their own tests)."""
    n = vx.vx_registry_count()
    return [k for k in (vx.vx_registry_get(i) for i in range(n)) if k.op == 0]


def _shape_for(k, extra_m=3, extra_n=5, extra_k=8):
    """A ragged shape spanning 2 x 2 tiles and a K tail for kernel k."""
    M = 2 * k.mb + extra_m
    N = k.nb + (8 if k.align & 2 else extra_n)           # B's rows aligned only where the kernel needs it
    K = 2 * k.kb + (8 if k.align & 1 else extra_k + 1)   # likewise A's
    if k.k_max and K > k.k_max:                           # a kernel that holds its whole slice
        K = k.k_max - 8
    return M, N, K


@pytest.mark.parametrize("code", DTS)
def test_every_kernel_integer_exact(code):
    """Forces each compiled candidate of this dtype on a ragged multi-tile shape."""
    g = I.rng(400 + code)
    ran = 0
    for k in _kernel_cases():
        if k.dtype != code or not k.enabled:
            continue
        M, N, K = _shape_for(k)
        r = max(1, min(4, I.exact_range(K, code)))
        A = I.small_int(g, (M, K), code, -r, r)
        B = I.small_int(g, (K, N), code, -r, r)
        assert vx.vx_force_plan(k.id, 1) == 0
        C = run_gemm(A, B, code)
        vx.vx_force_plan(-1, 0)
        tolerance.check_exact(C, oracle.gemm(A, B, code, with_mag=False), code,
                              "kernel %d %s" % (k.id, (k.mb, k.nb, k.kb, k.wm, k.wn, k.mfma_m, k.vec)))
        ran += 1
    assert ran > 0


@pytest.mark.parametrize("code", [1, 2])
def test_every_ring_kernel_long_k(code):
    """Each direct-to-LDS kernel on a K range longer than its LDS ring: the
    prologue, the steady state with the ring full, the wrap of the stage
    index and the drain all run (plus a K tail in the last step)."""
    g = I.rng(450 + code)
    ran = 0
    for k in _kernel_cases():
        if k.dtype != code or not k.enabled or k.family != 1:
            continue
        M, N, _ = _shape_for(k)
        K = (k.stages + 2) * k.kb + 8
        r = max(1, min(4, I.exact_range(K, code)))
        A = I.small_int(g, (M, K), code, -r, r)
        B = I.small_int(g, (K, N), code, -r, r)
        assert vx.vx_force_plan(k.id, 1) == 0
        C = run_gemm(A, B, code)
        vx.vx_force_plan(-1, 0)
        tolerance.check_exact(C, oracle.gemm(A, B, code, with_mag=False), code,
                              "kernel %d %s stages %d K %d" % (k.id, (k.mb, k.nb, k.kb, k.wm, k.wn), k.stages, K))
        ran += 1
    assert ran > 0


@pytest.mark.parametrize("code", DTS)
def test_vector_alu_kernels_random_within_bound(code):
    """Every kernel of the vector-ALU family on random inputs: ragged M (below
    and above one tile's rows), a partial N tile, a K that ends inside a step;
    unsplit and with 3 K slices."""
    g = I.rng(470 + code)
    ran = 0
    for k in _kernel_cases():
        if k.dtype != code or not k.enabled or k.family != 2:
            continue
        for (M, N, K, split) in ((1, 200, 1000, 1), (k.mb + 3, 72, 3 * k.kb + 24, 3)):
            A = I.normal(g, (M, K), code)
            B = I.normal(g, (K, N), code, 0.02)
            assert vx.vx_force_plan(k.id, split) == 0
            C = run_gemm(A, B, code)
            vx.vx_force_plan(-1, 0)
            ref, mag = oracle.gemm(A, B, code)
            tolerance.check(C, ref, mag, code, "vector-ALU kernel %d M %d split %d" % (k.id, M, split))
        ran += 1
    assert ran > 0


@pytest.mark.parametrize("code", DTS)
@pytest.mark.parametrize("split", [2, 3, 5, 8])
def test_split_k_integer_exact(code, split):
    g = I.rng(500 + 10 * code + split)
    picked = [k for k in _kernel_cases() if k.dtype == code and k.enabled][::7]
    for k in picked:
        M, N, _ = _shape_for(k)
        K = split * k.kb + (8 if k.align & 1 else 5)
        r = max(1, min(4, I.exact_range(K, code)))
        A = I.small_int(g, (M, K), code, -r, r)
        B = I.small_int(g, (K, N), code, -r, r)
        assert vx.vx_force_plan(k.id, split) == 0
        C1 = run_gemm(A, B, code)
        C2 = run_gemm(A, B, code)      # counters must have reset themselves
        vx.vx_force_plan(-1, 0)
        ref = oracle.gemm(A, B, code, with_mag=False)
        tolerance.check_exact(C1, ref, code, "kernel %d split %d" % (k.id, split))
        assert np.array_equal(C1, C2)


@pytest.mark.parametrize("code", DTS)
def test_split_k_random_within_bound(code):
    g = I.rng(600 + code)
    M, N, K = 45, 72, 1000
    A = I.normal(g, (M, K), code)
    B = I.normal(g, (K, N), code, 0.02)
    ref, mag = oracle.gemm(A, B, code)
    for k in [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.vec][::11]:
        for split in (2, 4, 7):
            assert vx.vx_force_plan(k.id, split) == 0
            C = run_gemm(A, B, code)
            tolerance.check(C, ref, mag, code, "kernel %d split %d" % (k.id, split))
    vx.vx_force_plan(-1, 0)


@pytest.mark.parametrize("code", DTS)
def test_guard_bands_and_canaries(code):
    """NaN guard bands around A and B (an out-of-bounds read would leak NaN into
    C) and canaries around C (an out-of-bounds write would change them)."""
    import torch
    from .gpu_util import to_dev, empty_out
    g = I.rng(700 + code)
    nan = 0x7fc0 if code else 0x7fc00000
    for (M, N, K) in [(77, 96, 80), (33, 41, 19), (130, 264, 520), (5, 3, 1)]:
        pad = 4096
        A = I.normal(g, (M, K), code)
        B = I.normal(g, (K, N), code)
        bits_dt = np.uint32 if code == 0 else np.uint16
        Ag = np.full(M * K + 2 * pad, nan, dtype=bits_dt)
        Ag[pad:pad + M * K] = A.reshape(-1).view(bits_dt)
        Bg = np.full(K * N + 2 * pad, nan, dtype=bits_dt)
        Bg[pad:pad + K * N] = B.reshape(-1).view(bits_dt)
        At = to_dev(Ag.view(np.float32) if code == 0 else Ag, code)
        Bt = to_dev(Bg.view(np.float32) if code == 0 else Bg, code)
        Ct = empty_out((M * N + 2 * pad,), code, fill_bits=0x5a5a)
        for sp in (1, 3):
            ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.align == 0]
            for k in [None] + ks[::13]:
                vx.vx_force_plan(-1 if k is None else k.id, sp)
                st = vx.vx_gemm(M, N, K, code, At.data_ptr() + pad * At.element_size(),
                                Bt.data_ptr() + pad * Bt.element_size(), Ct.data_ptr() + pad * Ct.element_size(),
                                torch.cuda.current_stream().cuda_stream)
                vx.vx_force_plan(-1, 0)
                assert st == 0
                torch.cuda.synchronize()
                out = from_dev(Ct, code)
                raw = out.view(np.uint32) if code == 0 else out
                assert np.all(raw[:pad] == 0x5a5a) and np.all(raw[pad + M * N:] == 0x5a5a)
                ref, mag = oracle.gemm(A, B, code)
                tolerance.check(out[pad:pad + M * N].reshape(M, N), ref, mag, code, "guard %s" % ((M, N, K),))


def test_deterministic_bitwise():
    g = I.rng(800)
    A = I.normal(g, (300, 4096), I.BF16)
    B = I.normal(g, (4096, 1000), I.BF16, 0.02)
    C1 = run_gemm(A, B, I.BF16)
    for _ in range(3):
        assert np.array_equal(C1, run_gemm(A, B, I.BF16))


def test_error_codes_on_device():
    import torch
    s = torch.cuda.current_stream().cuda_stream
    x = torch.zeros(64, device="cuda", dtype=torch.float16)
    assert vx.vx_gemm(4, 4, 4, 9, x.data_ptr(), x.data_ptr() + 64, x.data_ptr() + 96, s) == 2
    assert vx.vx_gemm(4, 4, -1, 1, x.data_ptr(), x.data_ptr(), x.data_ptr(), s) == 1
    # C overlapping A
    assert vx.vx_gemm(4, 4, 4, 1, x.data_ptr(), x.data_ptr() + 64, x.data_ptr() + 8, s) == 1
    assert vx.vx_force_plan(10 ** 6, 1) == 3


def _hybrid_shape(k, code):
    """(M, N, tiles): an output one wave of kernel k's workgroups plus about a
    third of a wave, ragged in both directions."""
    num_cu = vx.vx_get_hwinfo().num_cu
    slots = num_cu * vx.vx_kernel_occupancy(k.id)
    target = slots + slots // 3 + 1
    tiles_n = max(2, min(16, target // 8))
    tiles_m = -(-target // tiles_n)
    M = tiles_m * k.mb - 3
    N = tiles_n * k.nb - (8 if k.align & 2 else 5)
    return M, N, tiles_m * tiles_n


def _tile_samples(g, M, N, mb, nb):
    """One random position in every output tile, plus the last row and column."""
    rows, cols = [], []
    for tm in range(-(-M // mb)):
        for tn in range(-(-N // nb)):
            rows.append(min(M - 1, tm * mb + int(g.integers(0, mb))))
            cols.append(min(N - 1, tn * nb + int(g.integers(0, nb))))
    rows += [M - 1] * 4 + list(g.integers(0, M, 4))
    cols += list(g.integers(0, N, 4)) + [N - 1] * 4
    return np.array(rows), np.array(cols)


@pytest.mark.parametrize("code", DTS)
def test_hybrid_grid_integer_exact(code):
    """The hybrid grid (whole waves of whole tiles, then the remaining tiles
    split into slices reduced by the last arrival) forced on kernels of each
    family: exact on integer inputs at one position of every tile, the same
    bits on a second call (the counters of the split tiles reset themselves)."""
    g = I.rng(900 + code)
    ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled]
    picked = {}
    for k in ks:
        picked.setdefault((k.family, k.align, k.mb * k.nb >= 128 * 128), k)
    ran = 0
    for k in picked.values():
        M, N, tiles = _hybrid_shape(k, code)
        for split in (2, 3):
            K = 2 * split * k.kb + (8 if k.align & 1 else 5)
            if k.k_max and K > k.k_max:
                continue
            r = max(1, min(3, I.exact_range(K, code)))
            A = I.small_int(g, (M, K), code, -r, r)
            B = I.small_int(g, (K, N), code, -r, r)
            assert vx.vx_force_plan(k.id, -split) == 0
            try:
                p = vx.vx_plan_query(1, M, N, K, code, M * K, K * N, M * N)
                assert p.dp_tiles > 0 and p.split_k == split and p.grid == p.dp_tiles + (tiles - p.dp_tiles) * split
                C1 = run_gemm(A, B, code)
                C2 = run_gemm(A, B, code)
            finally:
                vx.vx_force_plan(-1, 0)
            rows, cols = _tile_samples(g, M, N, k.mb, k.nb)
            ref, _ = oracle.gemm_sampled(A, B, code, M, N, K, rows, cols)
            tolerance.check_exact(C1[rows, cols], ref, code, "hybrid kernel %d split %d %dx%dx%d" % (k.id, split, M, N, K))
            assert np.array_equal(C1, C2)
            ran += 1
    assert ran >= 3


@pytest.mark.parametrize("code", [1, 2])
def test_hybrid_grid_random_within_bound(code):
    """The encoder's (M x 3072) x (3072 x 768) GEMM at M = 6976 with the hybrid
    grid forced on the 128 x 128 kernels for which it exists (330 tiles), random
    operands, sampled check."""
    g = I.rng(950 + code)
    M, N, K = 6976, 768, 3072
    A = I.normal(g, (M, K), code)
    B = I.normal(g, (K, N), code, 0.02)
    ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.vec and k.mb == 128 and k.nb == 128
          and vx.vx_plan_cost(1, M, N, K, code, k.id, -3, 3)[0] == 0]
    assert ks
    k = ks[0]
    assert vx.vx_force_plan(k.id, -3) == 0
    try:
        p = vx.vx_plan_query(1, M, N, K, code)
        C = run_gemm(A, B, code)
    finally:
        vx.vx_force_plan(-1, 0)
    assert p.dp_tiles > 0 and p.split_k == 3
    rows, cols = _tile_samples(g, M, N, k.mb, k.nb)
    ref, mag = oracle.gemm_sampled(A, B, code, M, N, K, rows, cols)
    tolerance.check(C[rows, cols], ref, mag, code, "hybrid kernel %d" % k.id)


@pytest.mark.parametrize("code", [1, 2])
def test_mixed_kernels_guard_bands(code):
    """Every mixed kernel (one operand by DMA, the one with unaligned rows
    through VGPRs) on a ragged shape whose other operand is unaligned, inside
    NaN guard bands (an out-of-bounds read would leak NaN into C) with
    canaries around C, random values within the bound."""
    import torch
    from .gpu_util import to_dev, empty_out
    g = I.rng(980 + code)
    nan = 0x7fc0
    pad = 4096
    ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.family == 1 and k.align in (1, 2)]
    assert ks
    for k in ks:
        M = 2 * k.mb + 3
        N = k.nb + (8 if k.align & 2 else 5)
        K = 2 * k.kb + (8 if k.align & 1 else 11)
        A = I.normal(g, (M, K), code)
        B = I.normal(g, (K, N), code)
        Ag = np.full(M * K + 2 * pad, nan, dtype=np.uint16)
        Ag[pad:pad + M * K] = A.reshape(-1).view(np.uint16)
        Bg = np.full(K * N + 2 * pad, nan, dtype=np.uint16)
        Bg[pad:pad + K * N] = B.reshape(-1).view(np.uint16)
        At, Bt = to_dev(Ag, code), to_dev(Bg, code)
        Ct = empty_out((M * N + 2 * pad,), code, fill_bits=0x5a5a)
        assert vx.vx_force_plan(k.id, 1) == 0
        try:
            st = vx.vx_gemm(M, N, K, code, At.data_ptr() + 2 * pad, Bt.data_ptr() + 2 * pad, Ct.data_ptr() + 2 * pad,
                            torch.cuda.current_stream().cuda_stream)
        finally:
            vx.vx_force_plan(-1, 0)
        assert st == 0, (k.id, vx.STATUS.get(st, st))
        torch.cuda.synchronize()
        out = from_dev(Ct, code)
        assert np.all(out[:pad] == 0x5a5a) and np.all(out[pad + M * N:] == 0x5a5a), k.id
        ref, mag = oracle.gemm(A, B, code)
        tolerance.check(out[pad:pad + M * N].reshape(M, N), ref, mag, code,
                        "mixed kernel %d align %d %s" % (k.id, k.align, (M, N, K)))


def _spread(ks, n):
    """Up to n kernels spread evenly over the list."""
    if len(ks) <= n:
        return ks
    return [ks[(i * (len(ks) - 1)) // (n - 1)] for i in range(n)]


@pytest.mark.parametrize("code", [1, 2])
def test_k_rotation_integer_exact_and_order_only(code):
    """Direct-to-LDS kernels of each schedule (plain ring, ping-pong, mixed)
    on a 3 x 3-tile shape whose K slice spans several steps and ends inside
    one, with the rotation switch on (the default; these operands fit in an
    XCD's L2, so the plain-ring kernels rotate their K order) and off, unsplit,
    split 3 and on a hybrid grid where the kernel has one.  Small-integer
    inputs make every sum exact, so both orders must equal the oracle bit for
    bit; repeated calls with the rotation must be bit-identical."""
    g = I.rng(1010 + code)
    ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.family == 1]
    groups = [[k for k in ks if k.schedule == 0 and k.align == 3], [k for k in ks if k.schedule == 1],
              [k for k in ks if k.align != 3]]
    assert all(groups), [len(x) for x in groups]
    ran = 0
    try:
        for grp in groups:
            for k in _spread(grp, 6):
                M = 3 * k.mb - 5
                N = 3 * k.nb - (8 if k.align & 2 else 3)
                K = 5 * k.kb + (8 if k.align & 1 else 9)
                r = max(1, min(3, I.exact_range(K, code)))
                A = I.small_int(g, (M, K), code, -r, r)
                B = I.small_int(g, (K, N), code, -r, r)
                ref = oracle.gemm(A, B, code, with_mag=False)
                for split in (1, 3, -2):
                    if vx.vx_plan_cost(1, M, N, K, code, k.id, split, k.align)[0] != 0:
                        continue   # no such plan for this kernel and shape (e.g. no hybrid split)
                    outs = []
                    for rot in (1, 0, 1):
                        assert vx.vx_enable_k_rotation(rot) == 0
                        assert vx.vx_force_plan(k.id, split) == 0
                        try:
                            C = run_gemm(A, B, code)
                        finally:
                            vx.vx_force_plan(-1, 0)
                        tolerance.check_exact(C, ref, code, "kernel %d sched %d align %d split %d rot %d %s" % (
                            k.id, k.schedule, k.align, split, rot, (M, N, K)))
                        outs.append(C)
                    assert np.array_equal(outs[0], outs[2]), k.id
                    ran += 1
    finally:
        vx.vx_enable_k_rotation(1)
    assert ran >= 12


@pytest.mark.parametrize("code", [1, 2])
def test_k_rotation_random_within_bound(code):
    """Random operands through rotated and in-order K on the same plans: both
    within the bound of the oracle, and the two results close to each other
    (they differ only in the fp32 summation order)."""
    g = I.rng(1030 + code)
    ks = [k for k in _kernel_cases() if k.dtype == code and k.enabled and k.family == 1 and k.align == 3]
    try:
        for k in _spread(ks, 8):
            M, N, K = 2 * k.mb + 7, 2 * k.nb + 8, 4 * k.kb + 24
            A = I.normal(g, (M, K), code)
            B = I.normal(g, (K, N), code, 0.02)
            ref, mag = oracle.gemm(A, B, code)
            res = []
            for rot in (1, 0):
                assert vx.vx_enable_k_rotation(rot) == 0
                assert vx.vx_force_plan(k.id, 1) == 0
                try:
                    C = run_gemm(A, B, code)
                finally:
                    vx.vx_force_plan(-1, 0)
                tolerance.check(C, ref, mag, code, "kernel %d rot %d" % (k.id, rot))
                res.append(oracle.decode(C, code).astype(np.float64))
            assert np.all(np.abs(res[0] - res[1]) <= 8e-3 * mag + 1e-6), k.id
    finally:
        vx.vx_enable_k_rotation(1)
