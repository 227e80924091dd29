"""GPU parity of the 2-D convolution (implicit GEMM on the same hierarchy)
against the CPU oracle's direct convolution, through the C ABI."""
import numpy as np
import pytest

import oracle
from oracle import tolerance
from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

from .gpu_util import from_dev, to_dev

pytestmark = pytest.mark.gpu

DTS = [0, 1, 2]


def run_conv(x, w, code, stride=(1, 1), pad=(0, 0), dil=(1, 1)):
    import torch
    y = vx.conv2d(to_dev(x, code), to_dev(w, code), stride, pad, dil)
    torch.cuda.synchronize()
    return from_dev(y, code)


CASES = [
    # N, H, W, Cin, Cout, KH, KW, stride, pad, dil
    (1, 9, 11, 3, 16, 3, 3, (1, 1), (1, 1), (1, 1)),       # first-layer channels: element gathers
    (2, 16, 13, 8, 24, 3, 3, (2, 2), (1, 1), (1, 1)),      # whole 16-byte chunks, stride 2
    (2, 12, 12, 16, 40, 5, 5, (1, 2), (2, 2), (1, 1)),
    (3, 10, 9, 24, 8, 3, 2, (1, 1), (2, 1), (2, 3)),       # dilation, asymmetric filter
    (1, 7, 7, 64, 72, 1, 1, (1, 1), (0, 0), (1, 1)),       # 1 x 1: a plain GEMM of the pixels
    (2, 8, 6, 5, 9, 7, 7, (1, 1), (3, 3), (1, 1)),         # filter larger than the image, ragged tiles
    (1, 33, 31, 32, 130, 3, 3, (1, 1), (1, 1), (1, 1)),    # several tiles in both directions
]


@pytest.mark.parametrize("code", DTS)
def test_conv_random_within_bound(code):
    g = I.rng(1100 + code)
    for (N, H, W, Cin, Cout, KH, KW, st, pd, dl) in CASES:
        x = I.normal(g, (N, H, W, Cin), code)
        w = I.normal(g, (KH, KW, Cin, Cout), code, 0.1)
        y = run_conv(x, w, code, st, pd, dl)
        ref, mag = oracle.conv2d(x, w, code, st, pd, dl)
        tolerance.check(y, ref, mag, code, "conv %s" % ((N, H, W, Cin, Cout, KH, KW, st, pd, dl),))


@pytest.mark.parametrize("code", DTS)
def test_every_conv_kernel_integer_exact(code):
    """Each convolution kernel forced on a ragged case with padding, stride
    and dilation; small integers make every result exact."""
    g = I.rng(1200 + code)
    ks = [k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count()))
          if k.op == 1 and k.dtype == code and k.enabled]
    assert ks
    for k in ks:
        # the direct-to-LDS kernels take channel counts that are multiples of 8
        for Cin in ((8, 24) if k.align & 1 else (3, 8)):   # image by DMA: channels in 16-byte chunks
            Cout = k.nb + (8 if k.align & 2 else 5)          # filter by DMA: rows of 16-byte chunks
            N, H, W, KH, KW, st, pd, dl = 2, 11, 10, 3, 3, (2, 1), (1, 2), (1, 2)
            x = I.small_int(g, (N, H, W, Cin), code, -3, 3)
            w = I.small_int(g, (KH, KW, Cin, Cout), code, -3, 3)
            assert vx.vx_force_plan(k.id, 1) == 0
            try:
                y = run_conv(x, w, code, st, pd, dl)
            finally:
                vx.vx_force_plan(-1, 0)
            ref = oracle.conv2d(x, w, code, st, pd, dl, with_mag=False)
            tolerance.check_exact(y, ref, code, "conv kernel %d Cin %d" % (k.id, Cin))


@pytest.mark.parametrize("code", DTS)
def test_every_register_conv_kernel_contiguous_taps(code):
    """The convolution kernels that gather the image through VGPRs (the
    register-staged ones, and the mixed ones that take the filter by DMA) with
    channel counts that are not multiples of the 16-byte chunk and unit
    dilation along the width: chunks that stay inside one filter row load as
    one vector, chunks across a filter row's end, on padding or past K are
    gathered element by element.  A 3 x 5 filter with c_in 3, 5 and 12 puts
    chunk boundaries at every position of a row; small integers make every
    result exact."""
    g = I.rng(1250 + code)
    ks = [k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count()))
          if k.op == 1 and k.dtype == code and k.enabled and not k.align & 1]
    assert ks
    for k in ks:
        for Cin in (3, 5, 12):
            Cout = k.nb + (8 if k.align & 2 else 5)
            N, H, W, KH, KW, st, pd, dl = 2, 11, 13, 3, 5, (1, 2), (2, 1), (2, 1)
            x = I.small_int(g, (N, H, W, Cin), code, -3, 3)
            w = I.small_int(g, (KH, KW, Cin, Cout), code, -3, 3)
            assert vx.vx_force_plan(k.id, 1) == 0
            try:
                y = run_conv(x, w, code, st, pd, dl)
            finally:
                vx.vx_force_plan(-1, 0)
            ref = oracle.conv2d(x, w, code, st, pd, dl, with_mag=False)
            tolerance.check_exact(y, ref, code, "conv kernel %d Cin %d, unit width dilation" % (k.id, Cin))


@pytest.mark.parametrize("code", DTS)
def test_conv_split_k_integer_exact(code):
    g = I.rng(1300 + code)
    conv = [k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count()))
            if k.op == 1 and k.dtype == code and k.enabled]
    N, H, W, Cout, KH, KW = 1, 9, 9, 24, 3, 3
    firsts = {}
    for k in conv:
        firsts.setdefault((k.family, k.align), k)
    for k, split in ((k, s) for k in firsts.values() for s in (2, 3)):
        Cin = 40 if k.align & 1 else 37   # channels in whole chunks only where the image is DMA'd
        x = I.small_int(g, (N, H, W, Cin), code, -2, 2)
        w = I.small_int(g, (KH, KW, Cin, Cout), code, -2, 2)
        ref = oracle.conv2d(x, w, code, (1, 1), (1, 1), (1, 1), with_mag=False)
        assert vx.vx_force_plan(k.id, split) == 0
        try:
            y1 = run_conv(x, w, code, (1, 1), (1, 1), (1, 1))
            y2 = run_conv(x, w, code, (1, 1), (1, 1), (1, 1))
        finally:
            vx.vx_force_plan(-1, 0)
        tolerance.check_exact(y1, ref, code, "conv kernel %d split %d" % (k.id, split))
        assert np.array_equal(y1, y2)


def test_conv_zero_channels_and_empty_output():
    import torch
    dev = torch.device("cuda:0")
    x = torch.zeros((1, 4, 4, 0), dtype=torch.float16, device=dev)
    w = torch.zeros((3, 3, 0, 8), dtype=torch.float16, device=dev)
    y = torch.full((1, 4, 4, 8), 7.0, dtype=torch.float16, device=dev)
    vx.conv2d(x, w, padding=(1, 1), out=y)
    torch.cuda.synchronize()
    assert torch.all(y == 0)
    # a filter larger than the padded image: no output, nothing written
    x = torch.ones((1, 2, 2, 8), dtype=torch.float16, device=dev)
    w = torch.ones((5, 5, 8, 8), dtype=torch.float16, device=dev)
    assert vx.conv2d(x, w).numel() == 0


@pytest.mark.parametrize("code", [1, 2])
def test_conv_hybrid_grid_integer_exact(code):
    """A convolution whose implicit GEMM has more tiles than one wave of the
    device (the image sized for the kernel), with the hybrid grid forced on a
    direct-to-LDS and a register-staged convolution kernel: exact on integer
    inputs, and the same bits on a second call."""
    g = I.rng(1400 + code)
    num_cu = vx.vx_get_hwinfo().num_cu
    Cin, KH, KW = 16, 3, 3
    ran = 0
    for fam in (1, 0):
        k = next(k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count()))
                 if k.op == 1 and k.dtype == code and k.enabled and k.family == fam)
        slots = num_cu * vx.vx_kernel_occupancy(k.id)
        Cout = 2 * k.nb - 8                                  # two tile columns, the second ragged
        tiles_m = -(-(slots + slots // 3 + 1) // 2)
        H = 32
        W = -(-(tiles_m * k.mb - k.mb // 2) // H)             # M = H * W, the last tile row ragged
        M = H * W
        tiles = -(-M // k.mb) * 2
        assert tiles > slots and tiles % slots != 0
        x = I.small_int(g, (1, H, W, Cin), code, -2, 2)
        w = I.small_int(g, (KH, KW, Cin, Cout), code, -2, 2)
        ref = oracle.conv2d(x, w, code, (1, 1), (1, 1), (1, 1), with_mag=False)
        assert vx.vx_force_plan(k.id, -2) == 0
        try:
            d = vx.conv_desc(1, H, W, Cin, Cout, KH, KW, code, pad=(1, 1))
            p = vx.vx_conv2d_plan_query(d)
            assert p.dp_tiles > 0 and p.split_k == 2
            y1 = run_conv(x, w, code, (1, 1), (1, 1), (1, 1))
            y2 = run_conv(x, w, code, (1, 1), (1, 1), (1, 1))
        finally:
            vx.vx_force_plan(-1, 0)
        tolerance.check_exact(y1, ref, code, "conv hybrid kernel %d" % k.id)
        assert np.array_equal(y1, y2)
        ran += 1
    assert ran == 2
