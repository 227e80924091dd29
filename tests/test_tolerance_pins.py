"""Pins for the acceptance checker (oracle/tolerance.py), on the CPU.

Every parity claim goes through ``tolerance.check`` (random inputs, bound
|C - Cref| <= 4e-3 Mag + 1e-6 for fp16/bf16; 1e-5 Mag elementwise and
1e-5 relative Frobenius norm for fp32) and ``tolerance.check_exact``
(integer-exact inputs, bit for bit).  These tests put C just inside and just
outside each bound, so that a slip in the checker (the bound taken against
|Cref| instead of Mag, an inverted comparison, a missing normwise test, a
value comparison where bits are meant) fails one of them.  C is given as the
stored bits of the output type; bit patterns below are written out from the
IEEE formats (fp16: 1 sign, 5 exponent, 10 fraction bits; bf16: the top 16
bits of an fp32).
"""
import numpy as np
import pytest

from oracle import F32, F16, BF16
from oracle import tolerance

# 1.0 and the next representable value up, per 16-bit type
ONE = {F16: 0x3C00, BF16: 0x3F80}
ULP_AT_ONE = {F16: 2.0 ** -10, BF16: 2.0 ** -7}


def _bits16(vals):
    return np.array(vals, dtype=np.uint16)


def _f32bits(vals):
    return np.array(vals, dtype=np.float32)


# ------------------------------------------------------ fp16 / bf16 bound ---

@pytest.mark.parametrize("code", [F16, BF16])
def test_16bit_one_ulp_inside_and_outside(code):
    """C = 1 + ulp against Cref = 1: passes when the bound is 1.1 ulp, fails
    when it is 0.9 ulp (Mag chosen from 4e-3 Mag + 1e-6 = target)."""
    ulp = ULP_AT_ONE[code]
    C = _bits16([ONE[code] + 1])
    for frac, ok in ((1.1, True), (0.9, False)):
        mag = (frac * ulp - 1e-6) / 4e-3
        if ok:
            r = tolerance.check(C, np.array([1.0]), np.array([mag]), code, "inside")
            assert 0.9 < r <= 1.0
        else:
            with pytest.raises(AssertionError):
                tolerance.check(C, np.array([1.0]), np.array([mag]), code, "outside")


@pytest.mark.parametrize("code", [F16, BF16])
def test_16bit_bound_edge_in_binary64(code):
    """|C - Cref| a hair below and a hair above 4e-3 Mag + 1e-6 exactly."""
    C = _bits16([ONE[code]] * 3)
    mag = np.array([0.5, 3.0, 0.0])
    bound = 4e-3 * mag + 1e-6
    r = tolerance.check(C, 1.0 - bound * (1 - 1e-9), mag, code, "below")
    assert r <= 1.0
    tolerance.check(C, 1.0 + bound * (1 - 1e-9), mag, code, "below, other side")
    for i in range(3):
        ref = 1.0 - bound * (1 - 1e-9)
        ref[i] = 1.0 - bound[i] * (1 + 1e-6)
        with pytest.raises(AssertionError):
            tolerance.check(C, ref, mag, code, "above at %d" % i)


@pytest.mark.parametrize("code", [F16, BF16])
def test_16bit_bound_uses_mag_not_cref(code):
    """Cancellation: Cref = 0 with Mag = 1.  An error of 1e-3 is inside
    4e-3 * Mag + 1e-6 (it would fail a bound taken on |Cref|); an error of
    5e-3 is outside."""
    small = np.float16(2.0 ** -10).view(np.uint16) if code == F16 else 0x3A80   # 2^-10 in bf16: exp 117
    C = _bits16([small])
    assert tolerance.check(C, np.array([0.0]), np.array([1.0]), code) <= 1.0
    big = np.float16(2.0 ** -7).view(np.uint16) if code == F16 else 0x3C00      # 2^-7 in bf16: exp 120
    with pytest.raises(AssertionError):
        tolerance.check(_bits16([big]), np.array([0.0]), np.array([1.0]), code)


@pytest.mark.parametrize("code", [F16, BF16])
def test_16bit_absolute_term(code):
    """Mag = 0 leaves the 1e-6 absolute term: 2^-24 (fp16 subnormal, ~6e-8)
    passes against 0; 2^-19 (~1.9e-6) fails."""
    if code == F16:
        tiny, over = 0x0001, 0x0020                 # 2^-24, 2^-19 (subnormals)
    else:
        tiny, over = 0x3380, 0x3600                 # 2^-24, 2^-19
    assert tolerance.check(_bits16([tiny]), np.array([0.0]), np.array([0.0]), code) <= 1.0
    with pytest.raises(AssertionError):
        tolerance.check(_bits16([over]), np.array([0.0]), np.array([0.0]), code)


@pytest.mark.parametrize("code", [F16, BF16])
@pytest.mark.parametrize("bad", ["nan", "inf", "-inf"])
def test_16bit_non_finite_rejected(code, bad):
    pattern = {F16: {"nan": 0x7E00, "inf": 0x7C00, "-inf": 0xFC00},
               BF16: {"nan": 0x7FC0, "inf": 0x7F80, "-inf": 0xFF80}}[code][bad]
    C = _bits16([ONE[code], pattern])
    with pytest.raises(AssertionError):
        tolerance.check(C, np.array([1.0, 1.0]), np.array([1e30, 1e30]), code)


@pytest.mark.parametrize("code", [F16, BF16, F32])
def test_shape_mismatch_rejected(code):
    C = _bits16([ONE[code]] * 6) if code != F32 else _f32bits([1.0] * 6)
    with pytest.raises(AssertionError):
        tolerance.check(C.reshape(2, 3), np.ones((3, 2)), np.ones((3, 2)), code)


def test_worst_offender_is_reported_not_first():
    """A large error after many small ones still fails (the maximum ratio is
    what is compared)."""
    C = _bits16([ONE[F16]] * 100)
    ref = np.ones(100)
    ref[97] = 1.0 + 0.05
    with pytest.raises(AssertionError, match="97"):
        tolerance.check(C, ref, np.ones(100), F16)


# ------------------------------------------------------------ fp32 bound ----

def test_f32_elementwise_inside_and_outside():
    """|C - Cref| at one element 1 % and (1 + 1e-6) times 1e-5 * Mag, while the
    other elements keep the relative Frobenius error far below 1e-5."""
    C = _f32bits([2.0] + [1000.0] * 10)
    mag = np.array([8.0] + [1000.0] * 10)
    ref = np.array([2.0] + [1000.0] * 10)
    assert tolerance.check(C, ref, mag, F32) == 0.0
    ref_in = ref.copy()
    ref_in[0] = 2.0 - 1e-5 * 8.0 * 0.99
    assert 0.98 < tolerance.check(C, ref_in, mag, F32) <= 1.0
    ref_out = ref.copy()
    ref_out[0] = 2.0 - 1e-5 * 8.0 * (1 + 1e-6)   # normwise 8e-5 / 3162 is far inside
    with pytest.raises(AssertionError, match="exceeds bound"):
        tolerance.check(C, ref_out, mag, F32)


def test_f32_normwise_checked_separately():
    """Every element within 1e-5 * Mag (Mag large), but the relative Frobenius
    error 2e-5 is over 1e-5: must fail on the norm."""
    n = 64
    ref = np.ones(n)
    C = (ref * (1 + 2e-5)).astype(np.float32)
    mag = np.full(n, 100.0)
    with pytest.raises(AssertionError, match="normwise"):
        tolerance.check(C, ref, mag, F32)
    C_ok = (ref * (1 + 2.0 ** -20)).astype(np.float32)   # ~9.5e-7 relative
    assert tolerance.check(C_ok, ref, mag, F32) <= 1.0


def test_f32_zero_mag():
    """Mag = 0 (an all-zero row or column): only C = Cref exactly passes."""
    assert tolerance.check(_f32bits([0.0, 1.0]), np.array([0.0, 1.0]), np.array([0.0, 1.0]), F32) == 0.0
    with pytest.raises(AssertionError):
        tolerance.check(_f32bits([1e-30, 1.0]), np.array([0.0, 1.0]), np.array([0.0, 1.0]), F32)


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_f32_non_finite_rejected(bad):
    with pytest.raises(AssertionError):
        tolerance.check(_f32bits([1.0, bad]), np.array([1.0, 1.0]), np.array([1e30, 1e30]), F32)


# ------------------------------------------------------------ bit exact -----

@pytest.mark.parametrize("code", [F16, BF16, F32])
def test_exact_passes_identical_and_rejects_one_flipped_bit(code):
    vals = np.array([[1.0, -3.0, 0.5], [2048.0, 0.0, -7.0]])
    if code == F16:
        good = vals.astype(np.float16).view(np.uint16)
    elif code == BF16:
        good = (vals.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)   # exact in bf16
    else:
        good = vals.astype(np.float32)
    tolerance.check_exact(good, vals, code)
    for idx in [(0, 0), (1, 2), (1, 1)]:
        bad = good.copy()
        if code == F32:
            b = bad.view(np.uint32)
            b[idx] ^= 1
        else:
            bad[idx] ^= 1
        with pytest.raises(AssertionError, match="mismatching"):
            tolerance.check_exact(bad, vals, code)


def test_exact_compares_bits_not_values():
    """-0.0 and +0.0 are equal as values but not as bits: a comparison made on
    decoded values would pass them."""
    neg0 = np.array([-0.0])
    with pytest.raises(AssertionError):
        tolerance.check_exact(np.array([0.0], np.float32), neg0, F32)
    with pytest.raises(AssertionError):
        tolerance.check_exact(np.array([0.0], np.float16), neg0, F16)
    with pytest.raises(AssertionError):
        tolerance.check_exact(_bits16([0x0000]), neg0, BF16)
    tolerance.check_exact(_bits16([0x8000]), neg0, BF16)
    tolerance.check_exact(np.array([-0.0], np.float32), neg0, F32)


def test_exact_storage_views():
    """fp16 outputs as float16, uint16 or int16 arrays are read as the same bits."""
    vals = np.array([1.0, -2.5, 65504.0])
    h = vals.astype(np.float16)
    tolerance.check_exact(h, vals, F16)
    tolerance.check_exact(h.view(np.uint16), vals, F16)
    tolerance.check_exact(h.view(np.int16), vals, F16)
    with pytest.raises(AssertionError):
        tolerance.check_exact(h.view(np.int16)[::-1].copy(), vals, F16)


def test_exact_rounds_reference_to_nearest_even():
    """The reference is the RNE encoding of Cref: 2049 -> 2048 and 2051 -> 2052
    in fp16; C holding 2050 (the other neighbour of 2049) is rejected."""
    C = np.array([2048.0, 2052.0], np.float16)
    tolerance.check_exact(C, np.array([2049.0, 2051.0]), F16)
    with pytest.raises(AssertionError):
        tolerance.check_exact(np.array([2050.0, 2052.0], np.float16), np.array([2049.0, 2051.0]), F16)


def test_exact_shape_mismatch():
    with pytest.raises(AssertionError):
        tolerance.check_exact(np.zeros((2, 3), np.float32), np.zeros((3, 2)), F32)
