"""Acceptance checks of a computed C against the oracle (test infrastructure).

Bounds, elementwise, with Mag = |A| x |B| from the oracle:
  * fp16 / bf16 inputs (fp32 accumulation, rounded output):
        |C - Cref| <= 4e-3 * Mag + 1e-6
    The bound covers the output rounding (at most 2^-9 |C| for bf16) plus fp32
    accumulation error (at most about K * 2^-24 * Mag, 6.6e-4 Mag at K=11008).
  * fp32 inputs: |C - Cref| <= 1e-5 * Mag elementwise and
        ||C - Cref||_F <= 1e-5 * ||Cref||_F.
  * integer-exact inputs: C must equal the oracle's RNE encoding bit for bit.
"""
import numpy as np

from . import F32, F16, BF16, dtype_code, encode, decode


def check(C_bits, Cref, Mag, dtype, what=""):
    """Raises AssertionError with the worst offender when the bound fails.

    Returns the max ratio |C - Cref| / bound (<= 1 passes).
    """
    code = dtype_code(dtype)
    C = decode(C_bits, code)
    Cref = np.asarray(Cref, dtype=np.float64)
    Mag = np.asarray(Mag, dtype=np.float64)
    if C.shape != Cref.shape:
        raise AssertionError("%s: shape %s != %s" % (what, C.shape, Cref.shape))
    if C.size == 0:
        return 0.0
    if not np.all(np.isfinite(C)):
        bad = np.argwhere(~np.isfinite(C))[0]
        raise AssertionError("%s: non-finite output at %s" % (what, tuple(bad)))
    err = np.abs(C - Cref)
    if code == F32:
        bound = 1e-5 * Mag
        ratio = np.where(bound > 0, err / np.where(bound > 0, bound, 1), np.where(err > 0, np.inf, 0))
        nref = np.linalg.norm(Cref)
        nerr = np.linalg.norm(C - Cref)
        if nerr > 1e-5 * nref:
            raise AssertionError("%s: normwise error %.3e > 1e-5 * %.3e" % (what, nerr, nref))
    else:
        bound = 4e-3 * Mag + 1e-6
        ratio = err / bound
    worst = float(ratio.max())
    if worst > 1.0:
        idx = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
        raise AssertionError("%s: |C-Cref| exceeds bound at %s: C=%r ref=%r mag=%r ratio=%.3f"
                             % (what, idx, C[idx], Cref[idx], Mag[idx], worst))
    return worst


def check_exact(C_bits, Cref, dtype, what=""):
    """Bit-exact comparison with RNE_dtype(Cref) (integer-exact inputs)."""
    code = dtype_code(dtype)
    want = encode(Cref, code)
    got = np.ascontiguousarray(C_bits)
    if code == F16 and got.dtype == np.float16:
        got = got.view(np.uint16)
    if got.dtype == np.int16:
        got = got.view(np.uint16)
    if code == F32:
        got = got.view(np.uint32)
        want = want.view(np.uint32)
    if got.shape != want.shape:
        raise AssertionError("%s: shape %s != %s" % (what, got.shape, want.shape))
    diff = got != want
    if diff.any():
        idx = tuple(np.argwhere(diff)[0])
        raise AssertionError("%s: %d mismatching elements, first at %s: got bits %#x want %#x"
                             % (what, int(diff.sum()), idx, int(got[idx]), int(want[idx])))
