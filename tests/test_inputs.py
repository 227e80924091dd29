"""The seeded workload recipes stay inside the ranges the paper's CNN family
states (Table 4: batch 1..64, map 4..768, filter 1..11, Cin 3..832,
Cout 16..512) and inside the size caps the convolution set applies."""
import pytest

from paper_2409_01075_amd import inputs as I


@pytest.mark.parametrize("cin", ["models", "plain"])
def test_conv_trial_ranges(cin):
    layers = [I.conv_trial(t, cin) for t in range(40)]
    for (N, H, W, Ci, Co, F, st, pd) in layers:
        assert 1 <= N <= 64 and H == W and F <= H <= 768 and F in (1, 3, 5, 7, 11)
        assert 3 <= Ci <= 832 and 16 <= Co <= 512 and pd == F // 2 and st in (1, 2, 4)
        OH = (H + 2 * pd - F) // st + 1
        assert N * H * W * Ci <= 2 ** 25 and N * OH * OH * Co <= 2 ** 25
        assert 2.0 * N * OH * OH * Co * F * F * Ci <= 4e11
    odd = sum(L[3] % 8 != 0 for L in layers)
    if cin == "models":
        assert all(L[3] == 3 or L[3] % 8 == 0 for L in layers)
    else:
        assert odd >= 30          # log-uniform over 3..832: about 7 in 8 are not multiples of 8


def test_conv_trial_plain_keeps_other_draws():
    for t in range(40):
        a, b = I.conv_trial(t), I.conv_trial(t, "plain")
        assert a[4:] == b[4:]     # Cout, filter, stride, padding come from the same stream
    with pytest.raises(ValueError):
        I.conv_trial(0, "other")
