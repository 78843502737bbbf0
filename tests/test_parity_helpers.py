"""The y checks of the GPU parity tests, on the CPU: they accept the
correctly rounded oracle output, and catch an element a few bf16 ulps off."""

import numpy as np
import pytest

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I

from parity_helpers import check_y_elements, check_y_per_token, oracle_factors, scale_pieces, y_abs_terms


@pytest.fixture(scope="module")
def small_layer():
    d = I.custom(M=64, K=256, N=16, r=16, seed=3, n_outliers=2)
    f = oracle_factors(d, 16)
    ref = O.asp_linear(d.x, f)
    at = y_abs_terms(ref["sx"], ref["sw"], ref["P"], ref["t"], f["L2"])
    return ref, at


def test_correctly_rounded_output_passes(small_layer):
    ref, at = small_layer
    yb = O.f64_to_bf16_bits(ref["y"])
    check_y_per_token(yb, ref["y"], at, ref["P"].shape[2], 16)
    check_y_elements(yb, ref["y"], at, ref["P"].shape[2], 16)


@pytest.mark.parametrize("ulps", [2, 3, -3])
def test_element_off_by_ulps_is_caught(small_layer, ulps):
    ref, at = small_layer
    yb = O.f64_to_bf16_bits(ref["y"]).copy()
    yb[5, 3] = np.uint16(int(yb[5, 3]) + ulps)
    with pytest.raises(AssertionError):
        check_y_elements(yb, ref["y"], at, ref["P"].shape[2], 16)
    if abs(ulps) >= 3:
        with pytest.raises(AssertionError):
            check_y_per_token(yb, ref["y"], at, ref["P"].shape[2], 16)


def test_scale_pieces_are_the_nearest_two_bf16_split():
    """wsp's two pieces: hi is the nearest bf16 of s, lo the nearest bf16 of
    the exact remainder: |hi - s| <= 2^-8 |s| (half a unit in hi's eighth
    significant bit) and |hi + lo - s| <= 2^-16 |s|."""
    rng = np.random.default_rng(0)
    s = (rng.lognormal(-4, 2, 4096)).astype(np.float32)
    s[:4] = [0.0, 1.0, 3.0 / 7.0, np.float32(2.0 ** -120)]
    w = scale_pieces(s)
    hi = O.bf16_bits_to_f64((w & 0xFFFF).astype(np.uint16))
    lo = O.bf16_bits_to_f64((w >> 16).astype(np.uint16))
    s64 = s.astype(np.float64)
    assert (np.abs(hi - s64) <= 2.0 ** -8 * np.abs(s64)).all()
    assert (np.abs(hi + lo - s64) <= 2.0 ** -16 * np.abs(s64)).all()
    assert w[0] == 0 and w[1] == 0x3F80
