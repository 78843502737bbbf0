"""The y checks of the GPU parity tests, on the CPU: they accept the
correctly rounded oracle output, and catch an element a few bf16 ulps off."""

import numpy as np
import pytest

from oracle import qwam_oracle as O
from paper_2609_33269_amd import inputs as I

from parity_helpers import check_y_elements, check_y_per_token, oracle_factors, y_abs_terms


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
