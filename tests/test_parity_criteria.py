"""The row criterion of T2 on constructed rows (no GPU).

O_i = num_i / den_i (Eq.(linear att)).  While the rounding bound of den_i,
4 u den_abs_i, is below |den_i|, a row's relative error is bounded by
4 u times its condition number.  Where the bound reaches |den_i|, den_i may
change sign within rounding and O_i is not determined: such a row is checked
on num_i and den_i against their absolute scales.
"""
import numpy as np
import pytest

from tests.parity import check_forward, UNIT


N, DV = 64, 2


def _rows():
    rng = np.random.default_rng(5)
    num_ref = rng.uniform(0.5, 1.5, (1, 1, N, DV))
    den_ref = rng.uniform(0.5, 1.5, (1, 1, N))
    den_abs = np.full((1, 1, N), 10.0)
    num_abs = np.full((1, 1, N, DV), 10.0)
    den_ref[0, 0, 7] = 1e-3          # 4 u den_abs = 0.078 > |den|: O_7 undetermined
    O_ref = num_ref / den_ref[..., None]
    kappa = den_abs / np.abs(den_ref)
    return O_ref, den_ref, (num_abs, den_abs), kappa


def test_undetermined_row_checked_on_num_and_den():
    O_ref, den_ref, scales, kappa = _rows()
    den = den_ref.copy()
    den[0, 0, 7] = 1e-6              # |error| 1e-3, 1 % of the den bound; O_7 off by 1000x
    O = O_ref * (den_ref / den)[..., None]
    check_forward("bf16", O, den, O_ref, den_ref, kappa, scales)


def test_undetermined_row_den_error_beyond_its_scale_fails():
    O_ref, den_ref, scales, kappa = _rows()
    den = den_ref.copy()
    den[0, 0, 7] = 0.2               # |error| 0.2 > 4 u den_abs = 0.078
    assert 0.2 > 4 * UNIT["bf16"] * 10.0
    O = O_ref * (den_ref / den)[..., None]
    with pytest.raises(AssertionError):
        check_forward("bf16", O, den, O_ref, den_ref, kappa, scales)


def test_determined_row_relative_error_fails():
    O_ref, den_ref, scales, kappa = _rows()
    O = O_ref.copy()
    O[0, 0, 3] *= 1.5                # a well-conditioned row 50 % off
    with pytest.raises(AssertionError):
        check_forward("bf16", O, den_ref.copy(), O_ref, den_ref, kappa, scales)


def test_zero_den_row_passes_only_where_den_is_undetermined():
    """den_i = 0 exactly gives a non-finite O_i (no epsilon, as defined).  At an
    undetermined row that is within rounding; at a determined row it fails."""
    O_ref, den_ref, scales, kappa = _rows()
    for row, ok in ((7, True), (3, False)):
        den = den_ref.copy()
        den[0, 0, row] = 0.0
        O = O_ref.copy()
        O[0, 0, row] = np.nan
        if ok:
            check_forward("bf16", O, den, O_ref, den_ref, kappa, scales)
        else:
            with pytest.raises(AssertionError):
                check_forward("bf16", O, den, O_ref, den_ref, kappa, scales)
