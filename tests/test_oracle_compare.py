"""Pins of the parity metric (oracle/compare.py) by hand-computed values.

rel = max over rows r of ||T_r - R_r||_inf / max(||R_r||_inf, 1e-3 ||R||_inf); the rows are the first
axis (everything after it flattened), one row for 1-D tensors and for whole=True.  Every expected value
below is worked out by hand from that definition, so a metric that loosened (min instead of max over
rows, the floor dropped or applied to the wrong norm, whole= ignored, rows cut along another axis) or
that let a NaN pass fails here."""
import math

import numpy as np
import pytest

from oracle.compare import rel_err


def test_row_below_the_floor_is_judged_against_the_floor():
    R = np.array([[10.0, -2.0], [0.001, 0.0005]])
    T = np.array([[10.5, -2.0], [0.002, 0.0005]])
    # row 0: 0.5 / 10 = 0.05; row 1: |0.002 - 0.001| / max(0.001, 1e-3 * 10) = 0.001 / 0.01 = 0.1
    assert rel_err(T, R) == pytest.approx(0.1, rel=1e-12)


def test_row_above_the_floor_uses_its_own_scale():
    R = np.array([[10.0, -2.0], [0.5, -0.25]])
    T = np.array([[10.0, -2.0], [0.5, -0.30]])
    # row 1: 0.05 / 0.5 = 0.1 (the floor 0.01 is below the row's own max 0.5)
    assert rel_err(T, R) == pytest.approx(0.1, rel=1e-12)


def test_the_worst_row_decides():
    R = np.array([[1.0, 1.0], [1.0, 1.0], [4.0, 0.0]])
    T = np.array([[1.1, 1.0], [1.0, 0.7], [4.0, 0.0]])
    # rows: 0.1, 0.3, 0.0 -> 0.3
    assert rel_err(T, R) == pytest.approx(0.3, rel=1e-12)


def test_negative_reference_uses_the_absolute_maximum():
    R = np.array([[-8.0, 1.0]])
    T = np.array([[-8.0, 1.4]])
    # 0.4 / 8 = 0.05
    assert rel_err(T, R) == pytest.approx(0.05, rel=1e-12)


def test_whole_tensor_is_one_row():
    R = np.array([[10.0, -2.0], [0.001, 0.0005]])
    T = np.array([[10.5, -2.0], [0.002, 0.0005]])
    # one row: max |T - R| = 0.5 over max(10, 0.01) = 0.05
    assert rel_err(T, R, whole=True) == pytest.approx(0.05, rel=1e-12)


def test_one_dimensional_tensor_is_one_row():
    R = np.array([10.0, 0.001])
    T = np.array([10.0, 0.003])
    # one row: 0.002 / 10 = 2e-4 (not 0.002 / 0.01 as it would be with one row per element)
    assert rel_err(T, R) == pytest.approx(2e-4, rel=1e-12)


def test_rows_are_the_first_axis_of_a_three_dimensional_tensor():
    R = np.zeros((2, 2, 3))
    R[0] = 5.0
    R[1, 0, 0] = 0.5
    T = R.copy()
    T[1, 1, 2] = 0.05
    # row 1 (R[1] flattened): max |diff| = 0.05 over max(0.5, 5e-3) = 0.1; row 0 exact
    assert rel_err(T, R) == pytest.approx(0.1, rel=1e-12)
    # rows cut along the last axis instead would give row [1, 1, :] = 0.05 / 5e-3 = 10
    assert rel_err(T.reshape(4, 3), R.reshape(4, 3)) == pytest.approx(10.0, rel=1e-12)


def test_all_zero_reference_reports_the_absolute_error():
    R = np.zeros((2, 3))
    T = np.zeros((2, 3))
    T[1, 2] = -3e-7
    assert rel_err(T, R) == pytest.approx(3e-7, rel=1e-12)
    assert rel_err(np.zeros(4), np.zeros(4)) == 0.0


def test_exact_match_is_zero():
    rng = np.random.default_rng(0)
    R = rng.normal(size=(5, 7))
    assert rel_err(R.copy(), R) == 0.0
    assert rel_err(R.astype(np.float32), R) <= 2.0 ** -24 * 1.01


def test_nan_never_passes():
    R = np.ones((3, 2))
    T = R.copy()
    T[2, 1] = np.nan
    e = rel_err(T, R)
    assert math.isnan(e) and not (e <= 1e-5)
    e = rel_err(T, R, whole=True)
    assert math.isnan(e) and not (e <= 1e-5)


def test_shape_mismatch_raises():
    with pytest.raises(ValueError):
        rel_err(np.zeros((2, 3)), np.zeros((3, 2)))
    with pytest.raises(ValueError):
        rel_err(np.zeros(6), np.zeros((2, 3)))


def test_empty_tensor_is_zero():
    assert rel_err(np.zeros((0, 4)), np.zeros((0, 4))) == 0.0
