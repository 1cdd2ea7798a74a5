"""The bf16-aware max-abs bar (CPU only): the distance from the oracle's
value to the rounding interval of the stored bf16 number."""
import numpy as np

from tolerance import bf16_interval_distance, errors


def _bf16(x):
    """Round float64 values (in the normal float32 range) to the nearest bf16
    number, ties to even, in one step from the float64 bits, as float32."""
    b = np.asarray(x, dtype=np.float64).view(np.uint64)
    low = np.uint64(45)  # float64 keeps 52 fraction bits, bf16 keeps 7
    b = (b + np.uint64((1 << 44) - 1) + ((b >> low) & np.uint64(1))) & ~np.uint64((1 << 45) - 1)
    return b.view(np.float64).astype(np.float32)


def test_values_that_round_to_the_stored_number_are_at_distance_zero():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal(100000) * rng.choice([1e-3, 1.0, 3.0, 100.0], 100000)
    assert np.all(bf16_interval_distance(_bf16(ref), ref) == 0.0)


def test_distance_on_the_binade_of_two():
    # on [2, 4) the bf16 spacing is 2^-6; 2.453125 covers [2.4453125, 2.4609375]
    g = np.float32(-2.453125)
    d = bf16_interval_distance(np.array([g]), np.array([-2.4633527]))[0]
    assert abs(d - (2.4633527 - 2.4609375)) < 1e-12
    d = bf16_interval_distance(np.array([g]), np.array([-2.44]))[0]
    assert abs(d - (2.4453125 - 2.44)) < 1e-12


def test_power_of_two_has_a_narrower_gap_below():
    # below 1.0 the spacing is 2^-8, above it 2^-7
    one = np.array([np.float32(1.0)] * 2)
    d = bf16_interval_distance(one, np.array([1.0 - 2 ** -9 - 1e-3, 1.0 + 2 ** -8 + 1e-3]))
    assert np.allclose(d, [1e-3, 1e-3], atol=1e-12, rtol=0)


def test_opposite_sign_and_zero():
    d = bf16_interval_distance(np.array([np.float32(0.5), np.float32(0.0)]), np.array([-0.5, 0.25]))
    assert abs(d[0] - (1.0 - 2 ** -10)) < 1e-12   # gap below 0.5 is 2^-9, half of it 2^-10
    assert abs(d[1] - 0.25) < 1e-30 + 1e-12


def test_errors_reports_interval_distance_and_plain_mean():
    g = np.array([np.float32(-2.453125), np.float32(1.0)])
    ref = np.array([-2.4633527, 1.0])
    mx, mean = errors(g, ref)
    assert abs(mx - (2.4633527 - 2.4609375)) < 1e-12
    assert abs(mean - (2.4633527 - 2.453125) / 2) < 1e-12


def test_rejects_values_off_the_bf16_grid():
    import pytest
    with pytest.raises(ValueError):
        bf16_interval_distance(np.array([np.float32(1.0 + 2 ** -12)]), np.array([1.0]))
