"""The max-abs bar (CPU only): plain |stored - ref| below |ref| = 4, and
above it the distance from the oracle's value to the rounding interval of
the stored bf16 number."""
import numpy as np

from tolerance import GRID_LIMIT, MAX_ABS, bar_errors, bf16_interval_distance, errors


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


def test_plain_bar_below_four():
    """Sweep seed 141's row: the oracle is -2.4633527 and the kernel stored
    -2.453125 (0.0102 away).  Below 4 the bar is the plain difference, so
    that element fails, although the oracle lies only 0.0024 from the stored
    number's rounding interval."""
    g = np.array([np.float32(-2.453125), np.float32(1.0)])
    ref = np.array([-2.4633527, 1.0])
    mx, mean = errors(g, ref)
    assert abs(mx - (2.4633527 - 2.453125)) < 1e-12 and mx > MAX_ABS
    assert abs(mean - (2.4633527 - 2.453125) / 2) < 1e-12


def test_correct_rounding_always_meets_the_plain_bar_below_four():
    rng = np.random.default_rng(1)
    ref = rng.uniform(-GRID_LIMIT, GRID_LIMIT, 200000)
    ref = ref[np.abs(ref) < GRID_LIMIT]
    assert bar_errors(_bf16(ref), ref).max() <= 2.0 ** -8 * 2 + 1e-15


def test_interval_reading_from_four_up():
    # on [4, 8) the spacing is 2^-5: a correctly rounded value can sit
    # 2^-6 = 0.0156 from the oracle, beyond a plain 1e-2
    ref = np.array([4.0 + 2 ** -6 - 1e-9])
    g = _bf16(ref)
    assert abs(float(g[0]) - ref[0]) > MAX_ABS
    assert bar_errors(g, ref)[0] == 0.0
    # 1e-3 past the rounding interval counts as 1e-3
    ref2 = np.array([-(5.0 + 2 ** -6 + 1e-3)])
    assert abs(bar_errors(np.array([np.float32(-5.0)]), ref2)[0] - 1e-3) < 1e-12


def test_rejects_values_off_the_bf16_grid():
    import pytest
    with pytest.raises(ValueError):
        bf16_interval_distance(np.array([np.float32(1.0 + 2 ** -12)]), np.array([1.0]))
