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


def test_half_spacing_of_bf16():
    from tolerance import half_spacing_bf16
    x = np.array([1.0, 1.99, 2.0, 3.0, 0.75, -4.5, 2.0 ** -20])
    want = np.array([2 ** -8, 2 ** -8, 2 ** -7, 2 ** -7, 2 ** -9, 2 ** -6, 2.0 ** -28])
    assert np.array_equal(half_spacing_bf16(x), want)
    # a correctly rounded value is within half a spacing
    rng = np.random.default_rng(3)
    r = rng.standard_normal(100000) * 3
    assert np.all(np.abs(_bf16(r).astype(np.float64) - r) <= half_spacing_bf16(r))


def _peaky_rows(rng, n, keys, d, qscale):
    """Exact outputs, attention over |V|, and outputs with bf16 weights in the
    numerator (fp32-exact row sums), rounded to bf16, for random peaky rows."""
    q = rng.standard_normal((n, d)) * qscale
    k = rng.standard_normal((n, keys, d))
    v = _bf16(rng.standard_normal((n, keys, d))).astype(np.float64)
    s = np.einsum("nd,nkd->nk", q, k) / np.sqrt(d)
    w = np.exp(s - s.max(axis=1, keepdims=True))
    p = w / w.sum(axis=1, keepdims=True)
    exact = np.einsum("nk,nkd->nd", p, v)
    absv = np.einsum("nk,nkd->nd", p, np.abs(v))
    wb = _bf16(w).astype(np.float64)
    stored = _bf16(np.einsum("nk,nkd->nd", wb, v) / w.sum(axis=1, keepdims=True))
    return exact, absv, stored


def test_weight_rounding_bound_holds_and_is_tight():
    """Rows whose weight sits on a few keys (Q scaled by 4 and 8): bf16
    weights with an exact row sum, then the output's own rounding, stay within
    the bound everywhere; the largest element uses most of it, the plain bar
    fails on some, and an error of twice the bound is caught."""
    from tolerance import weight_rounding_bound
    rng = np.random.default_rng(5)
    worst_use, plain_max = 0.0, 0.0
    for qscale in (4.0, 8.0):
        for keys in (2, 3, 8, 64):
            exact, absv, stored = _peaky_rows(rng, 2000, keys, 64, qscale)
            bound = weight_rounding_bound(exact, absv)
            err = np.abs(stored.astype(np.float64) - exact)
            assert np.all(err <= bound)
            worst_use = max(worst_use, float((err / bound).max()))
            plain_max = max(plain_max, float(err[np.abs(exact) < GRID_LIMIT].max()))
            bad = stored.astype(np.float64) + 2 * bound * np.sign(rng.standard_normal(bound.shape))
            assert np.all(np.abs(bad - exact) > bound)
    assert worst_use > 0.8
    assert plain_max > MAX_ABS
