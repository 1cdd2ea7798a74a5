"""The bar of the GPU path against the oracle (numpy only, no GPU).

O is stored in bf16 and compared after upcasting, element by element:

- Where the oracle's value lies below 4 in magnitude, the bar is the plain
  |stored - ref| <= 1e-2.  Half a bf16 spacing is at most 2^-8 * 2 = 0.0078
  there, so a correctly rounded exact result always meets it.
- From 4 up, half a bf16 spacing is 2^-8 * 4 = 0.0156 or more, and even a
  correctly rounded exact result can miss a plain 1e-2.  There the bar is on
  the value before its final rounding: some real within 1e-2 of the oracle
  must round (to nearest) to the stored bf16 number, i.e. the distance from
  the oracle's value to the stored number's rounding interval is <= 1e-2.

The mean-abs bar of 1e-3 is taken on the stored values as they are.
"""
from __future__ import annotations

import numpy as np

# the stated bar for O
MAX_ABS = 1e-2
MEAN_ABS = 1e-3
# |ref| from which half a bf16 spacing exceeds MAX_ABS (the binade [4, 8))
GRID_LIMIT = 4.0
# lse (natural log): the row sum adds the fp32 weights, one sum of at most
# 32 per 64-key step (16 per 32-key half-step) and one running sum over the
# steps, so ln(l) carries a relative rounding of at most (32 + steps) * 2^-24:
# 1.3e-4 at 2048 steps (131072 keys, the longest row tested).  fp32 scores,
# exp2/log2 and the split merge add a few 1e-6 at these score magnitudes.
LSE_ABS = 2.5e-4


def bf16_interval_distance(stored: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Distance from each ``ref`` value to the set of reals that round to
    nearest to the bf16 number ``stored`` (given as float32 values that are
    bf16 numbers).  Zero when ``ref`` itself rounds to ``stored``."""
    g = np.asarray(stored, dtype=np.float32)
    bits = g.view(np.uint32).astype(np.int64)
    if np.any(bits & 0xFFFF):
        raise ValueError("stored values are not bf16 numbers")
    mag = bits & 0x7FFFFFFF
    absg = np.abs(g.astype(np.float64))
    up = (mag + 0x10000).astype(np.uint32).view(np.float32).astype(np.float64)
    half_away = (up - absg) / 2
    dn = np.where(mag > 0, mag - 0x10000, 0).astype(np.uint32).view(np.float32).astype(np.float64)
    half_toward = np.where(mag > 0, (absg - dn) / 2, half_away)
    diff = np.asarray(ref, dtype=np.float64) - g.astype(np.float64)
    # ref lies farther from zero than g: the gap above |g| applies
    away = (diff != 0) & (np.sign(diff) == np.where(g < 0, -1.0, 1.0)) & (mag > 0)
    slack = np.where(away, half_away, half_toward)
    return np.maximum(np.abs(diff) - slack, 0.0)


def bar_errors(stored: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per element, the figure the max-abs bar bounds: the plain difference
    where |ref| < GRID_LIMIT, the distance to the rounding interval above."""
    stored = np.asarray(stored, dtype=np.float32)
    ref = np.asarray(ref, dtype=np.float64)
    plain = np.abs(stored.astype(np.float64) - ref)
    big = np.abs(ref) >= GRID_LIMIT
    if not big.any():
        return plain
    out = plain.copy()
    out[big] = bf16_interval_distance(stored[big], ref[big])
    return out


def errors(stored: np.ndarray, ref: np.ndarray):
    """(largest bar figure over the elements, see bar_errors; mean absolute
    difference of the stored values)."""
    if stored.size == 0:
        return 0.0, 0.0
    return (float(bar_errors(stored, ref).max()),
            float(np.abs(np.asarray(stored, dtype=np.float64) - ref).mean()))


def raw_max_abs(stored: np.ndarray, ref: np.ndarray) -> float:
    """Largest plain |stored - ref| over every element, reported beside the bar."""
    return float(np.abs(stored.astype(np.float64) - ref).max()) if stored.size else 0.0


# Peaky-logit stress inputs (scores spread over many log2 units, so that a
# few keys carry a row's weight).  There the plain bar is out of reach of a
# path that, like this one, enters the softmax weights into the PV product as
# bf16 numbers: each weight moves by up to 2^-8 of itself (8 significant
# bits, round to nearest), and with the row sum over the unrounded weights
# the output before its own rounding lies within 2^-8 * sum_j p_j |v_j| of the
# exact value (p_j: the exact normalised weights).  That sum is attention
# over |V| with the same weights, which the oracle computes when handed |V|.
# The bound adds the stored number's own rounding and a slack for the fp32
# scores, exp2 and sums.
WEIGHT_ROUNDING = 2.0 ** -8
WEIGHT_BOUND_SLACK = 1e-4


def half_spacing_bf16(x: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 numbers at magnitude |x| (2^(e - 8) on the
    binade [2^e, 2^(e+1)))."""
    a = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 8)


def weight_rounding_bound(ref: np.ndarray, ref_abs_v: np.ndarray) -> np.ndarray:
    """Per element bound on |stored - ref| for bf16 weights in the PV
    product: ``ref`` the exact output, ``ref_abs_v`` the exact attention
    over |V| with the same weights."""
    pre = WEIGHT_ROUNDING * np.asarray(ref_abs_v, dtype=np.float64) + WEIGHT_BOUND_SLACK
    return pre + half_spacing_bf16(np.abs(np.asarray(ref, dtype=np.float64)) + pre)
