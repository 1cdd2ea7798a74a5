"""Recomputation cost model of a two-segment cached request (Sec. 4.3).

A request's context is laid out as
``[l1 cached][q1 computed][l2 cached][q2 computed]``: ``l1`` and ``l2``
tokens are served from the cache, ``q1`` and ``q2`` are computed.

Eq. 4 (exact form).  The token-parallel parts of the model cost a constant
per token.  Attention adds, per computed segment, its rows times the keys
they see:

    T = k1 l1 + k2 q1 + k3 l2 + k4 q2
        + k5 q1 (l1 + q1) + k6 q2 (l1 + q1 + l2 + q2) + beta

Eq. 5.  Evicting the first block of the second cached run moves one token
from l2 to q1:

    dT = k5 (l1 + 2 q1) + (k2 - k3 + k5)

Eq. 6 (approximate form).  Eq. 5 depends on q1, which changes as blocks are
evicted.  The paper therefore replaces ``q1 (l1 + q1)`` with
``(l1 + q1)^2``.

Eq. 7.  The eviction cost then depends only on the block's fixed position
``l1 + q1`` (the tokens before it):

    dT = 2 k5 (l1 + q1) + (k2 - k3 + k5)

A third form, ``pairs``, counts the causal triangle exactly.  It is not in
the paper; it is kept here for comparison.  Each computed row at position p
sees p + 1 keys:

    T = k1 l1 + k2 q1 + k3 l2 + k4 q2
        + k5 (q1 l1 + q1 (q1 + 1) / 2)
        + k6 (q2 (l1 + q1 + l2) + q2 (q2 + 1) / 2) + beta

Its one-token eviction cost is

    dT = k5 (l1 + q1 + 1) + (k2 - k3)

This also depends only on the block's position, which is the form of Eq. 7.

Coefficients are fitted by ordinary least squares on measured
``(l1, q1, l2, q2) -> T`` samples.  The unit moved in Eq. 5 and Eq. 7 is one
token, as in the paper.  For a block of ``bs`` tokens,
:func:`delta_t_block` takes the exact difference of the fitted model.
"""
from __future__ import annotations

from typing import Dict, Sequence, Tuple

import numpy as np

MODELS = ("eq4", "eq6", "pairs")
COEFFS = ("k1", "k2", "k3", "k4", "k5", "k6", "beta")


def features(model: str, l1, q1, l2, q2) -> np.ndarray:
    """Design matrix [n, 7] of Eq. 4, Eq. 6 or the causal-pairs form: columns k1..k6, beta."""
    l1, q1, l2, q2 = (np.asarray(x, dtype=np.float64) for x in (l1, q1, l2, q2))
    if model == "eq4":
        quad1 = q1 * (l1 + q1)
        quad2 = q2 * (l1 + q1 + l2 + q2)
    elif model == "eq6":
        quad1 = (l1 + q1) ** 2
        quad2 = q2 * (l1 + q1 + l2 + q2)
    elif model == "pairs":
        quad1 = q1 * l1 + q1 * (q1 + 1) / 2
        quad2 = q2 * (l1 + q1 + l2) + q2 * (q2 + 1) / 2
    else:
        raise ValueError(f"unknown model {model!r}")
    ones = np.ones_like(l1)
    return np.stack([l1, q1, l2, q2, quad1, quad2, ones], axis=-1)


def predict(model: str, k: Dict[str, float], l1, q1, l2, q2) -> np.ndarray:
    vec = np.array([k[c] for c in COEFFS], dtype=np.float64)
    return features(model, l1, q1, l2, q2) @ vec


def fit(model: str, samples: Sequence[Tuple[float, float, float, float, float]]):
    """Least-squares fit of (l1, q1, l2, q2, T) samples.

    Returns (coefficients dict, R^2).  Columns are scaled to unit norm before
    solving, because the quadratic features are ~1e8 times the constant."""
    a = np.asarray(samples, dtype=np.float64)
    X = features(model, a[:, 0], a[:, 1], a[:, 2], a[:, 3])
    y = a[:, 4]
    scale = np.linalg.norm(X, axis=0)
    scale[scale == 0] = 1.0
    sol, *_ = np.linalg.lstsq(X / scale, y, rcond=None)
    coef = sol / scale
    resid = y - X @ coef
    ss_tot = float(((y - y.mean()) ** 2).sum())
    r2 = 1.0 - float((resid ** 2).sum()) / ss_tot if ss_tot > 0 else 1.0
    return dict(zip(COEFFS, map(float, coef))), r2


def delta_t_eq5(k: Dict[str, float], l1, q1) -> np.ndarray:
    """Eq. 5: one token moved from l2 to q1, under Eq. 4."""
    l1, q1 = np.asarray(l1, np.float64), np.asarray(q1, np.float64)
    return k["k5"] * (l1 + 2 * q1) + (k["k2"] - k["k3"] + k["k5"])


def delta_t_eq7(k: Dict[str, float], l1, q1) -> np.ndarray:
    """Eq. 7: one token moved from l2 to q1, under Eq. 6 (position only)."""
    l1, q1 = np.asarray(l1, np.float64), np.asarray(q1, np.float64)
    return 2 * k["k5"] * (l1 + q1) + (k["k2"] - k["k3"] + k["k5"])


def delta_t_pairs(k: Dict[str, float], l1, q1) -> np.ndarray:
    """One token moved from l2 to q1, under the causal-pairs form."""
    l1, q1 = np.asarray(l1, np.float64), np.asarray(q1, np.float64)
    return k["k5"] * (l1 + q1 + 1) + (k["k2"] - k["k3"])


def delta_t_block(model: str, k: Dict[str, float], l1, q1, l2, q2, bs: int = 16) -> np.ndarray:
    """Fitted model's cost of evicting the first ``bs``-token block of the
    second cached run: T(l1, q1 + bs, l2 - bs, q2) - T(l1, q1, l2, q2)."""
    l1, q1, l2, q2 = (np.asarray(x, np.float64) for x in (l1, q1, l2, q2))
    return predict(model, k, l1, q1 + bs, l2 - bs, q2) - predict(model, k, l1, q1, l2, q2)
