"""The two-segment cost model of Sec. 4.3 (CPU only).

* Eq. 5 and Eq. 7 are the paper's closed forms for moving one token from l2
  to q1.  Each must equal the finite difference of the model it comes from
  (Eq. 4 and Eq. 6), for arbitrary coefficients and layouts.
* The least-squares fit recovers known coefficients exactly from noise-free
  samples, with R^2 = 1.
* Brute-force attention work (visible query-key pairs counted one by one)
  is fitted by Eq. 4 with R^2 close to 1.  It is not fitted exactly: Eq. 4
  weights q1^2 like q1*l1, while the causal triangle counts q1^2 / 2.  The
  causal-pairs form fits it exactly.
"""
import numpy as np
import pytest

from paper_2606_02964_amd import cost_model as cm


def _layouts(rng, n):
    l1 = rng.integers(0, 4000, n)
    q1 = rng.integers(0, 4000, n)
    l2 = rng.integers(1, 4000, n)
    q2 = rng.integers(1, 1000, n)
    return l1, q1, l2, q2


def _coeffs(rng):
    return dict(zip(cm.COEFFS, rng.uniform(-2, 2, 7) * np.array([1, 1, 1, 1, 1e-3, 1e-3, 10])))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_eq5_is_the_finite_difference_of_eq4(seed):
    rng = np.random.default_rng(seed)
    k = _coeffs(rng)
    l1, q1, l2, q2 = _layouts(rng, 200)
    fd = cm.predict("eq4", k, l1, q1 + 1, l2 - 1, q2) - cm.predict("eq4", k, l1, q1, l2, q2)
    np.testing.assert_allclose(cm.delta_t_eq5(k, l1, q1), fd, rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(cm.delta_t_block("eq4", k, l1, q1, l2, q2, bs=1), fd, rtol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_eq7_is_the_finite_difference_of_eq6(seed):
    rng = np.random.default_rng(seed)
    k = _coeffs(rng)
    l1, q1, l2, q2 = _layouts(rng, 200)
    fd = cm.predict("eq6", k, l1, q1 + 1, l2 - 1, q2) - cm.predict("eq6", k, l1, q1, l2, q2)
    np.testing.assert_allclose(cm.delta_t_eq7(k, l1, q1), fd, rtol=1e-9, atol=1e-9)
    # Eq. 7 depends on the block's position l1 + q1 only
    np.testing.assert_allclose(cm.delta_t_eq7(k, l1 + 5, q1 - 5), cm.delta_t_eq7(k, l1, q1))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_pairs_closed_form_is_its_finite_difference(seed):
    rng = np.random.default_rng(seed)
    k = _coeffs(rng)
    l1, q1, l2, q2 = _layouts(rng, 200)
    fd = cm.predict("pairs", k, l1, q1 + 1, l2 - 1, q2) - cm.predict("pairs", k, l1, q1, l2, q2)
    np.testing.assert_allclose(cm.delta_t_pairs(k, l1, q1), fd, rtol=1e-9, atol=1e-9)


def test_pairs_features_count_the_causal_triangle():
    rng = np.random.default_rng(11)
    for _ in range(40):
        l1, q1, l2, q2 = (int(x) for x in rng.integers(0, 300, 4))
        f = cm.features("pairs", [l1], [q1], [l2], [q2])[0]
        assert f[4] + f[5] == _pairs_brute(l1, q1, l2, q2)


@pytest.mark.parametrize("model", cm.MODELS)
def test_fit_recovers_exact_coefficients(model):
    rng = np.random.default_rng(7)
    k = _coeffs(rng)
    l1, q1, l2, q2 = _layouts(rng, 150)
    t = cm.predict(model, k, l1, q1, l2, q2)
    fk, r2 = cm.fit(model, np.stack([l1, q1, l2, q2, t], axis=1))
    assert r2 > 1 - 1e-12
    for c in cm.COEFFS:
        assert fk[c] == pytest.approx(k[c], rel=1e-6, abs=1e-9), c


def _pairs_brute(l1, q1, l2, q2):
    """Visible (query, key) pairs of the computed tokens, counted one by one."""
    n = 0
    for p in range(l1, l1 + q1):
        n += p + 1
    for p in range(l1 + q1 + l2, l1 + q1 + l2 + q2):
        n += p + 1
    return n


def test_eq4_fits_true_attention_work_closely_but_not_exactly():
    rng = np.random.default_rng(3)
    rows = []
    for _ in range(120):
        l1, q1, l2, q2 = (int(x) for x in rng.integers(0, 600, 4))
        q2 = max(q2, 1)
        rows.append((l1, q1, l2, q2, 3.0 * (q1 + q2) + 1e-3 * _pairs_brute(l1, q1, l2, q2) + 5.0))
    _, r2_eq4 = cm.fit("eq4", rows)
    _, r2_eq6 = cm.fit("eq6", rows)
    k, r2_pairs = cm.fit("pairs", rows)
    assert 0.99 < r2_eq4 < 1 - 1e-9
    assert r2_eq6 < 1 - 1e-9
    assert r2_pairs > 1 - 1e-12
    assert k["k5"] == pytest.approx(1e-3, rel=1e-6) and k["k6"] == pytest.approx(1e-3, rel=1e-6)


def test_fit_rejects_unknown_model():
    with pytest.raises(ValueError):
        cm.features("eq9", [1], [1], [1], [1])
