"""Pins of the evictor oracle (CPU only), against facts the paper and plain
arithmetic fix.

* LRU: with one cost for every block, the policy is LRU (Sec. 4.2).  Each
  segment of f decreases with age, so blocks leave oldest release first.
* Equal release times: the age term is common, so blocks leave in
  increasing cost.
* Exact ties (same release time and cost) go to the smaller id.
* Hand-computed example 1 (Eq. 9 is not order preserving).  alpha = 10,
  beta = 1, tau0 = 9.  Block A is released at 0 with cost 3; block B at 5
  with cost 1.
  - At t = 6: ln wA = min(-0.6, 3) + ln 3 = 0.499 and ln wB = min(-0.1, 8) =
    -0.1, so B goes.
  - At t = 20: ln wA = min(-2, -11) + ln 3 = -9.90 and ln wB = min(-1.5, -6) =
    -6, so A goes.
* Hand-computed example 2 (Alg. 1's lambda and Eq. 10).  Same alpha, beta,
  tau0.  A is released at 0 with cost e^2; B at 4 with cost 1; eviction at
  t = 6.
  - With lambda = 1: ln wA = min(-0.6, 3) + 2 = 1.4 and ln wB = -0.2, so B
    goes.
  - After a lifespan update to 4, lambda = exp((4 - 9)/1 - 4/10) = e^-5.4.
    Then ln wA = min(-0.6, -5.4 + 3) + 2 = -0.4 and ln wB = min(-0.2, -5.4 +
    7) = -0.2, so A goes.

Plausible mistakes planted in a copy of the oracle source each fail one of
these pins.
"""
import math
import os
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(oracle.__file__)
SRC = os.path.join(HERE, "evictor_oracle.c")
MAIN = os.path.join(HERE, "msa_oracle.c")


def _evict_all(lib, alpha, beta, tau0, blocks, t_now, lam=1.0, lifespan=None):
    op, ids, t, cost = [], [], [], []
    for (i, tl, c) in blocks:
        op.append(0), ids.append(i), t.append(tl), cost.append(c)
    if lifespan is not None:
        op.append(3), ids.append(-1), t.append(lifespan), cost.append(0.0)
    for _ in blocks:
        op.append(2), ids.append(-1), t.append(t_now), cost.append(0.0)
    out = oracle.evictor_replay(alpha, beta, tau0, lam, op, ids, t, cost, lib=lib)
    return [int(x) for x, o in zip(out, op) if o == 2]


def _pins(lib):
    rng = np.random.default_rng(0)
    res = {}
    # LRU under uniform cost, for several parameter sets
    ok = True
    for (a, b, t0) in [(10.0, 1.0, 9.0), (276.0, 6.9, 269.1), (5.0, 5.0, 0.0)]:
        tl = rng.permutation(200).astype(float)
        blocks = [(i, float(tl[i]), 2.0) for i in range(200)]
        order = _evict_all(lib, a, b, t0, blocks, 500.0)
        ok &= order == [int(i) for i in np.argsort(tl, kind="stable")]
    res["lru"] = ok
    # cost order at equal release time
    cs = rng.permutation(100) + 1.0
    order = _evict_all(lib, 10.0, 1.0, 9.0, [(i, 3.0, float(cs[i])) for i in range(100)], 50.0)
    res["cost"] = order == [int(i) for i in np.argsort(cs, kind="stable")]
    # exact ties: smaller id first
    order = _evict_all(lib, 10.0, 1.0, 9.0, [(i, 1.0, 1.0) for i in (9, 3, 7, 1)], 4.0)
    res["ties"] = order == [1, 3, 7, 9]
    # example 1
    two = [(0, 0.0, 3.0), (1, 5.0, 1.0)]
    res["example1"] = (_evict_all(lib, 10.0, 1.0, 9.0, two, 6.0)[0] == 1 and
                       _evict_all(lib, 10.0, 1.0, 9.0, two, 20.0)[0] == 0)
    # example 2
    two = [(0, 0.0, math.exp(2.0)), (1, 4.0, 1.0)]
    res["example2"] = (_evict_all(lib, 10.0, 1.0, 9.0, two, 6.0)[0] == 1 and
                       _evict_all(lib, 10.0, 1.0, 9.0, two, 6.0, lifespan=4.0)[0] == 0 and
                       _evict_all(lib, 10.0, 1.0, 9.0, two, 6.0, lam=math.exp(-5.4))[0] == 0)
    return res


def test_oracle_pins():
    res = _pins(None)
    assert all(res.values()), res


def test_oracle_rejects_impossible_operations():
    with pytest.raises(ValueError):
        oracle.evictor_replay(1.0, 1.0, 0.0, 1.0, [0, 0], [4, 4], [0.0, 0.0], [1.0, 1.0])
    with pytest.raises(ValueError):
        oracle.evictor_replay(1.0, 1.0, 0.0, 1.0, [2], [-1], [0.0], [0.0])
    with pytest.raises(ValueError):
        oracle.evictor_replay(1.0, 1.0, 0.0, 1.0, [0], [4], [0.0], [0.0])


MUTANTS = {
    "max_instead_of_min": ("(seg1 < seg2 ? seg1 : seg2)", "(seg1 > seg2 ? seg1 : seg2)"),
    "cost_ignored": ("(seg1 < seg2 ? seg1 : seg2) + log(b[k].cost)", "(seg1 < seg2 ? seg1 : seg2)"),
    "lambda_on_first_segment": ("const double seg1 = -tau / alpha;\n        const double seg2 = log_lambda - (tau - tau0) / beta;",
                                "const double seg1 = log_lambda - tau / alpha;\n        const double seg2 = -(tau - tau0) / beta;"),
    "ties_to_larger_id": ("b[k].id < b[best].id", "b[k].id > b[best].id"),
    "age_sign_flipped": ("const double tau = t[i] - b[k].t_last;", "const double tau = b[k].t_last - t[i];"),
    "lifespan_rule_sign": ("log_lambda = (t[i] - tau0) / beta - t[i] / alpha;",
                           "log_lambda = (t[i] - tau0) / beta + t[i] / alpha;"),
}


def _build(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-pthread", MAIN, str(c), "-o", str(so), "-lm"])
    return oracle.load_library(str(so))


def test_unmutated_copy_passes(tmp_path):
    assert all(_pins(_build(tmp_path, "same", open(SRC).read())).values())


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    res = _pins(_build(tmp_path, name, src.replace(old, new)))
    assert not all(res.values()), res
