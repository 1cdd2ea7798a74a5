"""The computation-aware block evictor (Sec. 4.2, Alg. 1) against its oracle
(CPU only; the evictor is host code).

The oracle evaluates the policy from its definition at every eviction: it
scans all blocks for the least f_B(t) * dT_B (Eq. 3, Eq. 9, Alg. 1's lambda,
Eq. 10).  The library keeps two ordered trees of time-invariant keys instead.
On the same operation sequence both must evict the same blocks, in the same
order.  The sequences come from:

* multi-turn serving simulations on a block cache, with and without online
  lifespan updates;
* random operation streams.

The library's own O(n) mode must agree too.  The order-preserving rule
(Eq. 8) is checked as a property:

* within one exponential segment, eviction order does not depend on time;
* the piecewise function can flip two blocks' order over time, which is why
  Alg. 1 keeps two trees.
"""
import math

import numpy as np
import pytest

import oracle
import workloads
import paper_2606_02964_amd as msa

PARAMS = dict(alpha=276.0, beta=276.0 / 40, tau0=276.0 * (1 - 1 / 40))  # turning point 276 s


def _replays_agree(trace, params=PARAMS, lam=1.0):
    a, b, t0 = params["alpha"], params["beta"], params["tau0"]
    ref = oracle.evictor_replay(a, b, t0, lam, trace.op, trace.ids, trace.t, trace.cost)
    ev = trace.op == 2
    assert ev.sum() > 0, "trace never evicted"
    assert np.array_equal(ref[ev], trace.evicted[ev]), \
        f"first mismatch at eviction {int(np.argmax(ref[ev] != trace.evicted[ev]))}"
    for linear in (False, True):
        again = msa.Evictor(a, b, t0, lam, linear=linear).replay(trace.op, trace.ids, trace.t,
                                                                  trace.cost)
        assert np.array_equal(again[ev], trace.evicted[ev]), f"linear={linear}"


SMALL = dict(capacity=512, conversations=40, turns=5, first_prompt=(256, 2048),
             turn_tokens=(64, 512), max_tokens=6000, think_time=30.0, span=600.0)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_serving_trace_matches_oracle(seed):
    ev = msa.Evictor(**PARAMS)
    trace = workloads.simulate_block_cache(ev, seed, **SMALL)
    assert trace.hits > 0 and trace.misses > 0
    _replays_agree(trace)


def test_serving_trace_with_lifespan_updates_matches_oracle():
    ev = msa.Evictor(**PARAMS)
    trace = workloads.simulate_block_cache(ev, 9, lifespan_every=7, **SMALL)
    assert (trace.op == 3).sum() > 3
    _replays_agree(trace)


def test_linear_mode_drives_the_same_simulation():
    a = workloads.simulate_block_cache(msa.Evictor(**PARAMS), 4, **SMALL)
    b = workloads.simulate_block_cache(msa.Evictor(**PARAMS, linear=True), 4, **SMALL)
    for x, y in ((a.op, b.op), (a.ids, b.ids), (a.t, b.t), (a.evicted, b.evicted)):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("seed", [5, 6])
def test_random_operations_match_oracle(seed):
    rng = np.random.default_rng(seed)
    ev = msa.Evictor(alpha=3.0, beta=0.4, tau0=2.5, lam=1.7)
    present, next_id, clock = [], 0, 0.0
    op, ids, t, cost, out = [], [], [], [], []
    for _ in range(4000):
        clock += float(rng.exponential(0.05))
        r = rng.random()
        if r < 0.5 or not present:
            c = float(rng.uniform(0.1, 10.0))
            ev.add(next_id, clock, c)
            op.append(0), ids.append(next_id), t.append(clock), cost.append(c), out.append(-1)
            present.append(next_id)
            next_id += 1
        elif r < 0.7:
            k = int(rng.integers(len(present)))
            b = present.pop(k)
            ev.remove(b)
            op.append(1), ids.append(b), t.append(0.0), cost.append(0.0), out.append(-1)
        elif r < 0.97:
            v = ev.evict(clock)
            present.remove(v)
            op.append(2), ids.append(-1), t.append(clock), cost.append(0.0), out.append(v)
        else:
            tau = float(rng.uniform(0.0, 5.0))
            ev.set_lifespan(tau)
            op.append(3), ids.append(-1), t.append(tau), cost.append(0.0), out.append(-1)
    trace = workloads.EvictorTrace(np.array(op, np.int32), np.array(ids, np.int64),
                                   np.array(t), np.array(cost), np.array(out, np.int64),
                                   0, 0, 0, 0)
    _replays_agree(trace, dict(alpha=3.0, beta=0.4, tau0=2.5), lam=1.7)


def _order(ev_factory, blocks, t_now):
    ev = ev_factory()
    for (i, tl, c) in blocks:
        ev.add(i, tl, c)
    return [ev.evict(t_now) for _ in blocks]


@pytest.mark.parametrize("lam,times", [(1e200, (150.0, 400.0, 1000.0)),
                                       (1e-200, (150.0, 1e3, 1e5))])
def test_single_segment_order_does_not_depend_on_time(lam, times):
    """lam = 1e200 leaves only exp(-tau/alpha) in force for tau < ~1000 (the
    second segment decays faster and binds beyond); lam = 1e-200 leaves only
    the second segment at every tau >= 0.  Each is exponential, so eviction
    order is time-invariant (Eq. 8)."""
    rng = np.random.default_rng(0)
    blocks = [(i, float(rng.uniform(0, 100)), float(rng.uniform(0.5, 5))) for i in range(300)]
    make = lambda: msa.Evictor(alpha=20.0, beta=2.0, tau0=15.0, lam=lam)
    first = _order(make, blocks, 100.0)
    for t_now in times:
        assert _order(make, blocks, t_now) == first


def test_piecewise_function_flips_order_over_time():
    """A older but costlier than B: B goes first while both are young, A goes
    first once A has aged past the turning point (Eq. 9 is not order
    preserving, hence two trees)."""
    make = lambda: msa.Evictor(alpha=10.0, beta=1.0, tau0=9.0)
    blocks = [(0, 0.0, 3.0), (1, 5.0, 1.0)]
    assert _order(make, blocks, 6.0)[0] == 1
    assert _order(make, blocks, 20.0)[0] == 0
    for t_now in (6.0, 20.0):
        ref = oracle.evictor_replay(10.0, 1.0, 9.0, 1.0, [0, 0, 2], [0, 1, -1], [0.0, 5.0, t_now],
                                    [3.0, 1.0, 0.0])
        assert ref[2] == _order(make, blocks, t_now)[0]


def test_log_weight_and_lifespan():
    ev = msa.Evictor(alpha=10.0, beta=2.0, tau0=6.0)
    ev.add(7, 1.0, 2.5)
    t = 4.0  # tau = 3: first segment -0.3, second 1.5
    assert ev.log_weight(7, t) == pytest.approx(-0.3 + math.log(2.5), rel=1e-12)
    t = 31.0  # tau = 30: first -3, second -12
    assert ev.log_weight(7, t) == pytest.approx(-12.0 + math.log(2.5), rel=1e-12)
    # Eq. 10 puts the turning point at the given lifespan: both segments meet there
    lam = ev.set_lifespan(8.0)
    assert lam == pytest.approx(math.exp((8.0 - 6.0) / 2.0 - 8.0 / 10.0), rel=1e-12)
    seg1 = -8.0 / 10.0
    assert ev.log_weight(7, 9.0) == pytest.approx(seg1 + math.log(2.5), rel=1e-12)
    ev.set_lambda(1.0)
    assert ev.log_weight(7, 4.0) == pytest.approx(-0.3 + math.log(2.5), rel=1e-12)


def test_errors():
    with pytest.raises(msa.MsaError):
        msa.Evictor(alpha=0.0, beta=1.0, tau0=0.0)
    with pytest.raises(msa.MsaError):
        msa.Evictor(alpha=1.0, beta=-1.0, tau0=0.0)
    with pytest.raises(msa.MsaError):
        msa.Evictor(alpha=1.0, beta=1.0, tau0=float("nan"))
    ev = msa.Evictor(alpha=1.0, beta=1.0, tau0=0.0)
    with pytest.raises(msa.MsaError) as e:
        ev.evict(0.0)
    assert "no evictable block" in msa.msa_last_error()
    ev.add(1, 0.0, 1.0)
    with pytest.raises(msa.MsaError):
        ev.add(1, 0.0, 1.0)
    with pytest.raises(msa.MsaError):
        ev.add(2, 0.0, 0.0)
    with pytest.raises(msa.MsaError):
        ev.add(2, float("inf"), 1.0)
    with pytest.raises(msa.MsaError):
        ev.remove(3)
    with pytest.raises(msa.MsaError):
        ev.set_lambda(0.0)
    with pytest.raises(msa.MsaError):
        ev.set_lifespan(-1.0)
    assert len(ev) == 1
    with pytest.raises(msa.MsaError) as e:
        ev.replay([0, 2, 2, 2], [5, -1, -1, -1], [0.0, 1.0, 1.0, 1.0], [1.0, 0.0, 0.0, 0.0])
    assert "op 3" in str(e.value)  # block 1 and block 5 go first, then nothing is left
    with pytest.raises(ValueError):
        oracle.evictor_replay(1.0, 1.0, 0.0, 1.0, [1], [4], [0.0], [0.0])


def test_block_cost_is_position_linear():
    c = workloads.block_cost(np.arange(6))
    d = np.diff(c)
    assert np.allclose(d, d[0]) and d[0] > 0 and c[0] > 0
    # per-token part plus one pair per visible key, counted one by one
    brute = 16 * 1.0 + sum(p + 1 for p in range(48, 64)) / 4096
    assert workloads.block_cost(3) == pytest.approx(brute, rel=1e-15)
