"""Pins of the cost-model oracle (oracle/cost_ref.py) on hand-worked values,
and parity of the library's native cost model and routing with it."""
import ctypes

import numpy as np
import pytest

from oracle import cost_ref as R
from oracle.cost_ref import Coeffs, Instance, Traj

C = Coeffs(k1=1e-6, k2=1e-3, k3=1e-4, k4=1e-3, k5=1.0, budget=1e4)


def test_throughput_by_hand():
    c = Coeffs(1e-8, 1e-3, 1e-4, 1e-2, 2.0, 1e9)
    # 50 / (1e-8 * 1e6 + max(1e-3, 50 * 1e-4) + 1e-2) = 50 / 0.025
    assert R.throughput(c, Instance(0, 50, 0, 1e6)) == pytest.approx(2000.0, rel=1e-12)
    # memory-bound branch: n * k3 < k2
    assert R.throughput(c, Instance(0, 5, 0, 0.0)) == pytest.approx(5 / (1e-3 + 1e-2), rel=1e-12)
    assert R.throughput(c, Instance(0, 0, 0, 5e5)) == 0.0


def test_marginal_gain_is_zero_when_the_trajectory_would_wait():
    s = Instance(0, 10, 0, 9500.0)
    assert R.marginal_gain(C, s, 600.0) == 0.0          # 9500 + 600 > M
    assert R.marginal_gain(C, Instance(0, 10, 2, 0.0), 10.0) == 0.0   # waiting queue not empty
    assert R.after_routing(C, s, 600.0) == Instance(0, 10, 1, 9500.0)


def test_ideal_gain_is_the_gain_on_an_idle_instance():
    for length in (1.0, 100.0, 6000.0):
        assert R.ideal_gain(C, length) == R.marginal_gain(C, Instance(3, 0, 0, 0.0), length)
    # 1 / (1e-6 * 6000 + max(1e-3, 1e-4) + 1e-3) = 1 / 0.008
    assert R.ideal_gain(C, 6000.0) == pytest.approx(125.0, rel=1e-12)


INSTS = [Instance(1, 0, 0, 0.0), Instance(2, 10, 0, 5000.0), Instance(2, 0, 0, 0.0)]


def test_routing_by_hand():
    """Queues: version 1 [t2], version 2 [t0], initial [t1].
    t2 (l = 6000) may run anywhere; the version-1 group {A} is idle, so its
    gain equals the ideal 125 >= 0.3 * 125: A. t0 (l = 1000) may run on B or C
    (version 2): B loses throughput (10/0.007 -> 11/0.0081), idle C gains the
    ideal 333.3: C. t1 (initial, l = 100, versions >= 2 admitted): B gains
    11/0.0072 - 10/0.007 = 99.2, C gains 2/0.0031 - 1/0.003 = 311.8 >=
    0.3 * 476.2: C."""
    trajs = [Traj(2, 1000.0), Traj(None, 100.0), Traj(1, 6000.0)]
    target, after = R.route(C, 0.3, 2, INSTS, trajs)
    assert target == [2, 2, 0]
    assert after[0] == Instance(1, 1, 0, 6000.0)
    assert after[2] == Instance(2, 2, 0, 1100.0)
    assert after[1] == INSTS[1]
    # a higher threshold withholds t1 (311.8 < 0.7 * 476.2)
    target, _ = R.route(C, 0.7, 2, INSTS, trajs)
    assert target == [2, -1, 0]


def test_routing_stops_at_a_queue_with_no_candidate():
    """A version-3 trajectory has no instance of version >= 3: routing stops
    there, and the lower-priority initial queue is not served."""
    trajs = [Traj(2, 1000.0), Traj(None, 100.0), Traj(1, 6000.0), Traj(3, 10.0)]
    target, _ = R.route(C, 0.3, 2, INSTS, trajs)
    assert target == [2, -1, 0, -1]


def test_routing_prefers_the_older_version_group():
    """Both groups hold an idle instance with the same gain; the waterfall
    takes the lower-version group."""
    insts = [Instance(2, 0, 0, 0.0), Instance(1, 0, 0, 0.0)]
    target, _ = R.route(C, 0.3, 0, insts, [Traj(None, 50.0)])
    assert target == [1]


# ---------------------------------------------------------------------------
# the library's native version against the oracle
# ---------------------------------------------------------------------------
def _native():
    from paper_2601_12784_amd import binding as B
    return B


def _to_native(B, c):
    return B.sf_cost_model(c.k1, c.k2, c.k3, c.k4, c.k5, c.budget)


def test_native_matches_on_formulas():
    B = _native()
    m = _to_native(B, C)
    rng = np.random.default_rng(0)
    for _ in range(200):
        s = Instance(int(rng.integers(0, 4)), int(rng.integers(0, 300)), int(rng.integers(0, 3)),
                     float(rng.uniform(0, 1.2e4)))
        length = float(rng.uniform(1, 3000))
        ns = B.sf_instance_state(s.version, s.running, s.waiting, 0, s.kv)
        assert B.cost_throughput(m, ns) == pytest.approx(R.throughput(C, s), rel=1e-12, abs=0)
        assert B.cost_marginal_gain(m, ns, length) == pytest.approx(R.marginal_gain(C, s, length), rel=1e-9,
                                                                    abs=1e-9)
        assert B.cost_ideal_gain(m, length) == pytest.approx(R.ideal_gain(C, length), rel=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_native_routing_matches(seed):
    B = _native()
    rng = np.random.default_rng(seed)
    c = Coeffs(float(rng.uniform(1e-7, 1e-5)), 1e-3, 1e-4, float(rng.uniform(1e-4, 1e-2)), 1.0,
               float(rng.uniform(2e4, 2e5)))
    insts = [Instance(int(rng.integers(0, 4)), int(rng.integers(0, 200)), int(rng.integers(0, 2)),
                      float(rng.uniform(0, 1e5))) for _ in range(int(rng.integers(1, 12)))]
    trajs = [Traj(None if rng.random() < 0.3 else int(rng.integers(0, 4)), float(rng.integers(1, 20000)))
             for _ in range(int(rng.integers(0, 60)))]
    mu, minv = float(rng.choice([0.0, 0.3, 0.6])), int(rng.integers(0, 3))
    want_target, want_after = R.route(c, mu, minv, insts, trajs)
    got_target, got_after = B.route(_to_native(B, c), mu, minv, insts, trajs)
    assert got_target == want_target
    for g, w in zip(got_after, want_after):
        assert (g.version, g.running, g.waiting) == (w.version, w.running, w.waiting)
        assert g.kv == pytest.approx(w.kv, rel=1e-12, abs=0)


def test_native_rejects_bad_arguments():
    B = _native()
    L = B.lib()
    m = _to_native(B, C)
    out = np.zeros(4, np.int32)
    n = ctypes.c_int32()
    st = B.sf_instance_state(0, 1, 0, 0, 1.0)
    tr = B.sf_trajectory(0, 0, 1.0)
    assert L.sf_route(None, ctypes.c_double(0.3), 0, ctypes.byref(st), 1, ctypes.byref(tr), 1,
                      out.ctypes.data, ctypes.byref(n)) == 1
    assert L.sf_route(ctypes.byref(m), ctypes.c_double(0.3), 0, ctypes.byref(st), -1, ctypes.byref(tr), 1,
                      out.ctypes.data, ctypes.byref(n)) == 1
    assert L.sf_route(ctypes.byref(m), ctypes.c_double(float("nan")), 0, ctypes.byref(st), 1, ctypes.byref(tr), 1,
                      out.ctypes.data, ctypes.byref(n)) == 1
    neg = B.sf_trajectory(0, 0, -5.0)
    assert L.sf_route(ctypes.byref(m), ctypes.c_double(0.3), 0, ctypes.byref(st), 1, ctypes.byref(neg), 1,
                      out.ctypes.data, ctypes.byref(n)) == 1
