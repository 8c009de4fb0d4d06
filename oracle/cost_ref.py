"""Throughput cost model and the routing strategy, written plainly.

TEST INFRASTRUCTURE ONLY. The paper's coordinator estimates each rollout
instance's generation throughput from a snapshot (App. B.1, final throughput
equation) and routes trajectories by their marginal throughput gain with a
waterfall over instance model versions (Sec. 5.3, routing strategy; App. D,
check-routable and routing algorithms). This module states those steps in the
paper's order and notation, for comparison with the library's native version:

  T_i(S) = n / (k1 * kv + max(k2, k3 * n) + k4),   n = |run_trajs| (0 if n = 0)
  gamma_i = [kv_i + k5 * l <= M and |wait_i| = 0]
  S'[i]: kv += gamma * k5 * l, n += gamma;  dT_i = T_i(S') - T_i(S)
  dT_ideal = 1 / (k1 * k5 * l + max(k2, k3) + k4)
  routing: trajectories in queues by version, oldest first, initial ones last;
  for the head of the current queue: candidates = instances where it may run
  (initial: the staleness check admits the instance's version; else the
  instance's version >= the trajectory's); none -> stop. Candidates are
  grouped by increasing instance version; in the first group whose best gain
  (first maximum in instance order) is >= mu * dT_ideal, route there, update
  that instance as in S', and continue; if no group qualifies -> stop.
The staleness manager's check for an initial trajectory is modelled as
"instance version >= min_initial_version".
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass
class Coeffs:
    k1: float
    k2: float
    k3: float
    k4: float
    k5: float
    budget: float            # M, in the unit of kv (same as k5 * length)


@dataclass
class Instance:
    version: int
    running: int
    waiting: int
    kv: float


@dataclass
class Traj:
    version: int | None      # None: initial trajectory
    length: float


def throughput(c: Coeffs, s: Instance) -> float:
    n = s.running
    if n == 0:
        return 0.0
    return n / (c.k1 * s.kv + max(c.k2, c.k3 * n) + c.k4)


def after_routing(c: Coeffs, s: Instance, length: float) -> Instance:
    gamma = 1 if (s.kv + c.k5 * length <= c.budget and s.waiting == 0) else 0
    if gamma:
        return Instance(s.version, s.running + 1, s.waiting, s.kv + c.k5 * length)
    return Instance(s.version, s.running, s.waiting + 1, s.kv)


def marginal_gain(c: Coeffs, s: Instance, length: float) -> float:
    return throughput(c, after_routing(c, s, length)) - throughput(c, s)


def ideal_gain(c: Coeffs, length: float) -> float:
    return 1.0 / (c.k1 * (0 + c.k5 * length) + max(c.k2, c.k3 * 1) + c.k4) - 0


def routable(s: Instance, t: Traj, min_initial_version: int) -> bool:
    if t.version is None:
        return s.version >= min_initial_version
    return s.version >= t.version


def route(c: Coeffs, mu: float, min_initial_version: int, insts: list, trajs: list):
    """Returns (target per trajectory, or -1; updated instances)."""
    insts = [Instance(s.version, s.running, s.waiting, s.kv) for s in insts]
    target = [-1] * len(trajs)
    keyed = sorted(range(len(trajs)), key=lambda j: (trajs[j].version is None,
                                                     trajs[j].version if trajs[j].version is not None else 0, j))
    queues = []
    for j in keyed:
        v = trajs[j].version
        if queues and queues[-1][0] == v:
            queues[-1][1].append(j)
        else:
            queues.append((v, [j]))
    stop = False
    for _, queue in queues:
        if stop:
            break
        while queue:
            j = queue[0]
            t = trajs[j]
            cands = [i for i, s in enumerate(insts) if routable(s, t, min_initial_version)]
            if not cands:
                stop = True
                break
            versions = sorted({insts[i].version for i in cands})
            groups = [[i for i in cands if insts[i].version == v] for v in versions]
            ideal = ideal_gain(c, t.length)
            selected = None
            for grp in groups:
                best, best_gain = None, float("-inf")
                for i in grp:
                    g = marginal_gain(c, insts[i], t.length)
                    if g > best_gain:
                        best, best_gain = i, g
                if best_gain >= mu * ideal:
                    selected = best
                    break
            if selected is None:
                stop = True
                break
            target[j] = selected
            queue.pop(0)
            insts[selected] = after_routing(c, insts[selected], t.length)
    return target, insts
