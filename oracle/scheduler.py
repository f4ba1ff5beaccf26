"""Oracle for the out-of-order agent scheduler — TEST INFRASTRUCTURE ONLY.

Only ``tests/`` and ``bench.py``'s CPU legs may import this module; the product
(``libmetro.so``, ``include/metro_sched.h``) never uses it.

It follows the controller of AI Metropolis (arXiv 2411.03519) step by step, in
plain Python loops over agents, in the paper's terms:

* §3.3 (and the appendix, which derives them from the validity condition):
  agents A, B with steps s_A, s_B are *coupled* when s_A == s_B and
  dist(A, B) <= radius_p + max_vel; A is *blocked* by B when s_B < s_A and
  dist(A, B) <= (s_A - s_B + 1) * max_vel + radius_p.
* §3.4: a *cluster* is a group of coupled agents waiting at the same step
  (connected components of the coupled relation); it is ready when none of its
  members is blocked by any agent.
* §3.5 / Algorithm 3: ready clusters are served lowest step first (ties: the
  lowest agent id, the reading used here).
* Algorithm 1 (parallel-sync baseline): all agents form one cluster per step,
  released when every agent has finished the previous step.

The step of an agent counts the steps it has completed.  Distances are
Chebyshev (max(|dx|, |dy|), the square perception area of a grid world) or
Euclidean (compared as squares), as configured.

``valid_state`` checks the validity condition of §3.3 itself, which the rules
are meant to preserve, and is used as an independent pin.
"""

from __future__ import annotations

import math

CHEBYSHEV, EUCLIDEAN = 0, 1
WAITING, RUNNING, DONE = 0, 1, 2


def within(metric: int, a: tuple, b: tuple, thr: float) -> bool:
    """dist(a, b) <= thr."""
    dx = abs(float(a[0]) - float(b[0]))
    dy = abs(float(a[1]) - float(b[1]))
    if metric == CHEBYSHEV:
        return max(dx, dy) <= thr
    return dx * dx + dy * dy <= thr * thr


def distance(metric: int, a: tuple, b: tuple) -> float:
    dx = abs(a[0] - b[0])
    dy = abs(a[1] - b[1])
    return float(max(dx, dy)) if metric == CHEBYSHEV else math.sqrt(dx * dx + dy * dy)


class OracleScheduler:
    def __init__(self, positions, radius_p: float, max_vel: float, metric: int = CHEBYSHEV,
                 target_step: int = 10, sync: bool = False):
        self.pos = [tuple(int(v) for v in p) for p in positions]
        self.n = len(self.pos)
        self.r = float(radius_p)
        self.v = float(max_vel)
        self.metric = metric
        self.target = target_step
        self.sync = sync
        self.step = [0] * self.n
        self.state = [WAITING] * self.n
        self.running = {}   # cluster id -> (step, members)
        self.next_id = 0

    # --- §3.3 -------------------------------------------------------------
    def coupled(self, a: int, b: int) -> bool:
        return self.step[a] == self.step[b] and within(self.metric, self.pos[a], self.pos[b], self.v + self.r)

    def blocked_by(self, a: int, b: int) -> bool:
        if self.step[b] >= self.step[a]:
            return False
        thr = (self.step[a] - self.step[b] + 1) * self.v + self.r
        return within(self.metric, self.pos[a], self.pos[b], thr)

    def blocked(self, a: int) -> bool:
        return any(self.blocked_by(a, b) for b in range(self.n) if b != a)

    # --- §3.4 -------------------------------------------------------------
    def clusters(self):
        """Connected components of the coupled relation among waiting agents,
        each as a sorted member list, found by breadth-first search."""
        waiting = [a for a in range(self.n) if self.state[a] == WAITING]
        seen = set()
        out = []
        for a in waiting:
            if a in seen:
                continue
            comp, frontier = [a], [a]
            seen.add(a)
            while frontier:
                u = frontier.pop()
                for w in waiting:
                    if w not in seen and self.coupled(u, w):
                        seen.add(w)
                        comp.append(w)
                        frontier.append(w)
            out.append(sorted(comp))
        return out

    def ready_clusters(self):
        """Ready clusters in serving order: lowest step, then lowest agent id (§3.5)."""
        if self.sync:
            if self.running:
                return []
            waiting = [a for a in range(self.n) if self.state[a] == WAITING]
            return [waiting] if waiting else []
        ready = [c for c in self.clusters() if not any(self.blocked(a) for a in c)]
        return sorted(ready, key=lambda c: (self.step[c[0]], c[0]))

    # --- controller --------------------------------------------------------
    def next(self):
        """(cluster id, step, members) of the next ready cluster, or None."""
        ready = self.ready_clusters()
        if not ready:
            return None
        members = ready[0]
        cid = self.next_id
        self.next_id += 1
        for a in members:
            self.state[a] = RUNNING
        self.running[cid] = (self.step[members[0]], members)
        return cid, self.step[members[0]], list(members)

    def ack(self, cid: int, new_positions):
        step, members = self.running.pop(cid)
        for a, p in zip(members, new_positions):
            p = (int(p[0]), int(p[1]))
            if not within(self.metric, self.pos[a], p, self.v):
                raise ValueError(f"agent {a} moves farther than max_vel")
            self.pos[a] = p
            self.step[a] += 1
            self.state[a] = DONE if self.step[a] >= self.target else WAITING

    def done(self) -> bool:
        return all(s == DONE for s in self.state)


def valid_state(positions, steps, radius_p: float, max_vel: float, metric: int = CHEBYSHEV) -> bool:
    """The validity condition of §3.3: agents at different steps keep
    dist(A, B) > radius_p + (|s_A - s_B| - 1) * max_vel."""
    n = len(positions)
    for a in range(n):
        for b in range(a + 1, n):
            if steps[a] != steps[b]:
                thr = radius_p + (abs(steps[a] - steps[b]) - 1) * max_vel
                if distance(metric, positions[a], positions[b]) <= thr:
                    return False
    return True
