"""Pins for the scheduler oracle (oracle/scheduler.py) against what the paper
fixes, independently of how the oracle evaluates its rules:

* the thresholds of the coupled and blocked rules of §3.3 at their boundaries,
  worked out by hand for both distance metrics;
* clusters are the connected components of the coupled relation (§3.4), and a
  blocked member holds back its whole cluster;
* the ready queue serves the lowest step first (§3.5);
* the validity condition of §3.3 (agents at different steps never perceive
  each other: dist > radius_p + (|s_A - s_B| - 1) max_vel) holds after every
  completion in random runs -- the property the rules exist to keep;
* every agent reaches the target step (no deadlock), an isolated agent never
  waits for a far-away one, and with unlimited workers the out-of-order run
  never takes longer than the parallel-sync baseline of Algorithm 1 (each step
  of every agent starts no later than in the synchronous schedule).
"""

import pytest

from oracle.scheduler import CHEBYSHEV, EUCLIDEAN, DONE, OracleScheduler, valid_state
from paper_2411_03519_amd import synth


def sched(positions, steps=None, r=4.0, v=1.0, metric=CHEBYSHEV, target=10, sync=False):
    s = OracleScheduler(positions, r, v, metric, target, sync)
    if steps is not None:
        s.step = list(steps)
    return s


@pytest.mark.parametrize("metric", [CHEBYSHEV, EUCLIDEAN])
def test_coupled_threshold(metric):
    # r + v = 5: same step at distance 5 is coupled, at 6 is not
    assert sched([(0, 0), (5, 0)], metric=metric).coupled(0, 1)
    assert not sched([(0, 0), (6, 0)], metric=metric).coupled(0, 1)
    # different steps are never coupled
    assert not sched([(0, 0), (1, 0)], steps=[1, 0], metric=metric).coupled(0, 1)


def test_coupled_threshold_diagonal():
    # (4, 4): Chebyshev 4 <= 5 coupled; Euclidean 5.66 > 5 not
    assert sched([(0, 0), (4, 4)], metric=CHEBYSHEV).coupled(0, 1)
    assert not sched([(0, 0), (4, 4)], metric=EUCLIDEAN).coupled(0, 1)
    # (3, 4): Euclidean exactly 5 -> coupled
    assert sched([(0, 0), (3, 4)], metric=EUCLIDEAN).coupled(0, 1)


@pytest.mark.parametrize("metric", [CHEBYSHEV, EUCLIDEAN])
def test_blocked_threshold(metric):
    # A at step 2, B at step 0: blocked iff dist <= (2 - 0 + 1) * 1 + 4 = 7
    assert sched([(0, 0), (7, 0)], steps=[2, 0], metric=metric).blocked_by(0, 1)
    assert not sched([(0, 0), (8, 0)], steps=[2, 0], metric=metric).blocked_by(0, 1)
    # one step ahead: threshold 6
    assert sched([(0, 0), (0, 6)], steps=[1, 0], metric=metric).blocked_by(0, 1)
    assert not sched([(0, 0), (0, 7)], steps=[1, 0], metric=metric).blocked_by(0, 1)
    # the agent behind is never blocked by the one ahead
    assert not sched([(0, 0), (1, 0)], steps=[0, 3], metric=metric).blocked_by(0, 1)
    # other radius and speed: (3 - 1 + 1) * 2.5 + 1.5 = 9
    assert sched([(0, 0), (9, 0)], steps=[3, 1], r=1.5, v=2.5, metric=metric).blocked_by(0, 1)
    assert not sched([(0, 0), (10, 0)], steps=[3, 1], r=1.5, v=2.5, metric=metric).blocked_by(0, 1)


def test_clusters_are_connected_components():
    # chain 0-1-2 (each link 5 apart, ends 10 apart) and a lone agent 3
    s = sched([(0, 0), (5, 0), (10, 0), (50, 50)])
    assert s.clusters() == [[0, 1, 2], [3]]
    # different steps split the chain
    s = sched([(0, 0), (5, 0), (10, 0), (50, 50)], steps=[0, 0, 1, 0])
    assert sorted(s.clusters()) == [[0, 1], [2], [3]]


def test_blocked_member_holds_its_cluster():
    # 0 and 1 coupled at step 1; agent 2 at step 0 is within 6 of agent 1 only
    s = sched([(0, 0), (5, 0), (11, 0)], steps=[1, 1, 0])
    assert not s.blocked(0) and s.blocked(1)
    ready = s.ready_clusters()
    assert [0, 1] not in ready and [2] in ready


def test_priority_lowest_step_then_id():
    s = sched([(0, 0), (50, 0), (100, 0), (0, 100)], steps=[2, 1, 1, 3])
    assert s.ready_clusters() == [[1], [2], [0], [3]]
    assert s.next() == (0, 1, [1])
    assert s.next() == (1, 1, [2])


def test_sync_one_cluster_per_step():
    s = sched([(0, 0), (50, 0), (100, 0)], sync=True, target=2)
    cid, step, members = s.next()
    assert (step, members) == (0, [0, 1, 2]) and s.next() is None
    s.ack(cid, [(0, 1), (50, 1), (100, 1)])
    cid, step, members = s.next()
    assert (step, members) == (1, [0, 1, 2])
    s.ack(cid, [(0, 1), (50, 1), (100, 1)])
    assert s.next() is None and s.done()


def test_move_longer_than_max_vel_is_rejected():
    s = sched([(0, 0)])
    cid, _, _ = s.next()
    with pytest.raises(ValueError):
        s.ack(cid, [(2, 0)])


@pytest.mark.parametrize("seed,n,grid,r,metric,workers", [
    (0, 40, (30, 30), 4.0, CHEBYSHEV, None),
    (1, 80, (60, 60), 4.0, CHEBYSHEV, 3),
    (2, 60, (40, 40), 2.0, EUCLIDEAN, None),
    (3, 100, (100, 140), 4.0, CHEBYSHEV, 8),
    (4, 50, (25, 25), 0.0, EUCLIDEAN, 2),
])
def test_validity_condition_holds_throughout(seed, n, grid, r, metric, workers):
    world = synth.SimWorld(seed, n, grid=grid, diagonal=metric == CHEBYSHEV)
    s = OracleScheduler(world.start, r, 1.0, metric, target_step=8)
    checked = []

    def check(sc):
        assert valid_state(sc.pos, sc.step, r, 1.0, metric), "validity condition of §3.3 violated"
        checked.append(1)

    synth.run_event_sim(s, world, workers=workers, on_ack=check)
    assert s.done() and all(st == DONE for st in s.state)
    assert len(checked) > 0


def test_isolated_agent_runs_ahead():
    # agent 0 is far from the others (who are coupled into one slow cluster):
    # it finishes every step before they finish their first
    world = synth.SimWorld(5, 4, grid=(200, 200))
    world.start[:] = [(0, 0), (190, 190), (193, 190), (196, 190)]
    s = OracleScheduler(world.start, 4.0, 1.0, CHEBYSHEV, target_step=5)
    got = s.next()
    assert got[2] == [0]
    got2 = s.next()
    assert got2[2] == [1, 2, 3]
    # complete agent 0's steps while the cluster keeps running
    pos0 = (0, 0)
    for step in range(5):
        new = world.move(0, step, pos0)
        s.ack(got[0], [new])
        pos0 = new
        got = s.next()
        if step < 4:
            assert got is not None and got[2] == [0] and got[1] == step + 1
    assert got is None and s.step[0] == 5 and s.step[1] == 0


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_out_of_order_never_slower_than_sync(seed):
    world = synth.SimWorld(seed, 120, grid=(100, 140))
    ooo = OracleScheduler(world.start, 4.0, 1.0, CHEBYSHEV, target_step=10)
    syn = OracleScheduler(world.start, 4.0, 1.0, CHEBYSHEV, target_step=10, sync=True)
    _, t_ooo = synth.run_event_sim(ooo, world)
    _, t_syn = synth.run_event_sim(syn, world)
    assert t_ooo <= t_syn
    assert ooo.done() and syn.done()


def test_splitmix64_reference_values():
    # SplitMix64 outputs for counters 0, 1, 2 as published with the generator
    # (first outputs of a SplitMix64 stream seeded with 0)
    assert synth.splitmix64(0) == 0xE220A8397B1DCDAF
    assert synth.splitmix64(0x9E3779B97F4A7C15) == 0x6E789E6AA1B965F4
    assert synth.splitmix64((2 * 0x9E3779B97F4A7C15) & ((1 << 64) - 1)) == 0x06C45D188009454F
