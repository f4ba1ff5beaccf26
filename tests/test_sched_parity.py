"""The out-of-order scheduler of libmetro.so (include/metro_sched.h) against the
oracle (oracle/scheduler.py): both are driven by the same seeded synthetic
world and event clock (synth.run_event_sim), and every hand-out and
completion -- time, step and members -- must be identical.  Host-only code, so
these run without a GPU; the library still has to be built.

Also: the C ABI's error conventions and state queries.
"""

import numpy as np
import pytest

from oracle.scheduler import CHEBYSHEV, EUCLIDEAN, OracleScheduler, valid_state
from paper_2411_03519_amd import synth

metro = pytest.importorskip("paper_2411_03519_amd.metro", reason="libmetro.so is not built")

CASES = [
    # seed, agents, grid, radius_p, metric, target, workers
    (0, 1, (10, 10), 4.0, CHEBYSHEV, 5, None),
    (1, 2, (10, 10), 4.0, CHEBYSHEV, 5, None),
    (2, 30, (20, 20), 4.0, CHEBYSHEV, 6, None),
    (3, 120, (100, 140), 4.0, CHEBYSHEV, 10, None),
    (4, 120, (100, 140), 4.0, CHEBYSHEV, 10, 4),
    (5, 300, (100, 140), 4.0, CHEBYSHEV, 6, 16),
    (6, 80, (50, 50), 2.0, EUCLIDEAN, 8, None),
    (7, 80, (50, 50), 7.5, EUCLIDEAN, 8, 3),
    (8, 60, (40, 40), 0.0, CHEBYSHEV, 8, 1),
]


@pytest.mark.parametrize("sync", [False, True])
@pytest.mark.parametrize("seed,n,grid,r,metric,target,workers", CASES)
def test_scheduler_matches_oracle(seed, n, grid, r, metric, target, workers, sync):
    world = synth.SimWorld(seed, n, grid=grid, diagonal=metric == CHEBYSHEV)
    got = metro.Scheduler(world.start, r, 1.0, metric, target, sync)
    want = OracleScheduler(world.start, r, 1.0, metric, target, sync)
    log_got, t_got = synth.run_event_sim(got, world, workers=workers)
    log_want, t_want = synth.run_event_sim(want, world, workers=workers)
    assert t_got == t_want
    assert log_got == log_want
    st = got.state()
    assert st["done"] and st["running"] == 0
    np.testing.assert_array_equal(st["steps"], np.full(n, target))
    np.testing.assert_array_equal(st["xy"], np.array(want.pos))
    assert valid_state(want.pos, want.step, r, 1.0, metric)


def test_state_while_running():
    pos = [(0, 0), (1, 0), (50, 50)]
    s = metro.Scheduler(pos, 4.0, 1.0, target_step=3)
    c0 = s.next()
    assert c0[1:] == (0, [0, 1])
    st = s.state()
    assert list(st["state"]) == [1, 1, 0] and st["running"] == 1 and not st["done"]
    s.ack(c0[0], [(0, 1), (1, 1)])
    st = s.state()
    assert list(st["steps"]) == [1, 1, 0] and list(st["state"]) == [0, 0, 0]
    np.testing.assert_array_equal(st["xy"], [[0, 1], [1, 1], [50, 50]])


def test_error_conventions():
    with pytest.raises(metro.MetroError) as e:
        metro.Scheduler([(0, 0)], -1.0, 1.0)
    assert e.value.name == "METRO_E_INVAL"
    with pytest.raises(metro.MetroError):
        metro.Scheduler([(0, 0)], 4.0, 1.0, target_step=0)
    with pytest.raises(metro.MetroError):
        metro.Scheduler([(0, 0)], 4.0, 1.0, metric=7)
    s = metro.Scheduler([(0, 0), (1, 0), (2, 0)], 4.0, 1.0, target_step=2)
    # a cluster larger than the caller's buffer is not handed out
    with pytest.raises(metro.MetroError) as e:
        s.next(cap=2)
    assert e.value.name == "METRO_E_CAPACITY"
    cid, step, members = s.next()
    assert (step, members) == (0, [0, 1, 2])
    with pytest.raises(metro.MetroError):   # unknown cluster
        s.ack(cid + 5, [(0, 0)] * 3)
    with pytest.raises(metro.MetroError):   # a move longer than max_vel
        s.ack(cid, [(0, 2), (1, 0), (2, 0)])
    s.ack(cid, [(0, 1), (1, 1), (2, 1)])    # the failed ack changed nothing
    with pytest.raises(metro.MetroError):   # acknowledged twice
        s.ack(cid, [(0, 1), (1, 1), (2, 1)])
    assert list(s.state()["steps"]) == [1, 1, 1]
