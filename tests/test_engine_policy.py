"""Mixed continuous batching: the admission rule (CPU only).

The oracle (oracle/engine_policy.py) is pinned by forwards worked out by hand
from the rule: running requests first, then prompt chunks lowest step first
within the token budget.  The library's engine, created without a model (it
then plans forwards and appends stand-in tokens), must form exactly the
oracle's items forward after forward over seeded random request streams, and
retire the same requests.
"""

import numpy as np
import pytest

from oracle import engine_policy as P


def run_oracle(reqs, cfg, n_forwards):
    out = []
    for _ in range(n_forwards):
        items = P.plan(reqs, *cfg)
        done = P.apply(reqs, items)
        out.append((items, done))
    return out


def three_requests():
    # (id, step, arrival, prompt tokens, outputs)
    return [P.Request(0, 2, 0, 100, 3), P.Request(1, 0, 1, 700, 2), P.Request(2, 1, 2, 50, 1)]


def test_oracle_priority_by_hand():
    got = run_oracle(three_requests(), (512, 256, 8, True), 5)
    want = [
        # lowest step first: 256 of r1's 700, r2's 50 (its first token: done), r0's 100
        ([(1, 256, False), (2, 50, False), (0, 100, False)], [2]),
        # r0 runs (one token), then r1's next chunk
        ([(0, 1, True), (1, 256, False)], []),
        # r0's third token retires it; r1's last 188 prompt tokens give its first token
        ([(0, 1, True), (1, 188, False)], [0]),
        ([(1, 1, True)], [1]),
        ([], []),
    ]
    assert got == want


def test_oracle_submission_order_without_priority():
    got = run_oracle(three_requests(), (512, 256, 8, False), 1)
    assert got[0][0] == [(0, 100, False), (1, 256, False), (2, 50, False)]


def test_oracle_budget_cuts_the_last_chunk():
    got = run_oracle(three_requests(), (300, 256, 8, True), 1)
    # 256 for r1, the remaining 44 of the budget for r2, nothing left for r0
    assert got[0][0] == [(1, 256, False), (2, 44, False)]


def test_oracle_running_requests_first_and_item_cap():
    reqs = [P.Request(i, s, i, 10, 5) for i, s in enumerate((3, 1, 2, 0))]
    run_oracle(reqs, (64, 16, 8, True), 1)           # all four prompts in: all running
    items = P.plan(reqs, 64, 16, 2, True)
    assert items == [(3, 1, True), (1, 1, True)]      # steps 0 and 1 of the four running
    reqs.append(P.Request(9, 0, 9, 40, 1))
    items = P.plan(reqs, 6, 16, 8, True)
    assert items == [(3, 1, True), (1, 1, True), (2, 1, True), (0, 1, True), (9, 2, False)]


@pytest.fixture(scope="module")
def metro(repo_root):
    import os
    if not os.path.exists(os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro as m
    return m


@pytest.mark.parametrize("seed,priority", [(0, True), (1, True), (2, False), (3, True)])
def test_engine_plans_equal_the_oracle(metro, seed, priority):
    rng = np.random.default_rng(seed)
    cfg = (int(rng.integers(64, 1024)), int(rng.integers(16, 300)), int(rng.integers(2, 12)), priority)
    eng = metro.Engine(None, max_tokens=cfg[0], chunk=cfg[1], max_items=cfg[2], priority=priority)
    reqs, next_id = [], 0
    for forward in range(200):
        for _ in range(int(rng.poisson(0.6))):
            n_prompt, n_out, step = int(rng.integers(1, 900)), int(rng.integers(1, 12)), int(rng.integers(0, 6))
            reqs.append(P.Request(next_id, step, next_id, n_prompt, n_out))
            eng.submit(next_id, step, np.zeros(n_prompt, np.int32), n_out)
            next_id += 1
        want = P.plan(reqs, *cfg)
        done = P.apply(reqs, want)
        n = eng.step()
        assert n == len(want)
        assert eng.last_plan() == want, f"forward {forward}"
        got_done = eng.finished()
        assert got_done == done
        for rid in done:
            assert len(eng.result(rid)) == next(r.n_out for r in reqs if r.rid == rid)
        reqs = [r for r in reqs if r.rid not in done]
    st = eng.stats()
    assert st["live"] == len(reqs)
    assert st["waiting"] == sum(r.waiting for r in reqs)


def test_engine_rejects_bad_arguments(metro):
    with pytest.raises(metro.MetroError):
        metro.Engine(None, max_tokens=0, chunk=16, max_items=4)
    eng = metro.Engine(None, max_tokens=64, chunk=16, max_items=4)
    eng.submit(5, 0, [1, 2, 3], 2)
    with pytest.raises(metro.MetroError, match="live"):
        eng.submit(5, 1, [1], 1)
    with pytest.raises(metro.MetroError):
        eng.submit(6, 0, [], 1)
    with pytest.raises(metro.MetroError, match="unknown"):
        eng.result(77)
