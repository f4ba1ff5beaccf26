"""The seeded input generators (paper_2411_03519_amd/synth.py): ranges,
determinism and the agent-trace readiness rule, checked on the CPU.

The generators hold none of the method's arithmetic; these tests pin the
workload recipes the parity tests and bench.py rely on.
"""

import numpy as np

from paper_2411_03519_amd import synth


def test_weight_draws_are_seeded_per_tensor():
    cfg = dict(synth.TINY, n_layers=1)
    a = synth.draw_tensor(cfg, "wq", 0, 7)
    b = synth.draw_tensor(cfg, "wq", 0, 7)
    c = synth.draw_tensor(cfg, "wk", 0, 7)
    np.testing.assert_array_equal(a, b)
    assert a.dtype == np.uint16 and a.shape == synth.tensor_shape(cfg, "wq")
    assert not np.array_equal(a[: c.shape[0]], c)
    vals = (a.astype(np.uint32) << 16).view(np.float32)
    assert abs(float(vals.std()) - 0.02) < 0.002
    norm = synth.draw_tensor(cfg, "attn_norm", 0, 7)
    assert np.all(norm == 0x3F80)  # 1.0


def test_agent_batches_follow_their_recipes():
    prompts, n_new = synth.llama8b_agent_batch(0)
    lens = np.array([len(p) for p in prompts])
    assert len(prompts) == 25 and n_new == 64
    assert lens.min() >= 256 and lens.max() <= 4096 and lens.sum() == 31527
    assert all(p.min() >= 0 and p.max() < synth.LLAMA3_8B["vocab"] for p in prompts)
    prefix, suffixes, n_new = synth.prefix_heavy_batch(0)
    assert len(prefix) == 1024 and len(suffixes) == 64 and n_new == 32
    assert min(len(s) for s in suffixes) >= 512 and max(len(s) for s in suffixes) <= 2048
    ctx, n_new = synth.llama70b_agent_batch(0)
    assert len(ctx) == 128 and n_new == 32
    assert min(len(c) for c in ctx) >= 1024 and max(len(c) for c in ctx) <= 3072
    starts = synth.trace_start_contexts(0)
    lens = np.array([len(c) for c in starts])
    assert len(starts) == 1000 and lens.min() >= 256 and lens.max() <= 4096
    assert 1300 < np.median(lens) < 1700
    feeds = synth.feed_tokens(3, 5, 4, 100)
    assert feeds.shape == (5, 4) and feeds.min() >= 0 and feeds.max() < 100
    np.testing.assert_array_equal(feeds, synth.feed_tokens(3, 5, 4, 100))


def test_agent_trace_ready_batches():
    batches = synth.agent_trace(0)
    sizes = np.array([len(b) for b in batches])
    assert len(batches) == 200
    assert sizes.min() >= 50 and sizes.max() <= 800 and sizes.max() >= 700
    assert all(len(np.unique(b)) == len(b) and b.min() >= 0 and b.max() < 1000 for b in batches if len(b))
    again = synth.agent_trace(0)
    assert all(np.array_equal(x, y) for x, y in zip(batches, again))


def test_agent_trace_readiness_rule_on_a_small_world():
    """Replay the documented rule step by step with plain loops on a small
    world and compare the ready batches (same seeded draws)."""
    n, grid, radius, ticks = 30, (12, 15), 2, 25
    got = synth.agent_trace(5, n_agents=n, grid=grid, radius=radius, ticks=ticks)
    H, W = grid
    rng = np.random.Generator(np.random.PCG64(5))
    rows, cols = rng.integers(0, H, n), rng.integers(0, W, n)  # the generator's draw order
    pos = [[int(rows[i]), int(cols[i])] for i in range(n)]
    step = [0] * n

    def new_budget(k):
        b = np.maximum(1, np.rint(np.exp(rng.normal(0.0, 1.5, k)))).astype(np.int64)
        return np.where(rng.random(k) < 0.2, 0, b)

    budget = list(new_budget(n))
    for t in range(ticks):
        ready = []
        for i in range(n):
            lag = any(max(abs(pos[i][0] - pos[j][0]), abs(pos[i][1] - pos[j][1])) <= radius and step[j] < step[i]
                      for j in range(n))
            ready.append(not lag)
        run = [i for i in range(n) if ready[i] and budget[i] > 0]
        np.testing.assert_array_equal(got[t], run)
        for i in run:
            budget[i] -= 1
        done = [i for i in range(n) if ready[i] and budget[i] == 0]
        mv = rng.integers(-1, 2, size=(len(done), 2))
        for k, i in enumerate(done):
            step[i] += 1
            pos[i] = [min(max(pos[i][0] + int(mv[k][0]), 0), H - 1), min(max(pos[i][1] + int(mv[k][1]), 0), W - 1)]
        nb = new_budget(len(done))
        for k, i in enumerate(done):
            budget[i] = int(nb[k])
