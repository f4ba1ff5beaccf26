"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds no part of the forward pass: it only draws weights, prompts,
context lengths and agent-trace batch sizes from seeded generators, so that the
HIP path and the oracle can be fed identical inputs.

The paper measures on recorded Generative-Agents traces and trained Llama-3
checkpoints (§4.1), neither of which is available; the inputs below stand in for
them with the shapes of those workloads (Llama-3 8B / 70B layer shapes,
random N(0, 0.02) weights, prompt lengths of the agents' calls, 100x140 grid
world with up to 1000 agents as in §4.2-§4.3).
"""

from __future__ import annotations

import math

import numpy as np

# ----------------------------------------------------------------------------
# Model shapes (Llama-3 family; the tiny one is a test-sized member)
# ----------------------------------------------------------------------------

TINY = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
            ffn_dim=688, vocab=4096, rope_base=10000.0, rms_eps=1e-5)
LLAMA3_8B = dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                 ffn_dim=14336, vocab=128256, rope_base=500000.0, rms_eps=1e-5)
LLAMA3_70B = dict(n_layers=80, d_model=8192, n_heads=64, n_kv_heads=8, head_dim=128,
                  ffn_dim=28672, vocab=128256, rope_base=500000.0, rms_eps=1e-5)

PAGE = 16  # tokens per KV page

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wgate", "wup", "wdown")
_TENSOR_ID = {name: i for i, name in enumerate(("embed", "final_norm", "lm_head") + LAYER_TENSORS)}


def with_layers(shape: dict, n_layers: int) -> dict:
    s = dict(shape)
    s["n_layers"] = n_layers
    return s


def tensor_shape(cfg: dict, name: str) -> tuple:
    d, F, V = cfg["d_model"], cfg["ffn_dim"], cfg["vocab"]
    nq, nkv, hd = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    return {
        "embed": (V, d), "lm_head": (V, d), "final_norm": (d,),
        "attn_norm": (d,), "ffn_norm": (d,),
        "wq": (nq * hd, d), "wk": (nkv * hd, d), "wv": (nkv * hd, d), "wo": (d, nq * hd),
        "wgate": (F, d), "wup": (F, d), "wdown": (d, F),
    }[name]


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 storage bits, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _rng(seed: int, name: str, layer: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, _TENSOR_ID[name], layer + 1])))


def draw_tensor(cfg: dict, name: str, layer: int, seed: int, norm: str = "ones") -> np.ndarray:
    """One weight tensor as bf16 bits.  Matrices ~ N(0, 0.02); RMSNorm gains are
    1.0 (``norm="ones"``, the Llama initialisation) or 1 + N(0, 0.1)
    (``norm="random"``, so that a kernel that ignored the gain would show)."""
    shp = tensor_shape(cfg, name)
    if name.endswith("norm"):
        if norm == "ones":
            return f32_to_bf16_bits(np.ones(shp, dtype=np.float32))
        g = _rng(seed, name, layer).standard_normal(shp, dtype=np.float32)
        return f32_to_bf16_bits(1.0 + np.float32(0.1) * g)
    w = _rng(seed, name, layer).standard_normal(shp, dtype=np.float32)
    w *= np.float32(0.02)
    return f32_to_bf16_bits(w)


def llama_weights(cfg: dict, seed: int, norm: str = "ones", workers: int = 1) -> dict:
    """All weights of a Llama-style decoder as bf16 bit arrays ([out, in] row-major).

    Every tensor has its own random stream, so ``workers`` > 1 (tensors drawn
    on that many threads) gives the same arrays."""
    jobs = [("embed", -1), ("final_norm", -1), ("lm_head", -1)]
    jobs += [(n, li) for li in range(cfg["n_layers"]) for n in LAYER_TENSORS]
    if workers > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=workers) as ex:
            arrs = list(ex.map(lambda j: draw_tensor(cfg, j[0], j[1], seed, norm), jobs))
    else:
        arrs = [draw_tensor(cfg, n, li, seed, norm) for n, li in jobs]
    got = dict(zip(jobs, arrs))
    return {
        "embed": got[("embed", -1)],
        "final_norm": got[("final_norm", -1)],
        "lm_head": got[("lm_head", -1)],
        "layers": [{n: got[(n, li)] for n in LAYER_TENSORS} for li in range(cfg["n_layers"])],
    }


# ----------------------------------------------------------------------------
# Prompts and context lengths
# ----------------------------------------------------------------------------

def prompt_tokens(rng: np.random.Generator, lengths, vocab: int) -> list:
    """Token ids uniform over [0, vocab) for each requested length."""
    return [rng.integers(0, vocab, size=int(n), dtype=np.int64) for n in lengths]


def lognormal_lengths(rng: np.random.Generator, n: int, median: float, sigma: float,
                      lo: int, hi: int) -> np.ndarray:
    """round(exp(N(ln median, sigma))) clipped to [lo, hi]."""
    x = np.exp(rng.normal(math.log(median), sigma, size=n))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def tiny_agent_batch(seed: int = 0):
    """4 agent requests, prompt lengths uniform in [32, 128], 16 generated tokens each."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lengths = rng.integers(32, 129, size=4)
    return prompt_tokens(rng, lengths, TINY["vocab"]), 16


def llama8b_agent_batch(seed: int = 0, n_agents: int = 25, vocab: int = LLAMA3_8B["vocab"]):
    """25 agent requests with prompt lengths lognormal (median 1200, sigma 0.5)
    clipped to [256, 4096]; 64 generated tokens each."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lengths = lognormal_lengths(rng, n_agents, 1200.0, 0.5, 256, 4096)
    return prompt_tokens(rng, lengths, vocab), 64


def prefix_heavy_batch(seed: int = 0, n_agents: int = 64, vocab: int = LLAMA3_8B["vocab"]):
    """A shared 1024-token system prefix plus one unique suffix per agent with
    length uniform in [512, 2048]; 32 generated tokens each."""
    rng = np.random.Generator(np.random.PCG64(seed))
    prefix = rng.integers(0, vocab, size=1024, dtype=np.int64)
    lengths = rng.integers(512, 2049, size=n_agents)
    return prefix, prompt_tokens(rng, lengths, vocab), 32


def agent_call_prompts(seed: int, n_agents: int, n_rounds: int, vocab: int, preamble: int = 256,
                       persona: int = 192, obs_median: float = 160.0, obs_sigma: float = 0.6, obs_lo: int = 16,
                       obs_hi: int = 1024, out_median: float = 18.0, out_sigma: float = 0.6, out_lo: int = 4,
                       out_hi: int = 64):
    """Successive LLM calls of agents whose prompts share text: a preamble
    common to every agent and call (instructions), a persona per agent that is
    the same in each of its calls, and a fresh observation per call (length
    lognormal, clipped); output lengths lognormal, clipped.  The defaults give
    a mean call of about 640 prompt and 22 output tokens.
    Returns (prompts[round][agent] int64 arrays, out_lens[round][agent])."""
    rng = np.random.Generator(np.random.PCG64([seed, 428]))
    pre = rng.integers(0, vocab, size=preamble, dtype=np.int64)
    pers = [rng.integers(0, vocab, size=persona, dtype=np.int64) for _ in range(n_agents)]
    prompts, outs = [], []
    for _ in range(n_rounds):
        obs = lognormal_lengths(rng, n_agents, obs_median, obs_sigma, obs_lo, obs_hi)
        prompts.append([np.concatenate([pre, pers[a], rng.integers(0, vocab, size=int(obs[a]), dtype=np.int64)])
                        for a in range(n_agents)])
        outs.append(lognormal_lengths(rng, n_agents, out_median, out_sigma, out_lo, out_hi))
    return prompts, outs


def uniform_contexts(seed: int, n_agents: int, lo: int, hi: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(lo, hi + 1, size=n_agents).astype(np.int64)


def trace_start_contexts(seed: int = 0, n_agents: int = 1000, vocab: int = LLAMA3_8B["vocab"]) -> list:
    """Starting contexts of the trace-driven workload: lengths lognormal
    (median 1500, sigma 0.5) clipped to [256, 4096], uniform token ids."""
    rng = np.random.Generator(np.random.PCG64([seed, 1500]))
    return prompt_tokens(rng, lognormal_lengths(rng, n_agents, 1500.0, 0.5, 256, 4096), vocab)


def llama70b_agent_batch(seed: int = 0, n_agents: int = 128, vocab: int = LLAMA3_70B["vocab"]):
    """128 agent contexts with lengths uniform in [1024, 3072]; 32 generated tokens each."""
    rng = np.random.Generator(np.random.PCG64([seed, 70]))
    return prompt_tokens(rng, rng.integers(1024, 3073, size=n_agents), vocab), 32


def feed_tokens(seed: int, n_rows: int, n_steps: int, vocab: int) -> np.ndarray:
    """Token ids [n_rows, n_steps] fed to decode steps under teacher forcing."""
    rng = np.random.Generator(np.random.PCG64([seed, 7]))
    return rng.integers(0, vocab, size=(n_rows, n_steps), dtype=np.int64)


# ----------------------------------------------------------------------------
# Synthetic agent trace: ready-batch sizes of an out-of-order simulation
# ----------------------------------------------------------------------------

def agent_trace(seed: int = 0, n_agents: int = 1000, grid=(100, 140), radius: int = 5,
                ticks: int = 200, p_idle: float = 0.2, budget_sigma: float = 1.5):
    """Ready batches of a seeded out-of-order agent simulation.

    Agents random-walk on a grid (one of the 8 neighbouring cells or stay,
    clamped at the border) each time they finish a simulation step.  A step of
    an agent carries a token budget (0 with probability ``p_idle``, else
    ``max(1, round(lognormal(0, budget_sigma)))``).  An agent is *ready* when no
    agent within Chebyshev distance ``radius`` is at a smaller step -- the
    perception radius plus one step of movement (4 + 1 in the paper's world,
    §3.2), with the blocking radius held constant.  Each tick decodes one token
    for every ready agent with budget left; an agent whose budget is spent
    advances its step and moves.

    Returns a list with, per tick, the int64 array of agent ids decoded.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    H, W = grid
    pos = np.stack([rng.integers(0, H, n_agents), rng.integers(0, W, n_agents)], axis=1)
    step = np.zeros(n_agents, dtype=np.int64)

    def new_budget(n):
        b = np.maximum(1, np.rint(np.exp(rng.normal(0.0, budget_sigma, n)))).astype(np.int64)
        return np.where(rng.random(n) < p_idle, 0, b)

    budget = new_budget(n_agents)
    batches = []
    for _ in range(ticks):
        d = np.maximum(np.abs(pos[:, None, 0] - pos[None, :, 0]), np.abs(pos[:, None, 1] - pos[None, :, 1]))
        lagging = (d <= radius) & (step[None, :] < step[:, None])
        ready = ~lagging.any(axis=1)
        run = ready & (budget > 0)
        batches.append(np.nonzero(run)[0].astype(np.int64))
        budget[run] -= 1
        done = ready & (budget == 0)
        idx = np.nonzero(done)[0]
        step[idx] += 1
        mv = rng.integers(-1, 2, size=(len(idx), 2))
        pos[idx] = np.clip(pos[idx] + mv, 0, [H - 1, W - 1])
        budget[idx] = new_budget(len(idx))
    return batches


# ----------------------------------------------------------------------------
# Synthetic world for the out-of-order scheduler (inputs only: positions,
# moves and per-step work, drawn from a counter-based generator so that they
# do not depend on the order in which a scheduler runs the agents)
# ----------------------------------------------------------------------------

_M64 = (1 << 64) - 1


def splitmix64(z: int) -> int:
    """SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): one 64-bit output for counter z."""
    z = (z + 0x9E3779B97F4A7C15) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def agent_draw(seed: int, agent: int, step: int, k: int) -> int:
    """The k-th 64-bit draw of (agent, step)."""
    return splitmix64((((seed * 1_000_003 + agent) * 1_000_033 + step) * 16 + k) & _M64)


class SimWorld:
    """Agents on a W x H grid (the paper's world is 100 x 140, §4.2).

    Each agent's step ends with a move to one of the 8 neighbouring cells or
    staying (4 neighbours for the Euclidean metric, so a move is at most 1),
    clamped at the border, and costs some LLM work: none with probability
    p_idle, else ``max(1, round(exp(N(0, sigma))))`` units (a token budget, or
    ticks of an abstract clock)."""

    def __init__(self, seed: int, n_agents: int, grid=(100, 140), p_idle: float = 0.2, sigma: float = 1.5,
                 diagonal: bool = True):
        self.seed, self.n = seed, n_agents
        self.H, self.W = grid
        self.p_idle, self.sigma, self.diagonal = p_idle, sigma, diagonal
        rng = np.random.Generator(np.random.PCG64([seed, 3]))
        self.start = np.stack([rng.integers(0, self.H, n_agents), rng.integers(0, self.W, n_agents)], axis=1)

    def move(self, agent: int, step: int, pos) -> tuple:
        h = agent_draw(self.seed, agent, step, 0)
        if self.diagonal:
            dx, dy = h % 3 - 1, (h >> 8) % 3 - 1
        else:
            dx, dy = ((0, 0), (1, 0), (-1, 0), (0, 1), (0, -1))[h % 5]
        return (min(max(int(pos[0]) + dx, 0), self.H - 1), min(max(int(pos[1]) + dy, 0), self.W - 1))

    def work(self, agent: int, step: int) -> int:
        h1, h2, h3 = (agent_draw(self.seed, agent, step, k) for k in (1, 2, 3))
        if (h1 >> 11) * 2.0 ** -53 < self.p_idle:
            return 0
        # Box-Muller on two 53-bit uniforms
        u1 = ((h2 >> 11) + 1) * 2.0 ** -53
        u2 = (h3 >> 11) * 2.0 ** -53
        z = math.sqrt(-2.0 * math.log(u1)) * math.cos(2.0 * math.pi * u2)
        return max(1, int(round(math.exp(self.sigma * z))))


def run_event_sim(sched, world: SimWorld, workers: int | None = None, on_ack=None):
    """Drive a scheduler (``next()`` -> (cluster, step, members) or None,
    ``ack(cluster, positions)``) on an abstract clock: a cluster takes as long
    as its slowest member's work; at most ``workers`` clusters run at once (None:
    no limit); completions at the same time are acknowledged lowest step first,
    then in hand-out order (the priority ack queue of §3.5).

    Returns (log, makespan); the log lists ("run" | "ack", time, step, members)."""
    import heapq

    pos = [tuple(int(v) for v in p) for p in world.start]
    log, events, t = [], [], 0
    while True:
        while workers is None or len(events) < workers:
            got = sched.next()
            if got is None:
                break
            cid, step, members = got
            dur = max(world.work(a, step) for a in members)
            heapq.heappush(events, (t + dur, step, cid, tuple(members)))
            log.append(("run", t, step, tuple(members)))
        if not events:
            break
        t = events[0][0]
        while events and events[0][0] == t:
            _, step, cid, members = heapq.heappop(events)
            new = [world.move(a, step, pos[a]) for a in members]
            for a, p in zip(members, new):
                pos[a] = p
            sched.ack(cid, new)
            log.append(("ack", t, step, members))
            if on_ack is not None:
                on_ack(sched)
    return log, t
