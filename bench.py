#!/usr/bin/env python3
"""Benchmark of the batched agent-LLM forward pass on one MI355X.

Workload (one step = the whole hot path over one batch): 25 agents call a
Llama-3-8B-shaped decoder (32 layers, d 4096, 32/8 heads of 128, FFN 14336,
vocab 128256, random N(0, 0.02) bf16 weights initialised on the device) with
prompts of lognormal length (median 1200, sigma 0.5, clipped to [256, 4096]);
all prompts are prefilled in one forward (all agents batched; --chunk sets a
smaller per-agent chunk, e.g. 512), then 64 tokens are generated greedily per
agent: the first from the prefill, 63 from batched decode steps (ready batch
B = 25).  KV pages of 16 tokens.

Reported ``value``: decode tokens/s = 25 * 63 * steps / (GPU time of the
decode steps), timed with HIP events on the launch stream.  ``ms_per_step``
is the whole step (prefill + decode).  ``roofline`` is the whole decode step:
its algorithmic bytes (weights, KV read and write, fp32 logits) over the
decode time, against the HBM peak; ``roofline_prefill`` the whole prefill's
algorithmic flops over the prefill time, against the bf16 matrix-core peak.
``roofline_kernel`` is the dominant decode kernel (the gate/up projection
GEMM with the SwiGLU epilogue), whose launches are timed with HIP events
inside the library in one more step of the same work right after the timed
region (an event pair per launch would slow the timed steps by about 3%),
with its HBM traffic from the committed counter summary; ``roofline_prefill_kernel`` the same GEMM during
the first warm-up step's prefill.  ``cpu_baseline`` times the CPU oracle on a
bounded sample.  ``other_workloads`` (skipped with --no-others) holds short
runs of two more configurations in the same process, after the timed region:
the agent-trace decode (1000 agents, 200 ticks, plus the fixed-batch sweep)
and one 70B step at B = 128, each with its own whole-step HBM roofline.

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
METRIC = "decode tokens/s at ready-batch B (8B shape, 1 GPU); % HBM / MFMA roofline"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def run_step(model, prompts, n_new, chunk, torch, step_events=None):
    """Prefill all prompts (chunked, batched), then n_new - 1 decode steps.
    Returns the three HIP events (start, prefill done, decode done); with a
    list ``step_events``, also appends an event after every decode step."""
    n = len(prompts)
    V = model.vocab
    seqs = [model.seq_open() for _ in range(n)]
    tok = torch.empty(n, dtype=torch.int32, device="cuda")
    tok2 = torch.empty_like(tok)
    logits = torch.empty(n, V, dtype=torch.float32, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record()
    off = 0
    while True:
        items = [i for i in range(n) if off < len(prompts[i])]
        if not items:
            break
        nt = torch.empty(len(items), dtype=torch.int32, device="cuda")
        model.prefill_chunk([seqs[i] for i in items], [prompts[i][off:off + chunk] for i in items], None, nt)
        done = [j for j, i in enumerate(items) if off + chunk >= len(prompts[i])]
        if done:
            dst = torch.tensor([items[j] for j in done], dtype=torch.int64, device="cuda")
            src = torch.tensor(done, dtype=torch.int64, device="cuda")
            tok[dst] = nt[src]
        off += chunk
    ev[1].record()
    for _ in range(n_new - 1):
        model.decode_step(seqs, tok, logits, tok2)
        tok, tok2 = tok2, tok
        if step_events is not None:
            step_events.append(torch.cuda.Event(enable_timing=True))
            step_events[-1].record()
    ev[2].record()
    for s in seqs:
        model.seq_close(s)
    return ev


def cpu_baseline(seed: int) -> dict:
    """The oracle (plain float64 numpy) on a bounded sample of the workload:
    one agent, Llama-3-8B widths with 2 of the 32 layers and the full LM head,
    a 256-token prompt (the workload's shortest) prefilled, then 4 decode
    tokens.  Per-token decode time is scaled to 32 layers:
    t = 16 * t(2 layers) + t(head)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import LlamaShape, OracleModel
    from paper_2411_03519_amd import synth

    shape = synth.with_layers(synth.LLAMA3_8B, 2)
    t0 = time.time()
    w = synth.llama_weights(shape, seed)
    om = OracleModel(LlamaShape(**shape), w)
    del w
    log(f"cpu baseline: weights ready in {time.time() - t0:.1f}s")
    rng = np.random.default_rng(seed)
    prompt = rng.integers(0, shape["vocab"], 256)
    c_full, c_layers = om.new_cache(), om.new_cache()
    t = time.perf_counter()
    om.prefill(c_full, prompt)
    t_prefill = time.perf_counter() - t
    om.hidden_layers(c_layers, prompt, 2)
    feed = rng.integers(0, shape["vocab"], 4)
    t = time.perf_counter()
    for x in feed:
        om.forward(c_full, [int(x)])
    t_fwd = (time.perf_counter() - t) / len(feed)
    t = time.perf_counter()
    for x in feed:
        om.hidden_layers(c_layers, [int(x)], 2)
    t_layers = (time.perf_counter() - t) / len(feed)
    t_head = max(t_fwd - t_layers, 0.0)
    per_token = 16 * t_layers + t_head
    threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    prefill_per_token = (16 * t_prefill) / len(prompt)  # head cost of one row is negligible here
    log(f"cpu baseline: 2-layer decode {t_layers * 1e3:.1f} ms, head {t_head * 1e3:.1f} ms, "
        f"prefill {t_prefill:.2f}s, total {time.time() - t0:.1f}s")
    return {"value": 1.0 / per_token, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "1 agent at Llama-3-8B widths, 2 of 32 layers + LM head, 256-token prompt then 4 decode "
                      "tokens, float64 numpy; decode time per token scaled to 32 layers "
                      "(16 x t(2 layers) + t(head)); the oracle serves agents one after another",
            "prefill_tokens_per_s_scaled": 1.0 / prefill_per_token,
            "host_cpu_count": os.cpu_count()}


# Sources of the decode gate/up kernel: its HBM traffic (rocprofv3 FETCH_SIZE /
# WRITE_SIZE, scaled by a copy of known size) is read from the committed
# profile summary only while these files are unchanged since the counters were
# taken.
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_gate_up_decode_8b_b25_traffic.txt")
KERNEL_SOURCES = ["paper_2411_03519_amd/csrc/kernels/gemm.hip", "paper_2411_03519_amd/csrc/kernels/common.h"]


def kernel_source_hash() -> str:
    return source_hash(KERNEL_SOURCES)


# The whole decode step's HBM traffic (the same counters summed over every
# kernel of the 63 decode steps of one c1 step) depends on every kernel and on
# the launch sequence.
STEP_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_step_8b_b25_traffic.txt")
STEP_SOURCES = KERNEL_SOURCES + ["paper_2411_03519_amd/csrc/kernels/attention.hip",
                                 "paper_2411_03519_amd/csrc/kernels/elementwise.hip",
                                 "paper_2411_03519_amd/csrc/kernels/kernels.h",
                                 "paper_2411_03519_amd/csrc/runtime.hip"]


def code_only(text: str) -> str:
    """C/C++/HIP source without its comments and with every run of white
    space made one blank: what the compiler sees of it, so that an edit of a
    comment does not mark a measurement of the code stale.  String and
    character literals are kept as they are."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_hash(sources=None) -> str:
    """sha256 over the code (code_only) of the listed sources, in order."""
    import hashlib
    h = hashlib.sha256()
    for rel in sources or KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(code_only(f.read()).encode())
        h.update(b"\0")
    return h.hexdigest()


def measured_traffic(summary=None, sources=None, key="traffic_bytes_per_launch"):
    """HBM bytes from a committed profile summary (default: per launch of the
    decode gate/up GEMM), or None if there is none or its sources changed
    since the counters were taken."""
    try:
        with open(summary or TRAFFIC_SUMMARY) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith(" "))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_sha256") != source_hash(sources):
        return None
    try:
        return int(float(kv[key]))
    except (KeyError, ValueError):
        return None


def calibrate_copy(torch):
    """A device-to-device copy of known size, run under rocprofv3 --pmc to turn
    FETCH_SIZE / WRITE_SIZE readings into bytes."""
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "copies": 3}), flush=True)


# ---------------------------------------------------------------------------
# Algorithmic work of the Llama forward (bf16 weights and KV, fp32 logits)
# ---------------------------------------------------------------------------

def layer_params(shape) -> int:
    d, F, hd = shape["d_model"], shape["ffn_dim"], shape["head_dim"]
    q, kv = shape["n_heads"] * hd, shape["n_kv_heads"] * hd
    return (q + 2 * kv) * d + d * q + 2 * F * d + d * F


def decode_weight_bytes(shape) -> int:
    """Weight bytes one decode step streams: every layer's projections and the
    LM head (the embedding is a gather of B rows, norms are negligible)."""
    return 2 * (shape["n_layers"] * layer_params(shape) + shape["vocab"] * shape["d_model"])


def kv_token_bytes(shape) -> int:
    return 2 * 2 * shape["n_kv_heads"] * shape["head_dim"] * shape["n_layers"]


def decode_step_bytes(shape, ctx_lens) -> int:
    """Weights + KV read of every row's context + KV write of the new token +
    fp32 logits, for one decode step over rows with these context lengths."""
    B = len(ctx_lens)
    return (decode_weight_bytes(shape) + (int(sum(ctx_lens)) + B) * kv_token_bytes(shape)
            + B * shape["vocab"] * 4)


def prefill_flops(shape, positions_per_item, logit_rows) -> float:
    """Linear layers per token + causal attention per (query, visible key) +
    the LM head for the rows that return logits."""
    L, hd, nq = shape["n_layers"], shape["head_dim"], shape["n_heads"]
    tokens = sum(len(p) for p in positions_per_item)
    keys = sum(int(np.sum(np.asarray(p, np.int64) + 1)) for p in positions_per_item)
    return (2.0 * L * layer_params(shape) * tokens + 4.0 * L * nq * hd * keys
            + 2.0 * logit_rows * shape["vocab"] * shape["d_model"])


def prefill_all(model, seqs, prompts, chunk, group, torch, next_tok=None):
    """Chunked prefill of prompts[i] into seqs[i], ``group`` items per call;
    the greedy token of each finished item goes to next_tok[i] (device)."""
    for g0 in range(0, len(seqs), group):
        idx = list(range(g0, min(len(seqs), g0 + group)))
        off = 0
        while True:
            items = [i for i in idx if off < len(prompts[i])]
            if not items:
                break
            nt = torch.empty(len(items), dtype=torch.int32, device="cuda")
            model.prefill_chunk([seqs[i] for i in items], [prompts[i][off:off + chunk] for i in items], None, nt)
            done = [j for j, i in enumerate(items) if off + chunk >= len(prompts[i])]
            if done and next_tok is not None:
                dst = torch.tensor([items[j] for j in done], dtype=torch.int64, device="cuda")
                next_tok[dst] = nt[torch.tensor(done, dtype=torch.int64, device="cuda")]
            off += chunk


def hbm_roofline(bytes_total, seconds, what):
    achieved = bytes_total / seconds / 1e9
    return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": what}


def sched_trace_batches(metro, synth, seed, n_agents=1000, ticks=200):
    """Ready batches of the agent trace with the readiness of the library's
    out-of-order scheduler (the rules of §3.3: coupled clusters, a blocking
    radius that grows with the step gap; radius_p 4, max_vel 1, Chebyshev)
    instead of the constant radius 5: on the seeded world of SimWorld, each
    tick hands out every ready cluster, decodes one token for every member
    with budget left (a busy step's budget is its work in tokens), and
    acknowledges a cluster with its members' moves once all budgets are
    spent."""
    world = synth.SimWorld(seed, n_agents, grid=(100, 140))
    sched = metro.Scheduler(world.start, 4.0, 1.0, metro.DIST_CHEBYSHEV, target_step=10 ** 6)
    pos = [tuple(int(v) for v in p) for p in world.start]
    budget = {}       # agent -> tokens left in its current step
    cluster_of = {}   # cluster -> (step, members)
    batches = []

    def ack(cid):
        step, members = cluster_of.pop(cid)
        new = [world.move(a, step, pos[a]) for a in members]
        for a, p in zip(members, new):
            pos[a] = p
        sched.ack(cid, new)

    for _ in range(ticks):
        while True:                      # hand out; idle clusters finish at once
            got = sched.next()
            if got is None:
                break
            cid, step, members = got
            cluster_of[cid] = (step, members)
            for a in members:
                budget[a] = world.work(a, step)
            if all(budget[a] == 0 for a in members):
                ack(cid)
        run = np.array(sorted(a for a, b in budget.items() if b > 0), np.int64)
        batches.append(run)
        for a in run:
            budget[a] -= 1
        for cid in [c for c, (_, m) in cluster_of.items() if all(budget[a] == 0 for a in m)]:
            ack(cid)
    return batches


def bench_trace(args, torch, metro, synth):
    """Decode driven by the seeded agent trace: 1000 agents with lognormal
    (median 1500) starting contexts, prefilled before timing; each of 200 ticks
    decodes one token for every ready agent (ready batches of ~50..800); then a
    fixed-batch sweep over agents 0..B-1.  ``--trace-rule sched`` takes the
    ready batches from the library's scheduler (sched_trace_batches)."""
    shape = synth.LLAMA3_8B
    V = shape["vocab"]
    ctx = synth.trace_start_contexts(args.seed)
    n = len(ctx)
    if args.trace_rule == "sched":
        batches = [b for b in sched_trace_batches(metro, synth, args.seed, n) if len(b)]
    else:
        batches = [b for b in synth.agent_trace(args.seed) if len(b)]
    sweep, sweep_steps = [50, 100, 200, 400, 800], 3
    lens = np.array([len(c) for c in ctx], np.int64)
    extra = np.zeros(n, np.int64)
    for b in batches:
        extra[b] += 1
    extra[:max(sweep)] += (1 + sweep_steps) * len(sweep)
    page_bytes = 16 * kv_token_bytes(shape)
    pages = int(np.sum((lens + extra + 15) // 16)) + 64
    log(f"trace: {n} agents, {lens.sum()} context tokens, {len(batches)} ticks, "
        f"{sum(len(b) for b in batches)} decode tokens; KV pool {pages * page_bytes / 1e9:.1f} GB")
    model = metro.Model(shape, max_batch=n, max_tokens=32 * 512, max_context=int((lens + extra).max()) + 16,
                        max_seqs=n + 8, kv_pool_bytes=pages * page_bytes, seed=args.seed)
    seqs = np.array([model.seq_open() for _ in range(n)], np.int64)
    last = torch.zeros(n, dtype=torch.int32, device="cuda")
    t0 = time.time()
    prefill_all(model, list(seqs), ctx, 512, 32, torch, last)
    torch.cuda.synchronize()
    log(f"trace: contexts prefilled in {time.time() - t0:.1f}s")
    logits = torch.empty(n, V, dtype=torch.float32, device="cuda")
    nxt = torch.empty(n, dtype=torch.int32, device="cuda")
    cur = lens.copy()

    def timed_step(rows):
        """One decode step over agent ids ``rows``; returns (GPU ms, algorithmic bytes)."""
        B = len(rows)
        idx = torch.from_numpy(rows).cuda()
        tok = last[idx]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        model.decode_step(seqs[rows], tok, logits[:B], nxt[:B])
        e1.record()
        last[idx] = nxt[:B]
        nbytes = decode_step_bytes(shape, cur[rows])
        cur[rows] += 1
        return e0, e1, nbytes

    recs = [timed_step(b) for b in batches]
    torch.cuda.synchronize()
    ms = [a.elapsed_time(b) for a, b, _ in recs]
    tokens = sum(len(b) for b in batches)
    value = tokens / (sum(ms) / 1e3)
    roof = hbm_roofline(sum(r[2] for r in recs), sum(ms) / 1e3, "whole decode step (weights + KV + logits)")
    sizes = np.array([len(b) for b in batches])
    log(f"trace: {tokens} tokens in {sum(ms):.1f} ms GPU time -> {value:.0f} tok/s, "
        f"{roof['frac'] * 100:.1f}% of HBM peak")
    fixed = {}
    for B in sweep:
        rows = np.arange(B, dtype=np.int64)
        timed_step(rows)
        r = [timed_step(rows) for _ in range(sweep_steps)]
        torch.cuda.synchronize()
        t = sum(a.elapsed_time(b) for a, b, _ in r) / 1e3
        fixed[str(B)] = {"tokens_per_s": round(B * sweep_steps / t, 1),
                         "hbm_frac": round(sum(x[2] for x in r) / t / 1e9 / HBM_PEAK_GBS, 4),
                         "ms_per_step": round(t * 1e3 / sweep_steps, 3)}
        log(f"trace sweep B={B}: {fixed[str(B)]}")
    model.close()
    return {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": 1, "warmup": 0,
            "ms_per_step": round(sum(ms), 2), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic: seeded agent trace and token ids, random N(0,0.02) bf16 weights",
            "config": {"workload": "Llama-3-8B-shaped decoder driven by a seeded agent trace: 1000 agents on a "
                                   "100x140 grid, 200 ticks, readiness "
                                   + ("of the out-of-order scheduler (rules of §3.3, radius_p 4, max_vel 1)"
                                      if args.trace_rule == "sched" else "Chebyshev radius 5")
                                   + "; contexts lognormal(median 1500) clipped to [256,4096], prefilled before "
                                     "timing",
                       "ticks": len(batches), "decode_tokens": tokens, "batch_min": int(sizes.min()),
                       "batch_median": float(np.median(sizes)), "batch_max": int(sizes.max()),
                       "context_tokens": int(lens.sum())},
            "roofline": roof, "fixed_batch": fixed,
            "batch_histogram": {f"{lo}-{hi - 1}": int(np.sum((sizes >= lo) & (sizes < hi)))
                                for lo, hi in ((1, 64), (64, 128), (128, 256), (256, 512), (512, 1024))},
            "tick_ms": {"p50": round(float(np.percentile(ms, 50)), 3), "p90": round(float(np.percentile(ms, 90)), 3),
                        "max": round(float(np.max(ms)), 3)}}


def sched_chain(world, seed, step, agent, vocab, max_calls):
    """The LLM calls of one agent step, issued one after another (an agent
    step of the paper's simulation chains calls such as perceive, plan and
    react): none for an idle step, else min(work, max_calls) calls, each a
    prompt of lognormal(median 640, sigma 0.5) tokens clipped to [128, 2048]
    and lognormal(median 18, sigma 0.6) outputs clipped to [4, 64] (the
    paper's calls average 642.6 tokens in and 21.9 out, §4.2)."""
    work = world.work(agent, step)
    calls = []
    for k in range(min(work, max_calls)):
        rng = np.random.Generator(np.random.PCG64([seed, 11, agent, step, k]))
        plen = int(np.clip(np.rint(np.exp(rng.normal(np.log(640.0), 0.5))), 128, 2048))
        n_out = int(np.clip(np.rint(np.exp(rng.normal(np.log(18.0), 0.6))), 4, 64))
        calls.append((rng.integers(0, vocab, size=plen, dtype=np.int64), n_out))
    return calls


def run_engine_loop(model, metro, sched, world, seed, shape, torch, max_items, max_tokens=8192, chunk=512,
                    priority=True, max_calls=4):
    """Closed loop of the scheduler (metro_sched_*) and the library's mixed
    continuous batching (metro_engine_*): every ready cluster is handed out;
    each member submits the first call of its step's chain, tagged with its
    step; each finished call submits the next; a cluster is acknowledged, with
    its agents' moves, once every member's chain is done.  One engine step is
    one forward.  Returns wall seconds, token counts and the achieved
    parallelism (outstanding requests averaged over the run, §4.2)."""
    V = shape["vocab"]
    eng = metro.Engine(model, max_tokens=max_tokens, chunk=chunk, max_items=max_items, priority=priority)
    pos = [tuple(int(v) for v in p) for p in world.start]
    clusters = {}      # cluster -> [step, members, chains still running]
    chains = {}        # request id -> (cluster, agent, step, calls still to issue)
    stats = {"forwards": 0, "agent_steps": 0, "calls": 0}
    next_id = [0]
    area = 0.0

    def submit(cid, agent, step, calls):
        rid = next_id[0]
        next_id[0] += 1
        prompt, n_out = calls[0]
        eng.submit(rid, step, prompt, n_out)
        chains[rid] = (cid, agent, step, calls[1:])
        stats["calls"] += 1

    def finish(cid):
        step, members, _ = clusters.pop(cid)
        new = [world.move(a, step, pos[a]) for a in members]
        for a, p in zip(members, new):
            pos[a] = p
        sched.ack(cid, new)
        stats["agent_steps"] += len(members)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while True:
        while True:
            got = sched.next()
            if got is None:
                break
            cid, step, members = got
            work = [(a, sched_chain(world, seed, step, a, V, max_calls)) for a in members]
            work = [(a, c) for a, c in work if c]
            clusters[cid] = [step, members, len(work)]
            if not work:
                finish(cid)
                continue
            for a, calls in work:
                submit(cid, a, step, calls)
        if not chains:
            break
        outstanding = len(chains)
        t1 = time.perf_counter()
        eng.step()
        area += outstanding * (time.perf_counter() - t1)
        stats["forwards"] += 1
        for rid in eng.finished():
            eng.result(rid)
            cid, agent, step, rest = chains.pop(rid)
            if rest:
                submit(cid, agent, step, rest)
                continue
            cl = clusters[cid]
            cl[2] -= 1
            if cl[2] == 0:
                finish(cid)
    torch.cuda.synchronize()
    stats["seconds"] = time.perf_counter() - t0
    es = eng.stats()
    eng.close()
    # output tokens: one per decode item plus each call's first token (from its last prompt chunk)
    stats.update(prompt_tokens=es["prompt_tokens"], decode_tokens=es["decode_tokens"] + stats["calls"],
                 items=es["items"])
    stats["achieved_parallelism"] = area / stats["seconds"]
    return stats


def bench_sched(args, torch, metro, synth):
    """The out-of-order scheduler (Algorithm 3) in closed loop with the
    library's mixed continuous batching, against the parallel-sync baseline
    (Algorithm 1) on the same seeded world and calls (100 x 140 grid, radius_p
    4, max_vel 1, chains of up to 4 calls per busy agent step), with step
    priority on and off: by default 25 agents for 12 steps (the paper's
    village size), 200 agents for 3 steps and 500 agents for 2 (--sched-cases;
    --sched-priority on skips the runs without priority).  ``value`` is the
    second case (or the only one), out of order, with priority."""
    shape = synth.LLAMA3_8B
    cases = [tuple(int(v) for v in c.split("x")) for c in args.sched_cases.split(",")]
    priorities = (True, False) if args.sched_priority == "both" else (True,)
    max_items = 256
    pages = 640 * ((2048 + 64 + 15) // 16 + 1) + 64
    model = metro.Model(shape, max_batch=max_items, max_tokens=8192 + max_items, max_context=2048 + 64 + 16,
                        max_seqs=1024, kv_pool_bytes=pages * 16 * kv_token_bytes(shape), seed=args.seed)
    warm = synth.SimWorld(args.seed + 1, 8)
    run_engine_loop(model, metro, metro.Scheduler(warm.start, 4.0, 1.0, target_step=1), warm, args.seed, shape,
                    torch, max_items)
    out = {}
    for n_agents, steps in cases:
        world = synth.SimWorld(args.seed, n_agents, grid=(100, 140))
        res = {}
        for priority in priorities:
            pol = "priority" if priority else "no_priority"
            for mode in ("parallel_sync", "out_of_order"):
                sched = metro.Scheduler(world.start, 4.0, 1.0, metro.DIST_CHEBYSHEV, steps,
                                        sync=mode == "parallel_sync")
                st = run_engine_loop(model, metro, sched, world, args.seed, shape, torch, max_items,
                                     priority=priority, max_calls=args.max_calls)
                st["seconds"] = round(st["seconds"], 3)
                st["achieved_parallelism"] = round(st["achieved_parallelism"], 2)
                st["tokens_per_s"] = round((st["prompt_tokens"] + st["decode_tokens"]) / st["seconds"], 1)
                st["mean_items"] = round(st["items"] / max(1, st["forwards"]), 1)
                res[f"{mode}/{pol}"] = st
                log(f"sched {n_agents} agents x {steps} steps, {mode}, {pol}: {st}")
            res[f"speedup_vs_parallel_sync/{pol}"] = round(
                res[f"parallel_sync/{pol}"]["seconds"] / res[f"out_of_order/{pol}"]["seconds"], 3)
        out[f"{n_agents}x{steps}"] = res
    model.close()
    head_case = "%dx%d" % cases[1 if len(cases) > 1 else 0]
    head = out[head_case]["out_of_order/priority"]
    flops = 2.0 * shape["n_layers"] * layer_params(shape) * (head["prompt_tokens"] + head["decode_tokens"])
    roof = {"bound": "mfma", "achieved": round(flops / head["seconds"] / 1e12, 1), "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(flops / head["seconds"] / 1e12 / BF16_PEAK_TFLOPS, 4), "traffic": None,
            "kernel": "whole closed loop, linear-layer flops of every prefill and decode token over wall time"}
    return {"metric": "simulation tokens/s (prefill + decode, wall clock) under the out-of-order scheduler",
            "value": head["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": 1, "warmup": 1,
            "ms_per_step": round(head["seconds"] * 1e3, 1), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic: seeded world (SplitMix64 moves and work), prompt ids and random N(0,0.02) weights",
            "config": {"workload": f"Llama-3-8B-shaped decoder serving agents on a 100x140 grid: chains of up to "
                                   f"{args.max_calls} LLM calls per busy agent step (prompts lognormal median 640, outputs median "
                                   "18), radius_p 4, max_vel 1, Chebyshev distance; library mixed continuous "
                                   "batching (8192-token forwards, 512-token chunks) with step priority on/off; "
                                   f"value: {head_case.replace('x', ' agents x ')} steps, out of order, priority",
                       "cases": [f"{n}x{s}" for n, s in cases]},
            "speedup_vs_parallel_sync": out[head_case]["speedup_vs_parallel_sync/priority"],
            "cases": out, "roofline": roof}


def run_call_round(model, calls, outs, torch, use_cache, chunk=512):
    """One round of agent calls as one batch: each call opens its sequence
    (through the prefix cache when on), the uncached rest of every prompt is
    prefilled in 512-token chunks, then decode steps run until each call has
    its output length (finished calls leave the batch).  Returns (cached
    prompt tokens, computed prompt tokens, decode tokens)."""
    n = len(calls)
    seqs, ks = [], []
    for p in calls:
        if use_cache:
            sq, k = model.seq_open_cached(p)
        else:
            sq, k = model.seq_open(), 0
        seqs.append(sq)
        ks.append(k)
    tok = torch.zeros(n, dtype=torch.int32, device="cuda")
    prefill_all(model, seqs, [p[k:] for p, k in zip(calls, ks)], chunk, n, torch, tok)
    left = np.asarray(outs, np.int64) - 1
    active = [i for i in range(n) if left[i] > 0]
    n_dec = 0
    while active:
        idx = torch.tensor(active, dtype=torch.int64, device="cuda")
        nt = torch.empty(len(active), dtype=torch.int32, device="cuda")
        model.decode_step([seqs[i] for i in active], tok[idx].contiguous(), None, nt)
        tok[idx] = nt
        n_dec += len(active)
        left[active] -= 1
        active = [i for i in active if left[i] > 0]
    for sq in seqs:
        model.seq_close(sq)
    return sum(ks), sum(len(p) - k for p, k in zip(calls, ks)), n_dec


def bench_apc(args, torch, metro, synth):
    """Automatic prefix caching on successive agent calls: 25 agents, 8 rounds
    of one call each (prompts: a 256-token preamble shared by all, a 192-token
    persona per agent, a fresh observation lognormal median 160; outputs
    lognormal median 18 -- about 640 prompt and 22 output tokens per call),
    each round run as one batch, with the prefix cache off and on."""
    shape = synth.LLAMA3_8B
    n, rounds = 25, 8
    prompts, outs = synth.agent_call_prompts(args.seed, n, rounds, shape["vocab"])
    warm_p, warm_o = synth.agent_call_prompts(args.seed + 1, n, 1, shape["vocab"])
    max_ctx = max(len(p) for r in prompts + warm_p for p in r) + 80
    pages = 16384
    model = metro.Model(shape, max_batch=n, max_tokens=n * 512, max_context=max_ctx, max_seqs=n + 8,
                        kv_pool_bytes=pages * 16 * kv_token_bytes(shape), seed=args.seed)
    run_call_round(model, warm_p[0], warm_o[0], torch, False)
    res = {}
    for mode in ("off", "on"):
        model.prefix_cache(0)
        if mode == "on":
            model.prefix_cache(pages)
        times, cached, computed, dec = [], 0, 0, 0
        for r in range(rounds):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            c, p, d = run_call_round(model, prompts[r], outs[r], torch, mode == "on")
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
            cached, computed, dec = cached + c, computed + p, dec + d + n
        total = sum(len(p) for r in prompts for p in r) + int(sum(np.sum(o) for o in outs))
        res[mode] = {"seconds": round(sum(times), 3), "round_ms": [round(t * 1e3, 1) for t in times],
                     "cached_prompt_tokens": cached, "computed_prompt_tokens": computed,
                     "output_tokens": dec, "tokens_per_s": round(total / sum(times), 1),
                     "steady_tokens_per_s": round(total * (rounds - 1) / rounds / sum(times[1:]), 1)}
        if mode == "on":
            res[mode]["cache"] = model.prefix_cache_stats()
        log(f"apc {mode}: {res[mode]}")
    model.close()
    on, off = res["on"], res["off"]
    gain = off["seconds"] / on["seconds"]
    flops = 2.0 * shape["n_layers"] * layer_params(shape) * (on["computed_prompt_tokens"] + on["output_tokens"])
    roof = {"bound": "mfma", "achieved": round(flops / on["seconds"] / 1e12, 1), "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(flops / on["seconds"] / 1e12 / BF16_PEAK_TFLOPS, 4), "traffic": None,
            "kernel": "all rounds with the cache on, linear-layer flops of computed prompt and output tokens "
                      "over wall time"}
    return {"metric": "agent-call throughput (prompt + output tokens/s, wall clock) with automatic prefix caching",
            "value": on["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": rounds, "warmup": 1,
            "ms_per_step": round(on["seconds"] / rounds * 1e3, 1), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic: seeded prompt ids (shared preamble, per-agent persona, fresh observation), random "
                    "N(0,0.02) bf16 weights",
            "config": {"workload": "Llama-3-8B-shaped decoder, 25 agents x 8 rounds of one call each, one batch per "
                                   "round; prompts = 256-token shared preamble + 192-token persona per agent + "
                                   "observation lognormal(median 160, sigma 0.6) in [16,1024]; outputs "
                                   "lognormal(median 18, sigma 0.6) in [4,64]; chunked prefill 512",
                       "agents": n, "rounds": rounds},
            "gain_vs_no_cache": round(gain, 3), "modes": res, "roofline": roof}


def bench_prefix(args, torch, metro, synth):
    """Prefix-heavy requests: a 1024-token prefix prefilled once and forked by
    page reference into 64 requests, their suffixes (512..2048 tokens)
    prefilled in 512-token chunks, then 31 decode steps at B = 64."""
    shape = synth.LLAMA3_8B
    V = shape["vocab"]
    prefix, suffixes, n_new = synth.prefix_heavy_batch(args.seed)
    n = len(suffixes)
    slen = np.array([len(s) for s in suffixes], np.int64)
    page_bytes = 16 * kv_token_bytes(shape)
    pages = 64 + int(np.sum((slen + n_new + 15) // 16)) + n + 64
    model = metro.Model(shape, max_batch=n, max_tokens=n * 512, max_context=1024 + int(slen.max()) + n_new + 16,
                        max_seqs=2 * n + 8, kv_pool_bytes=pages * page_bytes, seed=args.seed)
    positions = [np.arange(len(prefix))] + [np.arange(len(prefix), len(prefix) + L) for L in slen]
    flops = prefill_flops(shape, positions, 2 + n)
    tok = torch.zeros(n, dtype=torch.int32, device="cuda")
    tok2 = torch.empty_like(tok)
    logits = torch.empty(n, V, dtype=torch.float32, device="cuda")

    def step():
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record()
        base = model.seq_open()
        prefill_all(model, [base], [prefix], 512, 1, torch)
        forks = [model.seq_fork(base, len(prefix)) for _ in range(n)]
        model.seq_close(base)
        prefill_all(model, forks, suffixes, 512, n, torch, tok)
        ev[1].record()
        cur = [tok, tok2]
        for _ in range(n_new - 1):
            model.decode_step(forks, cur[0], logits, cur[1])
            cur.reverse()
        ev[2].record()
        for f in forks:
            model.seq_close(f)
        return ev

    for _ in range(args.warmup):
        step()
    evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    pre = sum(e[0].elapsed_time(e[1]) for e in evs) / 1e3
    dec = sum(e[1].elapsed_time(e[2]) for e in evs) / 1e3
    unique = len(prefix) + int(slen.sum())
    tflops = flops * args.steps / pre / 1e12
    value = n * (n_new - 1) * args.steps / dec
    log(f"prefix: prefill {pre / args.steps * 1e3:.1f} ms/step ({unique * args.steps / pre:.0f} tok/s, "
        f"{tflops:.0f} TFLOP/s), decode {dec / args.steps * 1e3:.1f} ms/step ({value:.0f} tok/s)")
    model.close()
    return {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round((pre + dec) / args.steps * 1e3, 2), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic: seeded token ids, random N(0,0.02) bf16 weights",
            "config": {"workload": "Llama-3-8B-shaped decoder, 64 requests sharing a 1024-token prefix (prefilled "
                                   "once, forked by page reference) plus suffixes uniform in [512,2048], chunked "
                                   "prefill 512, 32 greedy tokens each",
                       "requests": n, "unique_prefill_tokens": unique, "decode_steps": n_new - 1,
                       "ready_batch": n},
            "prefill_tokens_per_s": round(unique * args.steps / pre, 1),
            "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tflops / BF16_PEAK_TFLOPS, 4), "traffic": None,
                         "kernel": "whole prefill (linear layers + causal attention + LM head rows)"},
            "decode_hbm_frac": round(sum(decode_step_bytes(shape, slen + 1024 + k) for k in range(n_new - 1))
                                     * args.steps / dec / 1e9 / HBM_PEAK_GBS, 4)}


def bench_70b(args, torch, metro, synth):
    """Llama-3-70B shape unsharded on one GPU: 128 agents with contexts uniform
    in [1024, 3072] prefilled before timing; each timed step forks the 128
    sequences (prefix sharing, outside the timed region) and decodes 31 tokens
    at B = 128."""
    shape = synth.LLAMA3_70B
    V = shape["vocab"]
    ctx, n_new = synth.llama70b_agent_batch(args.seed)
    n = len(ctx)
    lens = np.array([len(c) for c in ctx], np.int64)
    page_bytes = 16 * kv_token_bytes(shape)
    runs = args.steps + args.warmup
    pages = int(np.sum((lens + 15) // 16)) + runs * n * (2 + (n_new + 15) // 16) + 64
    log(f"70b: {n} agents, {lens.sum()} context tokens; KV pool {pages * page_bytes / 1e9:.1f} GB")
    t0 = time.time()
    model = metro.Model(shape, max_batch=n, max_tokens=16 * 512, max_context=int(lens.max()) + n_new + 16,
                        max_seqs=2 * n + 8, kv_pool_bytes=pages * page_bytes, seed=args.seed)
    info = model.info()
    log(f"70b: model ready in {time.time() - t0:.1f}s, weights {info.weight_bytes / 1e9:.1f} GB")
    seqs = [model.seq_open() for _ in range(n)]
    first = torch.zeros(n, dtype=torch.int32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    prefill_all(model, seqs, ctx, 512, 16, torch, first)
    e1.record()
    torch.cuda.synchronize()
    pre_s = e0.elapsed_time(e1) / 1e3
    log(f"70b: contexts prefilled in {pre_s:.1f}s GPU time ({lens.sum() / pre_s:.0f} tok/s)")
    logits = torch.empty(n, V, dtype=torch.float32, device="cuda")

    def step():
        forks = [model.seq_fork(s, int(L)) for s, L in zip(seqs, lens)]
        tok, tok2 = first.clone(), torch.empty_like(first)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(n_new - 1):
            model.decode_step(forks, tok, logits, tok2)
            tok, tok2 = tok2, tok
        ev[1].record()
        torch.cuda.synchronize()
        for f in forks:
            model.seq_close(f)
        return ev[0].elapsed_time(ev[1]) / 1e3

    for _ in range(args.warmup):
        step()
    dec = sum(step() for _ in range(args.steps))
    value = n * (n_new - 1) * args.steps / dec
    nbytes = sum(decode_step_bytes(shape, lens + k) for k in range(n_new - 1)) * args.steps
    roof = hbm_roofline(nbytes, dec, "whole decode step (weights + KV + logits)")
    log(f"70b: decode {dec / args.steps * 1e3:.1f} ms per 31 steps ({value:.0f} tok/s), "
        f"{roof['frac'] * 100:.1f}% of HBM peak")
    model.close()
    flops = prefill_flops(shape, [np.arange(L) for L in lens], n)
    return {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(dec / args.steps * 1e3, 2), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic: seeded token ids, random N(0,0.02) bf16 weights",
            "config": {"workload": "Llama-3-70B-shaped decoder unsharded on one GPU, 128 agents with contexts "
                                   "uniform in [1024,3072] (prefilled before timing), 32 greedy tokens each",
                       "agents": n, "context_tokens": int(lens.sum()), "decode_steps": n_new - 1,
                       "ready_batch": n},
            "roofline": roof,
            "prefill_tokens_per_s": round(lens.sum() / pre_s, 1),
            "prefill_mfma_frac": round(flops / pre_s / 1e12 / BF16_PEAK_TFLOPS, 4)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--agents", type=int, default=25)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", choices=["agents", "trace", "prefix", "70b", "sched", "apc"], default="agents",
                    help="agents (default): 25 agents, the benchmarked workload; trace: decode driven by the "
                         "seeded agent trace; prefix: prefix-heavy requests; 70b: Llama-3-70B shape at B=128; "
                         "sched: the out-of-order scheduler in closed loop with the engine vs parallel-sync")
    ap.add_argument("--chunk", type=int, default=4096,
                    help="agents workload: prompt tokens of one agent per prefill call (4096: whole prompts)")
    ap.add_argument("--max-calls", type=int, default=4,
                    help="sched workload: longest chain of LLM calls in one busy agent step")
    ap.add_argument("--sched-cases", default="25x12,200x3,500x2",
                    help="sched workload: agents x steps of each closed-loop run, comma separated")
    ap.add_argument("--sched-priority", choices=["both", "on"], default="both",
                    help="sched workload: run with step priority on and off, or on only")
    ap.add_argument("--trace-rule", choices=["radius5", "sched"], default="radius5",
                    help="trace workload: ready batches from the constant Chebyshev-5 readiness rule (default) or "
                         "from the library's out-of-order scheduler with the rules of §3.3")
    ap.add_argument("--no-others", action="store_true",
                    help="agents workload: skip the short agent-trace and 70B runs reported under other_workloads")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy three times (counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one MI355X: the path is data-parallel over agents with no per-step collective, "
              "so each GPU would run this same single-GPU workload; --gpus must be 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2411_03519_amd import metro, synth

    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        calibrate_copy(torch)
        return
    if args.workload != "agents":
        fn = {"trace": bench_trace, "prefix": bench_prefix, "70b": bench_70b, "sched": bench_sched,
              "apc": bench_apc}[args.workload]
        print(json.dumps(fn(args, torch, metro, synth)), flush=True)
        return
    shape = synth.LLAMA3_8B
    prompts, n_new = synth.llama8b_agent_batch(args.seed, n_agents=args.agents)
    n = len(prompts)
    chunk = args.chunk
    lens = np.array([len(p) for p in prompts])
    log(f"workload: {n} agents, prompt tokens {lens.sum()} (min {lens.min()}, max {lens.max()}), "
        f"{n_new} generated each")

    t0 = time.time()
    model = metro.Model(shape, max_batch=max(64, n), max_tokens=int(min(n * chunk, lens.sum())), max_context=4096 + 128,
                        max_seqs=2 * n, kv_pool_bytes=24 << 30, seed=args.seed)
    info = model.info()
    log(f"model ready in {time.time() - t0:.1f}s: weights {info.weight_bytes / 1e9:.2f} GB, "
        f"KV pool {info.kv_pool_bytes / 1e9:.1f} GB ({info.n_pages} pages)")

    # warmup (untimed); the first one also measures the prefill gate/up GEMM
    dstep_ms = None  # decode step times of the first warm-up step (events between steps)
    for w in range(args.warmup):
        if w == 0:
            model.profile_start("gemm_gate_up", "prefill")
        marks = [] if w == 0 else None
        ev = run_step(model, prompts, n_new, chunk, torch, marks)
        torch.cuda.synchronize()
        if w == 0:
            pf_ms, pf_launches = model.profile_stop()
            dstep_ms = np.array([ev[1].elapsed_time(marks[0])] +
                               [a.elapsed_time(b) for a, b in zip(marks[:-1], marks[1:])])
        log(f"warmup {w}: prefill {ev[0].elapsed_time(ev[1]):.1f} ms, decode {ev[1].elapsed_time(ev[2]):.1f} ms")

    # timed region (no per-kernel events inside it: bracketing each gate/up
    # launch with an event pair costs about 4 us per launch, 3% of a step)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    events = [run_step(model, prompts, n_new, chunk, torch) for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    # the dominant kernel's launches, timed in one more step of the same work
    model.profile_start("gemm_gate_up", "decode")
    run_step(model, prompts, n_new, chunk, torch)
    torch.cuda.synchronize()
    gu_ms, gu_launches = model.profile_stop()

    prefill_ms = sum(e[0].elapsed_time(e[1]) for e in events)
    decode_ms = sum(e[1].elapsed_time(e[2]) for e in events)
    step_ms = sum(e[0].elapsed_time(e[2]) for e in events) / args.steps
    decode_tokens = n * (n_new - 1) * args.steps
    value = decode_tokens / (decode_ms / 1e3)
    prefill_tps = lens.sum() * args.steps / (prefill_ms / 1e3)
    log(f"timed: {args.steps} steps, wall {wall:.2f}s, step {step_ms:.1f} ms, prefill {prefill_ms / args.steps:.1f}"
        f" ms/step ({prefill_tps:.0f} tok/s), decode {decode_ms / args.steps:.1f} ms/step ({value:.0f} tok/s)")

    # roofline of the path: the whole decode step (algorithmic bytes of the 63
    # steps, contexts growing by one token per step) and the whole prefill
    step_bytes = sum(decode_step_bytes(shape, lens + k) for k in range(n_new - 1))
    roofline = hbm_roofline(step_bytes * args.steps, decode_ms / 1e3,
                            "whole decode step (weights + KV read and write + fp32 logits)")
    roofline["bytes_per_step"] = int(step_bytes // (n_new - 1))
    roofline["traffic"] = measured_traffic(STEP_TRAFFIC_SUMMARY, STEP_SOURCES, "traffic_bytes_per_step")
    items = sum(-(-int(L) // chunk) for L in lens)      # LM-head rows: one per item of every prefill call
    pf_all_flops = prefill_flops(shape, [np.arange(L) for L in lens], items)
    pf_all_tflops = pf_all_flops * args.steps / (prefill_ms / 1e3) / 1e12
    # roofline of the dominant decode kernel: algorithmic bytes per launch
    d, F = shape["d_model"], shape["ffn_dim"]
    gu_bytes = 2 * F * d * 2 + n * d * 2 + n * F * 2   # W_gate|W_up + h in + SwiGLU out (bf16)
    gu_avg_s = gu_ms / 1e3 / gu_launches
    achieved = gu_bytes / gu_avg_s / 1e9
    roofline_kernel = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                       "kernel": "gemm gate/up + SwiGLU (decode, M=25, N=28672, K=4096); launches timed with "
                                 "event pairs in one step of the same work after the timed region",
                       "bytes_per_launch": gu_bytes, "avg_launch_us": round(gu_avg_s * 1e6, 2),
                       "launches": gu_launches}
    out = {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(step_ms, 2), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic: seeded uniform token ids, random N(0,0.02) bf16 weights",
           "config": {"workload": "Llama-3-8B-shaped decoder, 25 agent requests, prompts lognormal(median 1200, "
                                  "sigma 0.5) clipped to [256,4096], "
                                  + ("all prompts prefilled in one forward" if chunk >= 4096 else
                                     f"chunked prefill {chunk}") + ", 64 greedy tokens each",
                      "agents": n, "prompt_tokens": int(lens.sum()), "decode_steps": n_new - 1,
                      "ready_batch": n, "page_size": 16},
           "roofline": roofline,
           "roofline_prefill": {"bound": "mfma", "achieved": round(pf_all_tflops, 1), "peak": BF16_PEAK_TFLOPS,
                                "unit": "TFLOP/s", "frac": round(pf_all_tflops / BF16_PEAK_TFLOPS, 4),
                                "traffic": None,
                                "kernel": "whole prefill (linear layers + causal attention + LM head rows)",
                                "flops_per_step": pf_all_flops},
           "roofline_kernel": roofline_kernel,
           "targets": {"decode_hbm_frac": 0.60, "prefill_mfma_frac": 0.50},
           "tolerance": {"stated": {"logits_max_abs": 2e-2, "logits_rel_l2": 1e-2, "greedy": "exact"},
                         "note": "met as stated at the tiny shape; at 8B/70B widths no fp32-accumulating "
                                 "evaluation meets 2e-2 max-abs (the oracle's own float32 evaluation misses "
                                 "it), so the bounds there are 1.25x the oracle's float32-vs-float64 spread "
                                 "on the same inputs and greedy choices may differ at fp32-undecidable steps "
                                 "(tests/parity.py)"},
           "decode_ms_per_step": round(decode_ms / args.steps, 2),
           "decode_step_ms": None if dstep_ms is None else {
               "p50": round(float(np.percentile(dstep_ms, 50)), 3), "p90": round(float(np.percentile(dstep_ms, 90)), 3),
               "max": round(float(dstep_ms.max()), 3), "n": int(dstep_ms.size),
               "note": "the 63 decode steps of the first warm-up step, timed between events"},
           "prefill_ms_per_step": round(prefill_ms / args.steps, 2),
           "prefill_tokens_per_s": round(prefill_tps, 1)}
    if args.warmup > 0 and pf_launches:
        pf_flops = 2.0 * 2 * F * d * lens.sum() * shape["n_layers"]
        pf_tflops = pf_flops / (pf_ms / 1e3) / 1e12
        out["roofline_prefill_kernel"] = {"bound": "mfma", "achieved": round(pf_tflops, 1),
                                          "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                          "frac": round(pf_tflops / BF16_PEAK_TFLOPS, 4),
                                          "kernel": "gemm gate/up + SwiGLU (prefill chunks; a split last round "
                                                    "includes its fixup kernel)", "launches": pf_launches}
    model.close()
    if not args.no_others:
        out["other_workloads"] = other_workloads(args, torch, metro, synth)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.seed)
    print(json.dumps(out), flush=True)


def other_workloads(args, torch, metro, synth):
    """The agent-trace decode and one 70B step, after the c1 timed region, so
    that one default run records them too.  A failure in either is reported
    in its entry and does not touch the c1 figures."""
    keep = ("value", "unit", "ms_per_step", "roofline", "fixed_batch", "batch_histogram", "tick_ms",
            "prefill_tokens_per_s", "prefill_mfma_frac")
    res = {}
    for name, fn, over in (("trace", bench_trace, {"trace_rule": "radius5"}),
                           ("70b", bench_70b, {"steps": 1, "warmup": 1})):
        sub = argparse.Namespace(**{**vars(args), **over})
        t0 = time.time()
        try:
            r = fn(sub, torch, metro, synth)
            res[name] = {k: r[k] for k in keep if k in r}
            res[name]["workload"] = r["config"]["workload"]
        except Exception as e:  # reported, not raised: the c1 line stands on its own
            res[name] = {"error": f"{type(e).__name__}: {e}"}
        res[name]["wall_s"] = round(time.time() - t0, 1)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        log(f"other workload {name}: {res[name].get('value', res[name].get('error'))}")
    return res


if __name__ == "__main__":
    main()
