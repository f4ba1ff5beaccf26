#!/usr/bin/env python3
"""Benchmark of the batched agent-LLM forward pass on one MI355X.

Workload (one step = the whole hot path over one batch): 25 agents call a
Llama-3-8B-shaped decoder (32 layers, d 4096, 32/8 heads of 128, FFN 14336,
vocab 128256, random N(0, 0.02) bf16 weights initialised on the device) with
prompts of lognormal length (median 1200, sigma 0.5, clipped to [256, 4096]);
the prompts are prefilled in 512-token chunks (all agents batched per call),
then 64 tokens are generated greedily per agent: the first from the prefill,
63 from batched decode steps (ready batch B = 25).  KV pages of 16 tokens.

Reported ``value``: decode tokens/s = 25 * 63 * steps / (GPU time of the
decode steps), timed with HIP events on the launch stream.  ``ms_per_step``
is the whole step (prefill + decode).  ``roofline`` is for the dominant
decode kernel (the gate/up projection GEMM with the SwiGLU epilogue), whose
launches are timed with HIP events inside the library during the timed
region; ``cpu_baseline`` times the CPU oracle on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
METRIC = "decode tokens/s at ready-batch B (8B shape, 1 GPU); % HBM / MFMA roofline"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def run_step(model, prompts, n_new, chunk, torch):
    """Prefill all prompts (chunked, batched), then n_new - 1 decode steps.
    Returns the three HIP events (start, prefill done, decode done)."""
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
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per launch of the decode gate/up GEMM from the profile summary,
    or None if there is none or the kernel sources changed since."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith(" "))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_sha256") != kernel_source_hash():
        return None
    try:
        return int(float(kv["traffic_bytes_per_launch"]))
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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--agents", type=int, default=25)
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    shape = synth.LLAMA3_8B
    prompts, n_new = synth.llama8b_agent_batch(args.seed, n_agents=args.agents)
    n = len(prompts)
    chunk = 512
    lens = np.array([len(p) for p in prompts])
    log(f"workload: {n} agents, prompt tokens {lens.sum()} (min {lens.min()}, max {lens.max()}), "
        f"{n_new} generated each")

    t0 = time.time()
    model = metro.Model(shape, max_batch=max(64, n), max_tokens=n * chunk, max_context=4096 + 128,
                        max_seqs=2 * n, kv_pool_bytes=24 << 30, seed=args.seed)
    info = model.info()
    log(f"model ready in {time.time() - t0:.1f}s: weights {info.weight_bytes / 1e9:.2f} GB, "
        f"KV pool {info.kv_pool_bytes / 1e9:.1f} GB ({info.n_pages} pages)")

    # warmup (untimed); the first one also measures the prefill gate/up GEMM
    for w in range(args.warmup):
        if w == 0:
            model.profile_start("gemm_gate_up", "prefill")
        ev = run_step(model, prompts, n_new, chunk, torch)
        torch.cuda.synchronize()
        if w == 0:
            pf_ms, pf_launches = model.profile_stop()
        log(f"warmup {w}: prefill {ev[0].elapsed_time(ev[1]):.1f} ms, decode {ev[1].elapsed_time(ev[2]):.1f} ms")

    # timed region
    model.profile_start("gemm_gate_up", "decode")
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    events = [run_step(model, prompts, n_new, chunk, torch) for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    gu_ms, gu_launches = model.profile_stop()

    prefill_ms = sum(e[0].elapsed_time(e[1]) for e in events)
    decode_ms = sum(e[1].elapsed_time(e[2]) for e in events)
    step_ms = sum(e[0].elapsed_time(e[2]) for e in events) / args.steps
    decode_tokens = n * (n_new - 1) * args.steps
    value = decode_tokens / (decode_ms / 1e3)
    prefill_tps = lens.sum() * args.steps / (prefill_ms / 1e3)
    log(f"timed: {args.steps} steps, wall {wall:.2f}s, step {step_ms:.1f} ms, prefill {prefill_ms / args.steps:.1f}"
        f" ms/step ({prefill_tps:.0f} tok/s), decode {decode_ms / args.steps:.1f} ms/step ({value:.0f} tok/s)")

    # roofline of the dominant decode kernel: algorithmic bytes per launch
    d, F = shape["d_model"], shape["ffn_dim"]
    gu_bytes = 2 * F * d * 2 + n * d * 2 + n * F * 2   # W_gate|W_up + h in + SwiGLU out (bf16)
    gu_avg_s = gu_ms / 1e3 / gu_launches
    achieved = gu_bytes / gu_avg_s / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                "kernel": "gemm gate/up + SwiGLU (decode, M=25, N=28672, K=4096)",
                "bytes_per_launch": gu_bytes, "avg_launch_us": round(gu_avg_s * 1e6, 2),
                "launches": gu_launches}
    out = {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(step_ms, 2), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic: seeded uniform token ids, random N(0,0.02) bf16 weights",
           "config": {"workload": "Llama-3-8B-shaped decoder, 25 agent requests, prompts lognormal(median 1200, "
                                  "sigma 0.5) clipped to [256,4096], chunked prefill 512, 64 greedy tokens each",
                      "agents": n, "prompt_tokens": int(lens.sum()), "decode_steps": n_new - 1,
                      "ready_batch": n, "page_size": 16},
           "roofline": roofline,
           "decode_ms_per_step": round(decode_ms / args.steps, 2),
           "prefill_ms_per_step": round(prefill_ms / args.steps, 2),
           "prefill_tokens_per_s": round(prefill_tps, 1)}
    if args.warmup > 0 and pf_launches:
        pf_flops = 2.0 * 2 * F * d * lens.sum() * shape["n_layers"]
        pf_tflops = pf_flops / (pf_ms / 1e3) / 1e12
        out["roofline_prefill"] = {"bound": "mfma", "achieved": round(pf_tflops, 1), "peak": BF16_PEAK_TFLOPS,
                                   "unit": "TFLOP/s", "frac": round(pf_tflops / BF16_PEAK_TFLOPS, 4),
                                   "kernel": "gemm gate/up + SwiGLU (prefill chunks)", "launches": pf_launches}
    model.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.seed)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
