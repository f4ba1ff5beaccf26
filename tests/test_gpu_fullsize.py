"""The HIP path against the oracle at the workloads' real sizes.

Each case runs the full batch in the launch configuration of the workload
(batched prefill with many agents per call, then decode steps over the whole
ready batch) and compares sampled agents with the oracle, which
evaluates them one by one (float64 with the bf16 storage points; the same
function in float32 gives the noise floor of the bounds, see tests/parity.py).
Decode steps are teacher-forced with seeded token ids on both sides, so one
oracle pass over prompt + fed tokens yields every compared row; a
free-running row instead feeds the GPU's own greedy tokens, and the oracle is
fed the GPU's stream.

- Llama-3-8B shape at full depth (32 layers): the benchmarked workload, 25
  agents with lognormal prompts (median 1200), all prefilled in one forward
  (31527 tokens), decode at B = 25 for 16 steps.  Compared: five agents
  teacher-forced (the longest prompt, 2376 tokens, and four of 637..844
  tokens) and one free-running greedy stream (the 375-token agent).
- 8B widths, 2 layers, a ready batch of 800 agents (the largest batch of the
  agent trace) with lognormal(median 1500) contexts: tiled GEMMs and 800-row
  attention in decode.  Two agents against the oracle; and 600 of the agents,
  decoded again (forked sequences) in another batch of 800 where the other 200
  rows are different agents, must give bitwise the same logits.  (The GEMM
  kernel and its k split are chosen from the number of rows, plan_gemm, so
  equal batch sizes form each row's sums in the same order.)
- 8B widths, 2 layers, the prefix-heavy batch: a 1024-token prefix prefilled
  once and forked by page reference into 64 requests with suffixes of
  512..2048 tokens.  Every request's block table starts with the same 64
  prefix pages, and the shortest request is compared with the oracle.
  (Bitwise equality with an unshared run is not asked for here: its calls
  would have other token counts, and the GEMM kernel, so the summation order,
  is chosen by the number of rows, plan_gemm.)
- Llama-3-70B widths (d 8192, 64/8 heads: GQA group 8, FFN 28672), 2 layers,
  128 agents with contexts uniform in [1024, 3072], decode at B = 128.
"""

import numpy as np
import pytest

from oracle import LlamaShape, OracleModel
from paper_2411_03519_amd import synth
from tests.parity import assert_logits_close, check_tokens, noise_floor

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DECODE_STEPS = 8
FULL_DEPTH_STEPS = 16


@pytest.fixture(scope="module")
def metro():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2411_03519_amd import metro as m
    return m


def say(*a):
    from tests.conftest import progress  # shown under -q too: the oracle runs for minutes
    progress(*a)


def oracle_rows(shape, weights, prompt, feed, dtype):
    """Oracle logits at the prompt's last position and after each fed token."""
    ref = OracleModel(LlamaShape(**shape), weights, dtype=dtype, lazy=True)
    n = len(prompt)
    seq = np.concatenate([np.asarray(prompt, np.int64), np.asarray(feed, np.int64)])
    return ref.forward(ref.new_cache(), seq, logits_for=list(range(n - 1, n + len(feed))))


def oracle_with_floor(shape, weights, prompt, feed, what):
    say(f"{what}: oracle float64 ({len(prompt)} + {len(feed)} tokens)")
    want = oracle_rows(shape, weights, prompt, feed, np.float64)
    say(f"{what}: oracle float32")
    f32 = oracle_rows(shape, weights, prompt, feed, np.float32)
    return want, f32, noise_floor(want, f32)


def oracle_rows_each(shape, weights, prompts, feeds, dtype, what):
    """oracle_rows for several sequences, layer by layer (each layer's weights
    converted once); progress printed per layer."""
    ref = OracleModel(LlamaShape(**shape), weights, dtype=dtype, lazy=True)
    seqs = [np.concatenate([np.asarray(p, np.int64), np.asarray(f, np.int64)]) for p, f in zip(prompts, feeds)]
    sel = [list(range(len(p) - 1, len(p) + len(f))) for p, f in zip(prompts, feeds)]
    name = np.dtype(dtype).name
    return ref.forward_each([ref.new_cache() for _ in seqs], seqs, sel,
                            on_layer=lambda li: say(f"{what}: oracle {name} layer {li + 1}/{shape['n_layers']}"))


def prefill_batched(m, seqs, prompts, chunk, group, keep):
    """Chunked prefill of prompts[i] into seqs[i], ``group`` items per call.
    Returns {i: (last-position logits, next token)} for i in keep."""
    keep = set(keep)
    out = {}
    for g0 in range(0, len(seqs), group):
        idx = list(range(g0, min(len(seqs), g0 + group)))
        off = 0
        while True:
            items = [i for i in idx if off < len(prompts[i])]
            if not items:
                break
            lg = torch.empty(len(items), m.vocab, device="cuda")
            nt = torch.empty(len(items), dtype=torch.int32, device="cuda")
            m.prefill_chunk([seqs[i] for i in items], [prompts[i][off:off + chunk] for i in items], lg, nt)
            for j, i in enumerate(items):
                if i in keep and off + chunk >= len(prompts[i]):
                    out[i] = (lg[j].cpu().numpy(), int(nt[j].item()))
            off += chunk
    return out


def decode_fed(m, seqs, feeds, keep):
    """feeds.shape[1] decode steps over all seqs in one batch, row i fed
    feeds[i, k].  Returns {i: (logits [steps, V], tokens [steps])} for i in keep."""
    B = len(seqs)
    lg = torch.empty(B, m.vocab, device="cuda")
    nt = torch.empty(B, dtype=torch.int32, device="cuda")
    sel = torch.tensor(list(keep), dtype=torch.int64, device="cuda")
    rows = {i: ([], []) for i in keep}
    for k in range(feeds.shape[1]):
        m.decode_step(seqs, torch.tensor(feeds[:, k], dtype=torch.int32, device="cuda"), lg, nt)
        lgh, nth = lg[sel].cpu().numpy(), nt[sel].cpu().numpy()
        for j, i in enumerate(keep):
            rows[i][0].append(lgh[j])
            rows[i][1].append(nth[j])
    return {i: (np.stack(a), np.array(b)) for i, (a, b) in rows.items()}


def stitched(pre, dec, i):
    """Prefill row then decode rows of agent i: logits [1+steps, V], tokens [1+steps]."""
    return (np.concatenate([pre[i][0][None], dec[i][0]]), np.concatenate([[pre[i][1]], dec[i][1]]))


def compare(what, got, toks, want, f32, bounds):
    assert_logits_close(got, want, what, max_abs_bound=bounds[0], rel_bound=bounds[1])
    check_tokens(toks, want, what, f32_logits=f32)


def decode_free_and_fed(m, seqs, feeds, first_tok, free, keep):
    """feeds.shape[1] decode steps over all seqs in one batch: row i is fed
    feeds[i, k], except the rows in ``free``, which are fed their own previous
    greedy token (first_tok[i] before the first step).  Returns {i: (logits
    [steps, V], tokens [steps], inputs [steps])} for i in keep."""
    B = len(seqs)
    lg = torch.empty(B, m.vocab, device="cuda")
    nt = torch.empty(B, dtype=torch.int32, device="cuda")
    sel = torch.tensor(list(keep), dtype=torch.int64, device="cuda")
    prev = dict(first_tok)
    rows = {i: ([], [], []) for i in keep}
    for k in range(feeds.shape[1]):
        inp = feeds[:, k].copy()
        for i in free:
            inp[i] = prev[i]
        m.decode_step(seqs, torch.tensor(inp, dtype=torch.int32, device="cuda"), lg, nt)
        lgh, nth = lg[sel].cpu().numpy(), nt[sel].cpu().numpy()
        for j, i in enumerate(keep):
            rows[i][0].append(lgh[j])
            rows[i][1].append(nth[j])
            rows[i][2].append(inp[i])
            prev[i] = int(nth[j])
    return {i: tuple(np.array(x) for x in r) for i, r in rows.items()}


@pytest.mark.timeout(1800)
def test_llama3_8b_full_depth_benchmark_batch(metro):
    shape = synth.LLAMA3_8B
    V = shape["vocab"]
    prompts, _ = synth.llama8b_agent_batch(0)
    lens = np.array([len(p) for p in prompts])
    order = np.argsort(lens, kind="stable")
    free = [int(order[0])]                                  # the shortest prompt runs free
    fed = [int(order[-1])] + [int(i) for i in order[1:5]]   # the longest and the next four shortest
    keep = fed + free
    feeds = synth.feed_tokens(0, len(prompts), FULL_DEPTH_STEPS, V)
    say(f"8B full depth: agents {keep} ({lens[keep].tolist()} prompt tokens), drawing 16 GB of weights")
    w = synth.llama_weights(shape, 0, workers=16)
    say("8B full depth: gpu (upload, prefill of 25 agents, decode at B = 25)")
    m = metro.Model(shape, max_batch=64, max_tokens=int(lens.sum()), max_context=4096 + 128,
                    max_seqs=2 * len(prompts), kv_pool_bytes=24 << 30)
    with m:
        m.load_weights(w)
        seqs = [m.seq_open() for _ in prompts]
        pre = prefill_batched(m, seqs, prompts, 4096, len(prompts), keep)   # all prompts in one forward
        dec = decode_free_and_fed(m, seqs, feeds, {i: pre[i][1] for i in free}, free, keep)
    # what the oracle is fed after each prompt: the fed tokens, or the GPU's own stream
    fed_in = {i: dec[i][2] for i in keep}
    for i in fed:
        np.testing.assert_array_equal(fed_in[i], feeds[i])
    assert fed_in[free[0]][0] == pre[free[0]][1]
    np.testing.assert_array_equal(fed_in[free[0]][1:], dec[free[0]][1][:-1])
    ps = [prompts[i] for i in keep]
    fs = [fed_in[i] for i in keep]
    want = oracle_rows_each(shape, w, ps, fs, np.float64, "8B full depth")
    f32 = oracle_rows_each(shape, w, ps, fs, np.float32, "8B full depth")
    bounds = noise_floor(np.stack(want), np.stack(f32))
    all_toks = []
    for a, i in enumerate(keep):
        got = np.concatenate([pre[i][0][None], dec[i][0]])
        toks = np.concatenate([[pre[i][1]], dec[i][1]])
        all_toks.append(toks)
        kind = "free-running" if i in free else "teacher-forced"
        what = f"8B full depth agent {i} ({lens[i]} tokens, {kind})"
        assert_logits_close(got, want[a], what, max_abs_bound=bounds[0], rel_bound=bounds[1])
        n_div = int(np.sum(toks != np.argmax(want[a], axis=-1)))
        say(f"{what}: {n_div} of {len(toks)} greedy choices differ from the float64 oracle's")
    # greedy choices judged over all compared steps together (tie rate ~ the
    # density of top-2 margins below 2e-2, a few percent at full depth)
    check_tokens(np.stack(all_toks), np.stack(want), "8B full depth, all agents", f32_logits=np.stack(f32))


def test_8b_widths_ready_batch_800(metro):
    shape = synth.with_layers(synth.LLAMA3_8B, 2)
    V = shape["vocab"]
    B = 800
    ctx_all = synth.trace_start_contexts(0)
    ctx = ctx_all[:B]
    extra = ctx_all[B:]
    lens = np.array([len(c) for c in ctx])
    s1 = int(np.argmin(lens))
    s2 = min((n, j) for j, n in enumerate(lens) if n > 1024)[1]
    feeds = synth.feed_tokens(1, B, DECODE_STEPS, V)
    say("B=800: drawing weights")
    w = synth.llama_weights(shape, 1, workers=16)
    wants = {s: oracle_with_floor(shape, w, ctx[s], feeds[s], f"B=800 agent {s}") for s in (s1, s2)}
    shared = [i for i in range(B) if i < 400 or i >= 600]
    say(f"B=800: gpu prefill of {lens.sum()} + {sum(len(c) for c in extra)} tokens, decode of two batches of {B}")
    m = metro.Model(shape, max_batch=B, max_tokens=32 * 512, max_context=4096 + 16, max_seqs=2 * B + 400,
                    kv_pool_bytes=20 << 30)
    with m:
        m.load_weights(w)
        seqs = [m.seq_open() for _ in range(B)]
        others = [m.seq_open() for _ in extra]
        pre = prefill_batched(m, seqs, ctx, 512, 32, [s1, s2])
        prefill_batched(m, others, extra, 512, 32, [])
        forks = [m.seq_fork(seqs[i], int(lens[i])) for i in shared]
        dec = decode_fed(m, seqs, feeds, shared)
        # the same agents at the same rows, the rows 400..599 taken by other agents
        batch2 = forks[:400] + others + forks[400:]
        feeds2 = np.concatenate([feeds[:400], synth.feed_tokens(5, len(others), DECODE_STEPS, V), feeds[600:]])
        rows2 = list(range(400)) + list(range(600, B))
        dec2 = decode_fed(m, batch2, feeds2, rows2)
    for i in shared:
        np.testing.assert_array_equal(dec2[i][0], dec[i][0], err_msg=f"agent {i}: other batch of {B}")
        np.testing.assert_array_equal(dec2[i][1], dec[i][1])
    for s in (s1, s2):
        got, toks = stitched(pre, dec, s)
        compare(f"B=800 agent {s} ({lens[s]} tokens)", got, toks, *wants[s])


def test_8b_widths_prefix_heavy_forked(metro):
    shape = synth.with_layers(synth.LLAMA3_8B, 2)
    V = shape["vocab"]
    prefix, suffixes, _ = synth.prefix_heavy_batch(0)
    n = len(suffixes)
    i = int(np.argmin([len(s) for s in suffixes]))
    feeds = synth.feed_tokens(2, n, DECODE_STEPS, V)
    say("prefix-heavy: drawing weights")
    w = synth.llama_weights(shape, 2, workers=16)
    full_i = np.concatenate([prefix, suffixes[i]])
    want, f32, bounds = oracle_with_floor(shape, w, full_i, feeds[i], "prefix-heavy")
    say(f"prefix-heavy: gpu, {n} forks of a {len(prefix)}-token prefix")
    m = metro.Model(shape, max_batch=64, max_tokens=n * 512, max_context=1024 + 2048 + 16, max_seqs=2 * n + 4,
                    kv_pool_bytes=8 << 30)
    with m:
        m.load_weights(w)
        base = m.seq_open()
        prefill_batched(m, [base], [prefix], 512, 1, [])
        forks = [m.seq_fork(base, len(prefix)) for _ in range(n)]
        m.seq_close(base)
        shared = m.seq_pages(forks[0])
        assert len(shared) == len(prefix) // 16
        pre = prefill_batched(m, forks, suffixes, 512, n, [i])
        dec = decode_fed(m, forks, feeds, [i])
        tables = [m.seq_pages(f) for f in forks]
    for t, suf in zip(tables, suffixes):
        np.testing.assert_array_equal(t[:len(shared)], shared)
        assert len(t) == (len(prefix) + len(suf) + DECODE_STEPS + 15) // 16
    own = np.concatenate([t[len(shared):] for t in tables])
    assert len(np.unique(own)) == len(own) and not np.isin(own, shared).any()
    got, toks = stitched(pre, dec, i)
    compare(f"prefix-heavy request {i} ({len(full_i)} tokens)", got, toks, want, f32, bounds)


def test_70b_widths_batch_128(metro):
    shape = synth.with_layers(synth.LLAMA3_70B, 2)
    V = shape["vocab"]
    ctx, _ = synth.llama70b_agent_batch(0)
    lens = np.array([len(c) for c in ctx])
    i = int(np.argmin(lens))
    feeds = synth.feed_tokens(3, len(ctx), DECODE_STEPS, V)
    say("70B widths: drawing weights")
    w = synth.llama_weights(shape, 3, workers=16)
    want, f32, bounds = oracle_with_floor(shape, w, ctx[i], feeds[i], "70B widths")
    say(f"70B widths: gpu prefill of {lens.sum()} tokens, decode at B = {len(ctx)}")
    m = metro.Model(shape, max_batch=len(ctx), max_tokens=32 * 512, max_context=3072 + 16,
                    max_seqs=len(ctx) + 4, kv_pool_bytes=8 << 30)
    with m:
        m.load_weights(w)
        seqs = [m.seq_open() for _ in ctx]
        pre = prefill_batched(m, seqs, ctx, 512, 32, [i])
        dec = decode_fed(m, seqs, feeds, [i])
    got, toks = stitched(pre, dec, i)
    compare(f"70B widths agent {i} ({lens[i]} tokens)", got, toks, want, f32, bounds)


def test_8b_widths_logit_drift_across_batch_sizes(metro):
    """The GEMM kernel and its k split are chosen from a call's row count, so
    one agent's decode logits are bitwise the same in batches of equal size but
    may differ by fp32 rounding across sizes.  This measures that drift: eight
    agents decoded alone and inside batches of 16 .. 800 (forks of the same
    sequences, the same fed tokens), 8B widths at depth 2.  Every batch's
    logits must stay within the float32 noise floor of the B = 1 ones (the
    parity bound at these widths is 1.25x the oracle's spread of ~3e-2 max-abs;
    two evaluations each inside it differ by at most twice that), and greedy
    choices may differ only where B = 1's top-2 margin is below 2e-2."""
    shape = synth.with_layers(synth.LLAMA3_8B, 2)
    V = shape["vocab"]
    Bmax = 800
    rng = np.random.default_rng(12)
    prompts = [rng.integers(0, V, int(n)) for n in rng.integers(40, 300, Bmax)]
    feed = rng.integers(0, V, Bmax)
    say("batch drift: drawing weights")
    w = synth.llama_weights(shape, 4, workers=16)
    m = metro.Model(shape, max_batch=Bmax, max_tokens=64 * 300, max_context=512, max_seqs=2 * Bmax + 8,
                    kv_pool_bytes=16 << 30)
    sizes = [1, 16, 25, 64, 65, 128, 200, 256, 400, 800]
    with m:
        m.load_weights(w)
        seqs = [m.seq_open() for _ in prompts]
        prefill_batched(m, seqs, prompts, 512, 64, [])
        lg = torch.empty(Bmax, V, device="cuda")

        def decode(rows_of_batch):
            forks = [m.seq_fork(seqs[i], len(prompts[i])) for i in rows_of_batch]
            B = len(forks)
            m.decode_step(forks, torch.tensor(feed[rows_of_batch], dtype=torch.int32, device="cuda"), lg[:B])
            out = lg[:min(B, 8)].cpu().numpy().astype(np.float64)
            for f in forks:
                m.seq_close(f)
            return out

        alone = np.stack([decode([i])[0] for i in range(8)])
        rows = {B: decode(list(range(B))) for B in sizes[1:]}
    margin = np.sort(alone, axis=1)[:, -1] - np.sort(alone, axis=1)[:, -2]
    for B in sizes[1:]:
        got = rows[B]
        d = np.abs(got - alone)
        rel = np.linalg.norm(got - alone, axis=1) / np.linalg.norm(alone, axis=1)
        flips = np.argmax(got, axis=1) != np.argmax(alone, axis=1)
        say(f"batch {B} vs alone: agents 0..7 max-abs drift {d.max():.3e}, max rel-L2 {rel.max():.3e}, "
            f"bitwise equal rows {int(np.sum(np.all(got == alone, axis=1)))} of 8, greedy changes {int(flips.sum())}")
        assert d.max() <= 8e-2 and rel.max() <= 1e-2
        assert not np.any(flips & (margin >= 2e-2))
