"""The HIP path against the oracle, through the C ABI (metro.h).

Tiny Llama-style shape (2 layers, d 256, 4/2 heads of 64, FFN 688, vocab
4096): agent batches with prompts of 32..128 tokens, batched prefill, chunked
prefill, greedy decode, prefix forks, page-order and batch-composition
invariance, and the error conventions.  The 8B-width case runs the real
Llama-3-8B layer widths at reduced depth.
"""

import numpy as np
import pytest

from oracle import LlamaShape, OracleModel
from oracle.prefix_cache import OraclePrefixCache
from paper_2411_03519_amd import synth
from tests.parity import assert_logits_close, check_tokens, noise_floor

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def metro():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2411_03519_amd import metro as m
    return m


def make_model(metro, shape, weights, **kw):
    args = dict(max_batch=64, max_tokens=1024, max_context=512, kv_pool_bytes=256 << 20)
    args.update(kw)
    m = metro.Model(shape, **args)
    m.load_weights(weights)
    return m


def gpu_teacher_forced(m, prompts, feeds, chunk=None):
    """Batched (optionally chunked) prefill of all prompts, then decode steps
    fed with ``feeds[i][k]``.  Returns logits [n, 1+steps, V] and tokens."""
    n = len(prompts)
    V = m.vocab
    seqs = [m.seq_open() for _ in range(n)]
    rows = [[None] for _ in range(n)]
    toks = [[None] for _ in range(n)]
    step = chunk or max(len(p) for p in prompts)
    off = 0
    while True:
        items = [i for i in range(n) if off < len(prompts[i])]
        if not items:
            break
        lg = torch.empty(len(items), V, device="cuda")
        nt = torch.empty(len(items), dtype=torch.int32, device="cuda")
        m.prefill_chunk([seqs[i] for i in items], [prompts[i][off:off + step] for i in items], lg, nt)
        lgh, nth = lg.cpu().numpy(), nt.cpu().numpy()
        for j, i in enumerate(items):
            if off + step >= len(prompts[i]):
                rows[i][0], toks[i][0] = lgh[j], nth[j]
        off += step
    n_steps = len(feeds[0])
    lg = torch.empty(n, V, device="cuda")
    nt = torch.empty(n, dtype=torch.int32, device="cuda")
    for k in range(n_steps):
        feed = torch.tensor([int(feeds[i][k]) for i in range(n)], dtype=torch.int32, device="cuda")
        m.decode_step(seqs, feed, lg, nt)
        lgh, nth = lg.cpu().numpy(), nt.cpu().numpy()
        for i in range(n):
            rows[i].append(lgh[i])
            toks[i].append(nth[i])
    for s in seqs:
        m.seq_close(s)
    return np.array([np.stack(r) for r in rows]), np.array([np.array(t) for t in toks])


@pytest.fixture(scope="module")
def tiny_case():
    prompts, n_new = synth.tiny_agent_batch(0)
    out = {}
    for norm in ("ones", "random"):
        w = synth.llama_weights(synth.TINY, 0, norm=norm)
        ref = OracleModel(LlamaShape(**synth.TINY), w)
        gens = [ref.generate(p, n_new) for p in prompts]
        out[norm] = (w, gens)
    return prompts, n_new, out


@pytest.mark.parametrize("norm", ["ones", "random"])
def test_tiny_agent_batch_teacher_forced(metro, tiny_case, norm):
    prompts, n_new, cases = tiny_case
    w, gens = cases[norm]
    print(f"tiny teacher-forced norm={norm}", flush=True)
    with make_model(metro, synth.TINY, w) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:-1] for g in gens])
    want = np.stack([g[1] for g in gens])
    assert_logits_close(logits, want, "tiny c0")
    ties = check_tokens(toks, want, "tiny c0")
    assert ties <= 2


def test_tiny_free_running_greedy_streams(metro, tiny_case):
    prompts, n_new, cases = tiny_case
    w, gens = cases["ones"]
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    with make_model(metro, synth.TINY, w) as m:
        seqs = [m.seq_open() for _ in prompts]
        lg = torch.empty(len(prompts), m.vocab, device="cuda")
        nt = torch.empty(len(prompts), dtype=torch.int32, device="cuda")
        m.prefill_chunk(seqs, prompts, lg, nt)
        streams = [nt.cpu().numpy()]
        for _ in range(n_new - 1):
            m.decode_step(seqs, nt.clone(), lg, nt)
            streams.append(nt.cpu().numpy())
    streams = np.stack(streams, axis=1)
    for i, p in enumerate(prompts):
        want = gens[i][0]
        if np.array_equal(streams[i], want):
            continue
        k = int(np.argmax(streams[i] != want))
        # the first divergence must be a tie of the oracle at that step
        assert check_tokens(streams[i][k:k + 1], gens[i][1][k:k + 1]) == 1
        # and the oracle, fed the GPU's stream, agrees with the rest of it
        tf = ref.teacher_forced(p, streams[i][:-1])
        check_tokens(streams[i], tf)


def test_decode_step_with_host_tokens_matches_device_tokens(metro, tiny_case):
    """The binding copies host tokens (list, numpy, CPU tensor) to the device;
    the library then runs exactly the device-token step."""
    prompts, n_new, cases = tiny_case
    w, gens = cases["ones"]
    feeds = [g[0][:3] for g in gens]
    outs = []
    for kind in ("device", "list", "numpy", "cpu_tensor"):
        with make_model(metro, synth.TINY, w) as m:
            seqs = [m.seq_open() for _ in prompts]
            lg = torch.empty(len(prompts), m.vocab, device="cuda")
            nt = torch.empty(len(prompts), dtype=torch.int32, device="cuda")
            m.prefill_chunk(seqs, prompts, lg, nt)
            rows = []
            for k in range(3):
                host = [int(f[k]) for f in feeds]
                feed = {"device": torch.tensor(host, dtype=torch.int32, device="cuda"), "list": host,
                        "numpy": np.array(host, np.int64), "cpu_tensor": torch.tensor(host)}[kind]
                m.decode_step(seqs, feed, lg, nt)
                rows.append((lg.cpu().numpy().copy(), nt.cpu().numpy().copy()))
        outs.append(rows)
    for kind, rows in zip(("list", "numpy", "cpu_tensor"), outs[1:]):
        for (a, ta), (b, tb) in zip(outs[0], rows):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)) and np.array_equal(ta, tb), kind


@pytest.mark.parametrize("chunk", [16, 23, 64])
def test_tiny_chunked_prefill(metro, tiny_case, chunk):
    prompts, n_new, cases = tiny_case
    w, gens = cases["random"]
    with make_model(metro, synth.TINY, w) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:3] for g in gens], chunk=chunk)
    want = np.stack([g[1][:4] for g in gens])
    assert_logits_close(logits, want, f"chunk {chunk}")
    check_tokens(toks, want)


def test_mixed_prefill_and_decode_items(metro, tiny_case):
    """One prefill call may carry one-token continuations of sequences that
    already hold context (decode steps through the prefill path) beside whole
    prompts and first chunks: the mixed batching the scheduler loop uses."""
    prompts, n_new, cases = tiny_case
    w, gens = cases["random"]
    print("tiny mixed prefill/decode items", flush=True)
    with make_model(metro, synth.TINY, w) as m:
        V = m.vocab
        s = [m.seq_open() for _ in range(4)]
        lg = torch.empty(4, V, device="cuda")
        nt = torch.empty(4, dtype=torch.int32, device="cuda")
        m.prefill_chunk(s[:2], prompts[:2], lg[:2], nt[:2])
        first = lg[:2].cpu().numpy()
        cut = len(prompts[3]) // 2
        # decode tokens of seqs 0 and 1, the whole prompt 2, the first half of prompt 3
        m.prefill_chunk(s, [gens[0][0][:1], gens[1][0][:1], prompts[2], prompts[3][:cut]], lg, nt)
        mixed = lg.cpu().numpy()
        # seq 0's next token beside the rest of prompt 3
        m.prefill_chunk([s[0], s[3]], [gens[0][0][1:2], prompts[3][cut:]], lg[:2], nt[:2])
        last = lg[:2].cpu().numpy()
    assert_logits_close(np.stack([first[0], mixed[0], last[0]])[None], gens[0][1][None, :3], "mixed seq 0")
    assert_logits_close(np.stack([first[1], mixed[1]])[None], gens[1][1][None, :2], "mixed seq 1")
    assert_logits_close(mixed[2][None, None], gens[2][1][None, :1], "mixed seq 2")
    assert_logits_close(last[1][None, None], gens[3][1][None, :1], "mixed seq 3")


def test_decode_rows_independent_of_batch_composition(metro):
    w = synth.llama_weights(synth.TINY, 1)
    rng = np.random.default_rng(21)
    prompts = [rng.integers(0, 4096, int(rng.integers(20, 90))) for _ in range(40)]
    with make_model(metro, synth.TINY, w, max_seqs=128) as m:
        seqs = [m.seq_open() for _ in prompts]
        for g in range(0, 40, 10):
            m.prefill_chunk(seqs[g:g + 10], prompts[g:g + 10])
        feed = torch.tensor(rng.integers(0, 4096, 40), dtype=torch.int32, device="cuda")
        results = []
        for B in (1, 4, 20, 40):
            forks = [m.seq_fork(s, m.seq_length(s)) for s in seqs[:B]]
            lg = torch.empty(B, m.vocab, device="cuda")
            m.decode_step(forks, feed[:B].contiguous(), lg)
            results.append(lg[0].cpu().numpy())
            for f in forks:
                m.seq_close(f)
    for r in results[1:]:
        np.testing.assert_array_equal(r, results[0])


def test_page_order_does_not_change_results(metro):
    w = synth.llama_weights(synth.TINY, 2)
    rng = np.random.default_rng(22)
    prompts = [rng.integers(0, 4096, n) for n in (77, 50)]
    outs = []
    for scramble in (False, True):
        with make_model(metro, synth.TINY, w) as m:
            if scramble:
                junk = [m.seq_open() for _ in range(12)]
                m.prefill_chunk(junk, [rng.integers(0, 4096, int(n)) for n in rng.integers(1, 60, 12)])
                for j in junk[::2]:
                    m.seq_close(j)
            seqs = [m.seq_open() for _ in prompts]
            lg = torch.empty(2, m.vocab, device="cuda")
            m.prefill_chunk(seqs, prompts, lg)
            feed = torch.tensor([5, 6], dtype=torch.int32, device="cuda")
            lg2 = torch.empty(2, m.vocab, device="cuda")
            m.decode_step(seqs, feed, lg2)
            outs.append((lg.cpu().numpy(), lg2.cpu().numpy(), [m.seq_pages(s) for s in seqs]))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])
    assert any(not np.array_equal(a, b) for a, b in zip(outs[0][2], outs[1][2]))


@pytest.mark.parametrize("prefix_len", [48, 37])
def test_prefix_fork_shares_pages(metro, prefix_len):
    w = synth.llama_weights(synth.TINY, 3, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    rng = np.random.default_rng(23)
    prefix = rng.integers(0, 4096, prefix_len)
    suffixes = [rng.integers(0, 4096, n) for n in (20, 33, 9)]
    with make_model(metro, synth.TINY, w) as m:
        base = m.seq_open()
        m.prefill_chunk([base], [prefix])
        forks = [m.seq_fork(base, prefix_len) for _ in suffixes]
        shared = prefix_len // 16
        for f in forks:
            assert np.array_equal(m.seq_pages(f)[:shared], m.seq_pages(base)[:shared])
            if prefix_len % 16:
                assert m.seq_pages(f)[shared] != m.seq_pages(base)[shared]
        lg = torch.empty(3, m.vocab, device="cuda")
        m.prefill_chunk(forks, suffixes, lg)
        got = lg.cpu().numpy()
        # the same chunks without sharing give bit-identical results
        plain = [m.seq_open() for _ in suffixes]
        for p in plain:  # same GEMM shapes as the base prefill
            m.prefill_chunk([p], [prefix])
        lg2 = torch.empty(3, m.vocab, device="cuda")
        m.prefill_chunk(plain, suffixes, lg2)
        np.testing.assert_array_equal(lg2.cpu().numpy(), got)
        for f in forks:
            m.seq_close(f)
        m.seq_close(base)
    want = np.stack([ref.prefill(ref.new_cache(), np.concatenate([prefix, s])) for s in suffixes])
    assert_logits_close(got, want, "fork")


def run_cached_calls(m, calls, n_steps, ref_cache=None):
    """One round of agent calls through the prefix cache: every call opens its
    sequence with its prompt, the uncached rest of all prompts is prefilled in
    one batch, then ``n_steps`` decode steps are fed with the greedy tokens of
    the previous step.  Returns (n_cached per call, logits [n, 1+steps, V],
    fed tokens [n, steps])."""
    seqs, ks = [], []
    for i, p in enumerate(calls):
        s, k = m.seq_open_cached(p)
        if ref_cache is not None:
            want = ref_cache.open_cached(s, p)
            assert k == want, f"call {i}: {k} tokens taken from the cache, oracle {want}"
        seqs.append(s)
        ks.append(k)
    n, V = len(calls), m.vocab
    lg = torch.empty(n, V, device="cuda")
    nt = torch.empty(n, dtype=torch.int32, device="cuda")
    m.prefill_chunk(seqs, [p[k:] for p, k in zip(calls, ks)], lg, nt)
    if ref_cache is not None:
        for s, p, k in zip(seqs, calls, ks):
            ref_cache.prefill(s, p[k:])
    rows, fed = [lg.cpu().numpy()], []
    for _ in range(n_steps):
        fed.append(nt.cpu().numpy().copy())
        m.decode_step(seqs, nt.clone(), lg, nt)
        rows.append(lg.cpu().numpy())
        if ref_cache is not None:
            for s in seqs:
                ref_cache.decode(s)
    for s in seqs:
        m.seq_close(s)
        if ref_cache is not None:
            ref_cache.close(s)
    return ks, np.stack(rows, axis=1), np.array(fed).T.reshape(n, n_steps)


def test_prefix_cache_hits_match_oracle(metro):
    """Agents' successive calls share a preamble and a persona: from the second
    round on, each call takes over exactly the pages the cache oracle names,
    by reference, and its logits match the oracle's full computation."""
    w = synth.llama_weights(synth.TINY, 5, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    prompts, _ = synth.agent_call_prompts(1, 4, 3, synth.TINY["vocab"], preamble=40, persona=24,
                                          obs_median=12, obs_sigma=0.5, obs_lo=3, obs_hi=40)
    oc = OraclePrefixCache()
    with make_model(metro, synth.TINY, w) as m:
        m.prefix_cache(4096)
        for r, calls in enumerate(prompts):
            ks, got, fed = run_cached_calls(m, calls, 3, oc)
            if r == 0:
                assert ks == [0] * 4
            else:
                assert ks == [64] * 4   # preamble + persona = 4 whole pages
            for i, p in enumerate(calls):
                want = ref.teacher_forced(p, fed[i])
                assert_logits_close(got[i], want, f"round {r} call {i} (cached {ks[i]})")
        st = m.prefix_cache_stats()
        assert st["hit_tokens"] == 2 * 4 * 64 and st["evicted"] == 0
        # each round enters its calls' whole prompt pages; the cache holds
        # exactly the distinct known prefixes of the oracle
        assert st["pages"] == len(oc.known)
        m.prefix_cache(0)
        assert m.prefix_cache_stats()["pages"] == 0 and m.info().free_pages == m.info().n_pages


def test_prefix_cache_under_page_pressure(metro):
    """A pool too small to keep every prompt: the cache gives pages back (least
    recently used first) when a call needs them, hits stay correct, and a
    cached open never takes over more than the no-eviction oracle allows."""
    w = synth.llama_weights(synth.TINY, 6, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    prompts, _ = synth.agent_call_prompts(2, 4, 5, synth.TINY["vocab"], preamble=40, persona=24,
                                          obs_median=30, obs_sigma=0.5, obs_lo=8, obs_hi=60)
    page_bytes = 2 * 2 * 64 * 16 * 2 * 2
    oc = OraclePrefixCache()
    with make_model(metro, synth.TINY, w, kv_pool_bytes=36 * page_bytes) as m:
        m.prefix_cache(1000)
        for r, calls in enumerate(prompts):
            bound = [OraclePrefixCache.open_cached(oc, -1 - i, p) for i, p in enumerate(calls)]
            for i in range(len(calls)):
                oc.close(-1 - i)
            ks, got, fed = run_cached_calls(m, calls, 2)
            for i, p in enumerate(calls):
                assert ks[i] % 16 == 0 and ks[i] <= bound[i]
                oc.open(1000 * r + i)
                oc.prefill(1000 * r + i, p)
                want = ref.teacher_forced(p, fed[i])
                assert_logits_close(got[i], want, f"round {r} call {i} (cached {ks[i]})")
        st = m.prefix_cache_stats()
        assert st["evicted"] > 0 and st["hit_tokens"] > 0
        inf = m.info()
        assert inf.free_pages + st["pages"] == inf.n_pages


def test_error_conventions(metro):
    w = synth.llama_weights(synth.TINY, 4)
    page_bytes = 2 * 2 * 64 * 16 * 2 * 2  # K+V, 2 kv heads, 16 slots, hd 64, bf16, 2 layers
    with make_model(metro, synth.TINY, w, max_batch=4, max_tokens=200, max_context=150,
                    kv_pool_bytes=10 * page_bytes, max_seqs=6) as m:
        assert m.info().n_pages == 10
        a, b = m.seq_open(), m.seq_open()
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([a, a], [[1, 2], [3]])
        assert e.value.name == "METRO_E_INVAL"
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([a, 12345], [[1, 2], [3]])
        assert e.value.name == "METRO_E_SEQ"
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([a], [[1] * 201])
        assert e.value.name == "METRO_E_CAPACITY"
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([a], [[1, 4096]])
        assert e.value.name == "METRO_E_INVAL"
        m.prefill_chunk([a], [list(range(100))])            # 7 pages
        free = m.info().free_pages
        with pytest.raises(metro.MetroError) as e:        # needs 1 + 3 more pages, 3 free
            m.prefill_chunk([a, b], [list(range(13)), list(range(40))])
        assert e.value.name == "METRO_E_NOPAGES"
        assert m.info().free_pages == free and m.seq_length(a) == 100 and m.seq_length(b) == 0
        m.prefill_chunk([b], [list(range(40))])          # 3 pages: fits exactly
        assert m.info().free_pages == 0
        m.seq_close(a)
        assert m.info().free_pages == 7
        with pytest.raises(metro.MetroError) as e:
            m.seq_close(a)
        assert e.value.name == "METRO_E_SEQ"
        with pytest.raises(metro.MetroError) as e:
            m.seq_fork(b, 41)
        assert e.value.name == "METRO_E_INVAL"
        c = m.seq_open()
        m.prefill_chunk([c], [list(range(100))])
        with pytest.raises(metro.MetroError) as e:        # 151 > max_context
            m.prefill_chunk([c], [list(range(51))])
        assert e.value.name == "METRO_E_CAPACITY"
        # out-of-range decode token: NaN logits and next_tok -1 for that row only
        lg = torch.empty(2, m.vocab, device="cuda")
        nt = torch.empty(2, dtype=torch.int32, device="cuda")
        m.decode_step([b, c], torch.tensor([7, 99999], dtype=torch.int32, device="cuda"), lg, nt)
        lgh = lg.cpu().numpy()
        assert np.all(np.isfinite(lgh[0])) and np.all(np.isnan(lgh[1]))
        assert nt.cpu().numpy()[1] == -1


def test_empty_calls_boundaries_and_maximum_sizes(metro, tiny_case):
    """Degenerate and limit cases against the oracle: a one-token prompt,
    prompts ending one short of, on, and one past a page boundary (15, 16, 17,
    32 tokens), all five prefilled in one call of exactly max_tokens tokens at
    exactly max_batch items, then decoded until the longest sequence holds
    exactly max_context tokens (every row crosses a page boundary on the way).
    One more step with that sequence is refused with nothing changed, the
    other four take it; empty calls and empty items are refused."""
    _, _, cases = tiny_case
    w = cases["random"][0]
    V = synth.TINY["vocab"]
    rng = np.random.default_rng(41)
    lens = [1, 15, 16, 17, 32]
    prompts = [rng.integers(0, V, n) for n in lens]
    n_new = 9  # the longest row reaches 32 + 7 = max_context after 7 decode steps
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    gens = [ref.generate(p, n_new) for p in prompts]
    page_bytes = 2 * 2 * 64 * 16 * 2 * 2  # K+V, 2 kv heads, 16 slots, hd 64, bf16, 2 layers
    with make_model(metro, synth.TINY, w, max_batch=5, max_tokens=sum(lens), max_context=39,
                    kv_pool_bytes=16 * page_bytes) as m:
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([], [])
        assert e.value.name == "METRO_E_INVAL"
        with pytest.raises(metro.MetroError) as e:
            m.decode_step([], torch.empty(0, dtype=torch.int32, device="cuda"))
        assert e.value.name == "METRO_E_INVAL"
        seqs = [m.seq_open() for _ in prompts]
        with pytest.raises(metro.MetroError) as e:
            m.prefill_chunk([seqs[0]], [[]])
        assert e.value.name == "METRO_E_INVAL"
        with pytest.raises(metro.MetroError) as e:
            m.decode_step(seqs + [seqs[0]], torch.zeros(6, dtype=torch.int32, device="cuda"))
        assert e.value.name == "METRO_E_CAPACITY"
        assert all(m.seq_length(s) == 0 for s in seqs)

        lg = torch.empty(5, V, device="cuda")
        nt = torch.empty(5, dtype=torch.int32, device="cuda")
        m.prefill_chunk(seqs, prompts, lg, nt)
        rows, toks = [lg.cpu().numpy()], [nt.cpu().numpy()]
        for k in range(1, 8):
            m.decode_step(seqs, [int(g[0][k - 1]) for g in gens], lg, nt)
            rows.append(lg.cpu().numpy())
            toks.append(nt.cpu().numpy())
        assert [m.seq_length(s) for s in seqs] == [n + 7 for n in lens]
        assert m.seq_length(seqs[4]) == 39
        free = m.info().free_pages
        with pytest.raises(metro.MetroError) as e:
            m.decode_step(seqs, [int(g[0][7]) for g in gens], lg, nt)
        assert e.value.name == "METRO_E_CAPACITY"
        assert [m.seq_length(s) for s in seqs] == [n + 7 for n in lens] and m.info().free_pages == free
        m.decode_step(seqs[:4], [int(g[0][7]) for g in gens[:4]], lg[:4], nt[:4])
        last, last_tok = lg[:4].cpu().numpy(), nt[:4].cpu().numpy()
    got = np.stack(rows, axis=1)
    want = np.stack([g[1][:8] for g in gens])
    assert_logits_close(got, want, "edge lengths")
    check_tokens(np.stack(toks, axis=1), want, "edge lengths")
    want_last = np.stack([g[1][8] for g in gens[:4]])
    assert_logits_close(last, want_last, "edge lengths, step past the full row")
    check_tokens(last_tok, want_last, "edge lengths, step past the full row")


def test_llama3_8b_widths_two_layers(metro):
    """Llama-3-8B layer widths (d 4096, 32/8 heads of 128, FFN 14336, vocab
    128256) at depth 2: two agents with 256- and 203-token prompts, prefilled in
    128-token chunks, then 8 decode steps."""
    shape = synth.with_layers(synth.LLAMA3_8B, 2)
    print("8B widths: drawing weights", flush=True)
    w = synth.llama_weights(shape, 0)
    rng = np.random.default_rng(24)
    prompts = [rng.integers(0, shape["vocab"], n) for n in (256, 203)]
    print("8B widths: oracle (float64)", flush=True)
    ref = OracleModel(LlamaShape(**shape), w)
    gens = [ref.generate(p, 9, chunk=128) for p in prompts]
    del ref
    print("8B widths: oracle in float32 (noise floor)", flush=True)
    r32 = OracleModel(LlamaShape(**shape), w, dtype=np.float32)
    f32 = np.stack([r32.teacher_forced(p, g[0][:-1], chunk=128) for p, g in zip(prompts, gens)])
    del r32
    want = np.stack([g[1] for g in gens])
    bound, rel_bound = noise_floor(want, f32)
    print("8B widths: gpu", flush=True)
    with make_model(metro, shape, w, max_batch=4, max_tokens=512, max_context=512, kv_pool_bytes=1 << 30) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:-1] for g in gens], chunk=128)
    assert_logits_close(logits, want, "8B widths", max_abs_bound=bound, rel_bound=rel_bound)
    check_tokens(toks, want, "8B widths", f32_logits=f32)


@pytest.mark.parametrize("hd", [64, 128])
@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_every_head_dim_and_group_the_config_accepts(metro, hd, group):
    """Each (head_dim, GQA group) pair that metro_create_model accepts selects
    its own decode and prefill attention kernels: a 2-layer model of d 256
    with 2 kv heads per pair, four agents prefilled in 64-token chunks (one
    call per chunk round), then 4 decode steps, against the oracle at the
    stated 2e-2 / 1e-2."""
    shape = dict(synth.TINY, n_heads=2 * group, n_kv_heads=2, head_dim=hd)
    w = synth.llama_weights(shape, 40 + group, norm="random")
    rng = np.random.default_rng(41 + hd + group)
    prompts = [rng.integers(0, shape["vocab"], n) for n in (1, 37, 130, 300)]
    ref = OracleModel(LlamaShape(**shape), w)
    gens = [ref.generate(p, 5, chunk=64) for p in prompts]
    with make_model(metro, shape, w, max_batch=8, max_tokens=512, max_context=512) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:-1] for g in gens], chunk=64)
    want = np.stack([g[1] for g in gens])
    assert_logits_close(logits, want, f"head dim {hd}, group {group}")
    check_tokens(toks, want, f"head dim {hd}, group {group}")


def test_long_contexts_split_decode_attention(metro):
    """Contexts of 2049 to 4300 tokens span two and three 128-page work items of
    the decode attention (merged by the combine kernel in split order); short
    rows ride along."""
    w = synth.llama_weights(synth.TINY, 5, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    rng = np.random.default_rng(25)
    prompts = [rng.integers(0, 4096, n) for n in (2049, 4300, 40, 513)]
    gens = [ref.generate(p, 4, chunk=512) for p in prompts]
    with make_model(metro, synth.TINY, w, max_batch=8, max_tokens=2048, max_context=4400) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:-1] for g in gens], chunk=512)
    want = np.stack([g[1] for g in gens])
    assert_logits_close(logits, want, "long contexts")
    check_tokens(toks, want, "long contexts")


def test_prefill_attention_past_staged_page_ids(metro):
    """A context of 8300 tokens (519 pages) runs past the 512 page ids that
    prefill attention stages in LDS; its last chunks read the rest from the
    block table."""
    w = synth.llama_weights(synth.TINY, 6, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    rng = np.random.default_rng(26)
    prompts = [rng.integers(0, 4096, n) for n in (8300, 97)]
    gens = [ref.generate(p, 2, chunk=512) for p in prompts]
    with make_model(metro, synth.TINY, w, max_batch=4, max_tokens=2048, max_context=8400,
                    kv_pool_bytes=64 << 20) as m:
        logits, toks = gpu_teacher_forced(m, prompts, [g[0][:-1] for g in gens], chunk=512)
    want = np.stack([g[1] for g in gens])
    assert_logits_close(logits, want, "prefill past staged page ids")
    check_tokens(toks, want, "prefill past staged page ids")


def test_launch_timing_spans_split_gemm_fixup(metro):
    """Launch timing of a GEMM whose last round is split over k covers the
    tiled kernel and its fixup kernel: a 1100-row gate/up (256 x 256 tiles, 30
    of them split in two) is timed no shorter than a 1000-row one (128 x 128
    tiles, no split), not as the fixup alone."""
    w = synth.llama_weights(synth.TINY, 9)
    rng = np.random.default_rng(29)
    per_launch = {}
    for n in (1000, 1100):
        with make_model(metro, synth.TINY, w, max_batch=4, max_tokens=1200, max_context=1200) as m:
            s = m.seq_open()
            m.prefill_chunk([s], [rng.integers(0, 4096, 64)])   # warm up
            t = m.seq_open()
            m.profile_start("gemm_gate_up", "prefill")
            m.prefill_chunk([t], [rng.integers(0, 4096, n)])
            ms, launches = m.profile_stop()
            assert launches == synth.TINY["n_layers"]
            per_launch[n] = ms / launches
    assert per_launch[1100] >= 0.6 * per_launch[1000], per_launch


def test_sync_check_mode_gives_the_same_results(metro, monkeypatch):
    """A model created with METRO_SYNC_CHECK=1 waits for and checks every
    launch; its prefill and decode outputs equal those of a normal model."""
    w = synth.llama_weights(synth.TINY, 10)
    rng = np.random.default_rng(30)
    prompts = [rng.integers(0, 4096, n) for n in (45, 130)]
    outs = []
    for flag in ("0", "1"):
        monkeypatch.setenv("METRO_SYNC_CHECK", flag)
        with make_model(metro, synth.TINY, w) as m:
            seqs = [m.seq_open() for _ in prompts]
            lg = torch.empty(2, m.vocab, device="cuda")
            nt = torch.empty(2, dtype=torch.int32, device="cuda")
            m.prefill_chunk(seqs, prompts, lg, nt)
            lg2 = torch.empty_like(lg)
            m.decode_step(seqs, nt, lg2)
            outs.append((lg.cpu().numpy(), lg2.cpu().numpy()))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


def test_engine_under_page_pressure_plans_again_and_matches_oracle(metro):
    """A forward whose pages the pool cannot hold fails in the model without
    changing anything; the engine then plans the step again with half the
    prompt tokens.  A stand-in sequence holds most of the pool until the
    engine has had to do so at least once (or until no forward fits at all,
    which the engine reports as E_NOPAGES), then releases it; every request
    must still finish with the oracle's greedy stream."""
    w = synth.llama_weights(synth.TINY, 12, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    rng = np.random.default_rng(32)
    reqs = [(i, int(rng.integers(0, 4)), rng.integers(0, synth.TINY["vocab"], int(n)), int(k))
            for i, (n, k) in enumerate([(70, 6), (5, 9), (130, 3), (33, 7), (64, 5), (1, 4)])]
    page_bytes = 16 * 2 * synth.TINY["n_layers"] * synth.TINY["n_kv_heads"] * synth.TINY["head_dim"] * 2
    with make_model(metro, synth.TINY, w, max_batch=8, max_tokens=128, max_context=512,
                    kv_pool_bytes=32 * page_bytes) as m:
        hold = m.seq_open()
        filler = rng.integers(0, synth.TINY["vocab"], 24 * 16)
        for c in range(0, len(filler), 128):
            m.prefill_chunk([hold], [filler[c:c + 128]])
        torch.cuda.synchronize()
        eng = metro.Engine(m, max_tokens=96, chunk=32, max_items=8, priority=True)
        for rid, step, prompt, n_out in reqs:
            eng.submit(rid, step, prompt, n_out)
        released = nopages = 0
        for _ in range(500):
            try:
                n = eng.step()
            except metro.MetroError as e:
                assert e.name == "METRO_E_NOPAGES" and hold is not None, e
                nopages += 1
                n = -1
            if hold is not None and (eng.stats()["page_retries"] > 0 or n == -1):
                m.seq_close(hold)
                hold, released = None, 1
            if n == 0:
                break
        st = eng.stats()
        assert sorted(eng.finished()) == [r[0] for r in reqs]
        streams = {rid: eng.result(rid) for rid, *_ in reqs}
        eng.close()
    print(f"engine under page pressure: {st['page_retries']} forwards planned again, {nopages} steps with no "
          f"forward that fit, {st['forwards']} forwards", flush=True)
    assert released and st["page_retries"] > 0
    assert st["prompt_tokens"] == sum(len(r[2]) for r in reqs)
    for rid, step, prompt, n_out in reqs:
        s = streams[rid]
        assert len(s) == n_out
        check_tokens(s, ref.teacher_forced(prompt, s[:-1]), f"engine request {rid} (page pressure)")


@pytest.mark.parametrize("priority", [True, False])
def test_engine_mixed_batches_match_oracle(metro, priority):
    """The library's mixed continuous batching (metro_engine_*): requests with
    different steps arrive over time; forwards mix one-token decode items with
    prompt chunks under a 96-token budget (32 per chunk), then run decode-only.
    Each request's greedy stream must be the oracle's (teacher-forced on the
    stream itself; the first difference, if any, a tie)."""
    w = synth.llama_weights(synth.TINY, 11, norm="random")
    ref = OracleModel(LlamaShape(**synth.TINY), w)
    rng = np.random.default_rng(31)
    reqs = [(i, int(rng.integers(0, 4)), rng.integers(0, synth.TINY["vocab"], int(n)), int(k))
            for i, (n, k) in enumerate([(70, 6), (5, 9), (130, 3), (33, 7), (64, 5), (1, 4)])]
    with make_model(metro, synth.TINY, w, max_batch=8, max_tokens=128, max_context=256) as m:
        eng = metro.Engine(m, max_tokens=96, chunk=32, max_items=8, priority=priority)
        mixed = 0
        for rid, step, prompt, n_out in reqs[:3]:
            eng.submit(rid, step, prompt, n_out)
        forwards = 0
        while True:
            if forwards == 2:
                for rid, step, prompt, n_out in reqs[3:]:
                    eng.submit(rid, step, prompt, n_out)
            n = eng.step()
            if n == 0 and forwards > 2:
                break
            plan = eng.last_plan()
            mixed += any(d for _, _, d in plan) and any(not d for _, _, d in plan)
            forwards += 1
        assert sorted(eng.finished()) == [r[0] for r in reqs]
        streams = {rid: eng.result(rid) for rid, *_ in reqs}
        st = eng.stats()
        eng.close()
    assert mixed > 0, "no forward mixed decode tokens with prompt chunks"
    assert st["prompt_tokens"] == sum(len(r[2]) for r in reqs)
    for rid, step, prompt, n_out in reqs:
        s = streams[rid]
        assert len(s) == n_out
        want = ref.teacher_forced(prompt, s[:-1])
        check_tokens(s, want, f"engine request {rid}")
