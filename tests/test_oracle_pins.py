"""Pins of the oracle against facts fixed outside it (CPU only).

Each building block is checked against a closed form, an invariant, brute force
or an independent library routine; the whole model (without the bf16 storage
points) is checked against the independent Llama implementation of the
``transformers`` library in float64.  ``test_oracle_mutations.py`` shows that
plausible mistakes planted in the oracle fail these pins.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import (LlamaShape, OracleModel, PagedKV, bf16_round, bf16_bits_to_f64, causal_gqa_attention,
                    greedy_argmax, rms_norm, rope_rotate, silu, softmax_rows)
from paper_2411_03519_amd import synth

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")

MICRO = dict(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn_dim=48, vocab=97,
             rope_base=10000.0, rms_eps=1e-5)


def shape_of(cfg):
    return LlamaShape(**cfg)


# ----------------------------------------------------------------------------
# bf16 rounding
# ----------------------------------------------------------------------------

def test_bf16_round_hand_cases():
    # spacing of bf16 in [1, 2) is 2^-7; halfway cases go to the even neighbour
    assert bf16_round(1.0 + 2.0 ** -8) == 1.0
    assert bf16_round(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert bf16_round(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    assert bf16_round(-(1.0 + 3 * 2.0 ** -8)) == -(1.0 + 2.0 ** -6)
    assert bf16_round(0.0) == 0.0
    # smallest subnormal 2^-133: half of it rounds to zero (even), 0.75 of it up
    assert bf16_round(2.0 ** -134) == 0.0
    assert bf16_round(1.5 * 2.0 ** -134) == 2.0 ** -133
    assert np.isinf(bf16_round(3.5e38))


def test_bf16_round_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(200000).astype(np.float32) * np.float32(3.0)
    # add exact ties: bf16 values plus half a bf16 ulp (representable in fp32)
    b = torch.tensor(x[:5000]).to(torch.bfloat16).to(torch.float32).numpy()
    _, e = np.frexp(b.astype(np.float64))
    ties = (b.astype(np.float64) + np.ldexp(1.0, e - 9)).astype(np.float32)
    x = np.concatenate([x, ties, np.float32([1e-39, -3e-40, 6e-41])])
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_round(x.astype(np.float64)), ref)


def test_bf16_bits_decode():
    bits = synth.f32_to_bf16_bits(np.float32([1.0, -2.5, 0.02, 3.0e-3]))
    ref = torch.tensor(np.float32([1.0, -2.5, 0.02, 3.0e-3])).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_bits_to_f64(bits), ref)


# ----------------------------------------------------------------------------
# RMSNorm
# ----------------------------------------------------------------------------

def test_rms_norm_closed_forms():
    g = np.linspace(0.5, 1.5, 16)
    c = 3.0
    np.testing.assert_allclose(rms_norm(np.full(16, c), g, 0.0), g, rtol=1e-15)
    np.testing.assert_allclose(rms_norm(np.full(16, c), g, 0.25), g * c / math.sqrt(c * c + 0.25), rtol=1e-15)
    np.testing.assert_allclose(rms_norm(np.full(16, -c), g, 0.0), -g, rtol=1e-15)
    x = np.random.default_rng(0).standard_normal((5, 16))
    y = rms_norm(x, np.ones(16), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-14)
    np.testing.assert_allclose(rms_norm(7.5 * x, g, 0.0), rms_norm(x, g, 0.0), rtol=1e-14)


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 64)) * 4
    g = rng.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (64,), torch.tensor(g), eps=1e-5).numpy()
    np.testing.assert_allclose(rms_norm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-14)


# ----------------------------------------------------------------------------
# RoPE
# ----------------------------------------------------------------------------

def test_rope_position_zero_is_identity():
    u = np.random.default_rng(3).standard_normal((3, 2, 16))
    np.testing.assert_array_equal(rope_rotate(u, np.zeros(3), 10000.0), u)


def test_rope_as_complex_rotation():
    # rotate-half RoPE: z_i = u_i + 1j*u_{i+hd/2} is multiplied by exp(1j*p*base^(-2i/hd))
    rng = np.random.default_rng(4)
    hd, base = 16, 500000.0
    u = rng.standard_normal((5, 3, hd))
    pos = np.array([0, 1, 7, 1000, 4099])
    z = u[..., :hd // 2] + 1j * u[..., hd // 2:]
    ang = pos[:, None] * np.exp(-np.log(base) * np.arange(0, hd, 2) / hd)[None, :]
    zr = z * np.exp(1j * ang)[:, None, :]
    np.testing.assert_allclose(rope_rotate(u, pos, base), np.concatenate([zr.real, zr.imag], -1),
                               rtol=1e-12, atol=1e-12)


def test_rope_hd4_by_hand():
    # hd = 4: pairs (0, 2) turned by p and (1, 3) turned by p / sqrt(base)
    base, p = 100.0, 3
    u = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    a0, a1 = p * 1.0, p / 10.0
    want = [1 * math.cos(a0) - 3 * math.sin(a0), 2 * math.cos(a1) - 4 * math.sin(a1),
            1 * math.sin(a0) + 3 * math.cos(a0), 2 * math.sin(a1) + 4 * math.cos(a1)]
    np.testing.assert_allclose(rope_rotate(u, np.array([p]), base)[0, 0], want, rtol=1e-14)


def test_rope_norm_and_relative_position():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 32))
    k = rng.standard_normal((1, 1, 32))
    np.testing.assert_allclose(np.linalg.norm(rope_rotate(q, np.array([123]), 1e4)), np.linalg.norm(q), rtol=1e-14)
    dots = []
    for m, n in [(10, 3), (17, 10), (1007, 1000)]:
        dots.append(float(np.sum(rope_rotate(q, np.array([m]), 1e4) * rope_rotate(k, np.array([n]), 1e4))))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)


# ----------------------------------------------------------------------------
# Softmax and attention
# ----------------------------------------------------------------------------

def test_softmax_rows_sum_to_one_and_shift_invariance():
    s = np.random.default_rng(6).standard_normal((9, 33)) * 30
    w = softmax_rows(s)
    np.testing.assert_allclose(w.sum(-1), 1.0, atol=1e-15)
    np.testing.assert_allclose(softmax_rows(s + 1000.0), w, rtol=1e-12)
    assert np.all(w >= 0)


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    o = causal_gqa_attention(q, k, v, np.array([0]))
    np.testing.assert_array_equal(o[0, 0], v[0, 0])
    np.testing.assert_array_equal(o[0, 3], v[0, 1])


def test_attention_uniform_scores_give_mean_of_visible_values():
    rng = np.random.default_rng(8)
    k = np.repeat(rng.standard_normal((1, 1, 8)), 10, axis=0)
    v = rng.standard_normal((10, 1, 8))
    q = rng.standard_normal((2, 2, 8))
    o = causal_gqa_attention(q, k, v, np.array([3, 9]))
    np.testing.assert_allclose(o[0, 1], v[:4, 0].mean(0), rtol=1e-13)
    np.testing.assert_allclose(o[1, 0], v[:, 0].mean(0), rtol=1e-13)


def test_attention_brute_force_loops():
    rng = np.random.default_rng(9)
    nq, nkv, hd, ctx = 6, 2, 4, 7
    q = rng.standard_normal((3, nq, hd))
    k = rng.standard_normal((ctx, nkv, hd))
    v = rng.standard_normal((ctx, nkv, hd))
    pos = np.array([4, 5, 6])
    o = causal_gqa_attention(q, k, v, pos)
    for i in range(3):
        for j in range(nq):
            kvh = j // (nq // nkv)
            sc = [sum(q[i, j, d] * k[t, kvh, d] for d in range(hd)) / math.sqrt(hd) for t in range(pos[i] + 1)]
            mx = max(sc)
            e = [math.exp(s - mx) for s in sc]
            z = sum(e)
            want = [sum(e[t] / z * v[t, kvh, d] for t in range(pos[i] + 1)) for d in range(hd)]
            np.testing.assert_allclose(o[i, j], want, rtol=1e-12)


def test_attention_matches_torch_sdpa_with_prior_context():
    rng = np.random.default_rng(10)
    nq, nkv, hd, ctx, n = 8, 2, 16, 40, 12
    q = rng.standard_normal((n, nq, hd))
    k = rng.standard_normal((ctx, nkv, hd))
    v = rng.standard_normal((ctx, nkv, hd))
    pos = np.arange(ctx - n, ctx)
    o = causal_gqa_attention(q, k, v, pos)
    tq = torch.tensor(q).transpose(0, 1)
    tk = torch.tensor(k).transpose(0, 1).repeat_interleave(nq // nkv, 0)
    tv = torch.tensor(v).transpose(0, 1).repeat_interleave(nq // nkv, 0)
    mask = torch.tensor(np.arange(ctx)[None, :] <= pos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask).transpose(0, 1).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)


def test_silu_matches_torch_and_limits():
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(z), torch.nn.functional.silu(torch.tensor(z)).numpy(), rtol=1e-13, atol=1e-300)
    assert silu(np.array(0.0)) == 0.0
    np.testing.assert_allclose(silu(np.array(40.0)), 40.0, rtol=1e-15)


def test_greedy_argmax_lowest_index_on_ties():
    x = np.float32([[0.5, 2.0, 2.0, -1.0], [3.0, 3.0, 3.0, 3.0], [-5.0, -4.0, -4.0, -4.5]])
    np.testing.assert_array_equal(greedy_argmax(x), [1, 0, 1])


# ----------------------------------------------------------------------------
# Whole model against an independent Llama implementation (float64)
# ----------------------------------------------------------------------------

def hf_logits(cfg: dict, weights: dict, tokens) -> np.ndarray:
    """Logits of the transformers-library Llama with the same float64 weights."""
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg["vocab"], hidden_size=cfg["d_model"], intermediate_size=cfg["ffn_dim"],
                     num_hidden_layers=cfg["n_layers"], num_attention_heads=cfg["n_heads"],
                     num_key_value_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"],
                     rope_theta=cfg["rope_base"], rms_norm_eps=cfg["rms_eps"], tie_word_embeddings=False,
                     max_position_embeddings=4096, attention_bias=False, mlp_bias=False)
    torch.manual_seed(0)
    m = LlamaForCausalLM(hc).double().eval()
    f = lambda a: torch.tensor(bf16_bits_to_f64(a))  # noqa: E731
    sd = {"model.embed_tokens.weight": f(weights["embed"]), "model.norm.weight": f(weights["final_norm"]),
          "lm_head.weight": f(weights["lm_head"])}
    names = {"attn_norm": "input_layernorm", "ffn_norm": "post_attention_layernorm",
             "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wgate": "mlp.gate_proj", "wup": "mlp.up_proj", "wdown": "mlp.down_proj"}
    for li, lw in enumerate(weights["layers"]):
        for k, hn in names.items():
            sd[f"model.layers.{li}.{hn}.weight"] = f(lw[k])
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in x for x in missing), (missing, unexpected)
    with torch.no_grad():
        return m(torch.tensor(np.asarray(tokens)[None, :])).logits[0].numpy()


def oracle_vs_hf_error(cfg, seed=11, n=21) -> float:
    w = synth.llama_weights(cfg, seed, norm="random")
    toks = np.random.default_rng(seed).integers(0, cfg["vocab"], n)
    om = OracleModel(shape_of(cfg), w, quantize=False)
    ours = om.forward(om.new_cache(), toks).astype(np.float64)
    ref = hf_logits(cfg, w, toks)
    return float(np.max(np.abs(ours - ref)) / np.max(np.abs(ref)))


def test_unquantized_oracle_matches_transformers_llama():
    # micro shape (GQA group 2) and a wider head to reach real rotation frequencies
    assert oracle_vs_hf_error(MICRO) < 1e-6
    wider = dict(MICRO, d_model=64, n_heads=8, n_kv_heads=2, head_dim=16, rope_base=500000.0)
    assert oracle_vs_hf_error(wider, seed=12, n=40) < 1e-6


# ----------------------------------------------------------------------------
# Invariants of the quantized oracle on the tiny shape
# ----------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tiny_model():
    return OracleModel(shape_of(synth.TINY), synth.llama_weights(synth.TINY, 3, norm="random"))


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_lazy_weight_conversion_is_bitwise_the_same(dtype):
    # vocabulary large enough for the threaded decode and several LM-head blocks
    cfg = dict(MICRO, vocab=140_000)
    W = synth.llama_weights(cfg, 21, norm="random")
    eager = OracleModel(shape_of(cfg), W, dtype=dtype)
    lazy = OracleModel(shape_of(cfg), W, dtype=dtype, lazy=True)
    prompt = np.random.default_rng(22).integers(0, cfg["vocab"], 19)
    t1, l1 = eager.generate(prompt, 3)
    t2, l2 = lazy.generate(prompt, 3)
    np.testing.assert_array_equal(t1, t2)
    np.testing.assert_array_equal(l1, l2)
    assert lazy.load(W["lm_head"]).dtype == dtype
    # the threaded draw gives the same tensors
    W4 = synth.llama_weights(cfg, 21, norm="random", workers=4)
    for name in ("embed", "lm_head", "final_norm"):
        np.testing.assert_array_equal(W4[name], W[name])
    for a, b in zip(W4["layers"], W["layers"]):
        for name in a:
            np.testing.assert_array_equal(a[name], b[name])
    # logits of selected positions only are the same rows
    rows = lazy.forward(lazy.new_cache(), prompt, logits_for=[3, -1])
    full = lazy.forward(lazy.new_cache(), prompt)
    np.testing.assert_array_equal(rows, full[[3, -1]])


@pytest.mark.parametrize("lazy", [False, True])
def test_forward_each_equals_separate_forwards_bitwise(lazy):
    cfg = synth.TINY
    W = synth.llama_weights(cfg, 23, norm="random")
    om = OracleModel(shape_of(cfg), W, lazy=lazy)
    rng = np.random.default_rng(23)
    toks = [rng.integers(0, cfg["vocab"], n) for n in (17, 40, 5)]
    sel = [None, [0, 39], [-1]]
    want = [om.forward(om.new_cache(), t, s) for t, s in zip(toks, sel)]
    got = om.forward_each([om.new_cache() for _ in toks], toks, sel)
    for a, b in zip(got, want):
        np.testing.assert_array_equal(a, b)


def test_paged_kv_equals_contiguous_bitwise(tiny_model):
    S = tiny_model.shape
    prompt = np.random.default_rng(13).integers(0, S.vocab, 45)
    ref = tiny_model.forward(tiny_model.new_cache(), prompt)
    perm = np.random.default_rng(14).permutation(32)
    paged = PagedKV(S, n_pages=32, page=16, free_pages=perm)
    got = tiny_model.forward(paged, prompt[:20])
    got2 = tiny_model.forward(paged, prompt[20:])
    np.testing.assert_array_equal(np.concatenate([got, got2]), ref)
    assert sorted(paged.block_table) != list(range(len(paged.block_table))) or len(paged.block_table) < 2


def test_prefill_then_decode_equals_full_recompute(tiny_model):
    S = tiny_model.shape
    prompt = np.random.default_rng(15).integers(0, S.vocab, 37)
    toks, logits = tiny_model.generate(prompt, 6)
    full = tiny_model.forward(tiny_model.new_cache(), np.concatenate([prompt, toks[:-1]]))
    np.testing.assert_allclose(logits, full[len(prompt) - 1:], rtol=0, atol=1e-5 * np.abs(full).max())
    np.testing.assert_array_equal(greedy_argmax(full[len(prompt) - 1:]), toks)


def test_chunked_prefill_equals_one_shot(tiny_model):
    S = tiny_model.shape
    prompt = np.random.default_rng(16).integers(0, S.vocab, 70)
    one = tiny_model.prefill(tiny_model.new_cache(), prompt)
    for chunk in (16, 23, 64):
        np.testing.assert_allclose(tiny_model.prefill(tiny_model.new_cache(), prompt, chunk), one,
                                   rtol=0, atol=1e-5 * np.abs(one).max())


def test_results_independent_of_batch_composition(tiny_model):
    S = tiny_model.shape
    rng = np.random.default_rng(17)
    prompts = [rng.integers(0, S.vocab, n) for n in (33, 50, 41)]
    alone = tiny_model.generate(prompts[1], 4)
    # the oracle serves agents one after another; interleaving others changes nothing
    caches = [tiny_model.new_cache() for _ in prompts]
    for c, p in zip(caches, prompts):
        tiny_model.prefill(c, p)
    cache = tiny_model.new_cache()
    tiny_model.prefill(cache, prompts[1])
    np.testing.assert_array_equal(tiny_model.generate(prompts[1], 4)[1], alone[1])


def test_gqa_equals_mha_with_replicated_kv_heads():
    cfg = dict(MICRO)
    w = synth.llama_weights(cfg, 18, norm="random")
    mha_cfg = dict(cfg, n_kv_heads=cfg["n_heads"])
    g = cfg["n_heads"] // cfg["n_kv_heads"]
    hd = cfg["head_dim"]
    w_mha = {**w, "layers": []}
    for lw in w["layers"]:
        rep = {}
        for name in ("wk", "wv"):
            m = lw[name].reshape(cfg["n_kv_heads"], hd, -1)
            rep[name] = np.repeat(m, g, axis=0).reshape(cfg["n_heads"] * hd, -1)
        w_mha["layers"].append({**lw, **rep})
    toks = np.random.default_rng(19).integers(0, cfg["vocab"], 25)
    a = OracleModel(shape_of(cfg), w).forward(OracleModel(shape_of(cfg), w).new_cache(), toks)
    mm = OracleModel(shape_of(mha_cfg), w_mha)
    b = mm.forward(mm.new_cache(), toks)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-6 * np.abs(a).max())


def test_quantized_close_to_unquantized(tiny_model):
    # the bf16 storage points perturb, but do not change the function
    w = synth.llama_weights(synth.TINY, 3, norm="random")
    exact = OracleModel(shape_of(synth.TINY), w, quantize=False)
    prompt = np.random.default_rng(20).integers(0, synth.TINY["vocab"], 30)
    a = tiny_model.forward(tiny_model.new_cache(), prompt)
    b = exact.forward(exact.new_cache(), prompt)
    rel = np.linalg.norm(a - b) / np.linalg.norm(b)
    assert 0 < rel < 0.05


def test_float32_evaluation_stays_within_tolerance_at_tiny_shape(tiny_model):
    # the same function in float32 arithmetic: the spread legitimate fp32
    # rounding causes (used as the noise floor of wider shapes)
    w = synth.llama_weights(synth.TINY, 3, norm="random")
    m32 = OracleModel(shape_of(synth.TINY), w, dtype=np.float32)
    prompt = np.random.default_rng(21).integers(0, synth.TINY["vocab"], 60)
    a = tiny_model.forward(tiny_model.new_cache(), prompt)
    b = m32.forward(m32.new_cache(), prompt)
    assert m32.layers[0]["wq"].dtype == np.float32
    d = np.abs(a.astype(np.float64) - b)
    assert 0 < d.max() < 2e-2
    assert np.linalg.norm(a - b) / np.linalg.norm(a) < 1e-2
