"""Pin of the oracle's bf16 storage points (CPU only).

The precision contract rounds to bfloat16 at exactly these points and nowhere
else: the normalised activation entering each projection (attention and FFN
RMSNorm outputs, final RMSNorm output), q and k after the rotary embedding, v,
the attention output o, and the SwiGLU product.  The residual stream, scores,
softmax weights and logits stay wide.

``contract_logits`` below evaluates that contract a second time, in torch
float64, with torch's own building blocks where the oracle has numpy ones:
``rms_norm``, RoPE as a complex multiplication of the (u_i, u_{i+hd/2}) pairs,
``scaled_dot_product_attention`` with a causal mask over KV heads repeated per
group, ``silu``.  Its bf16 rounding goes float64 -> float32 rounded to odd ->
bfloat16 by torch, which is correctly rounded for float64 inputs (Boldo &
Melquiond, "Emulation of FMA and correctly rounded sums: proved algorithms
using rounding to odd", IEEE TC 2008), and shares nothing with the oracle's
``bf16_round``.  The quantised oracle must agree with it to 1e-12 relative
(float64 summation order only; a single moved, dropped or added storage point
changes logits by ~1e-3).

The second half plants such mistakes in the oracle's block -- each drops,
adds or moves one storage point -- and checks that the pin notices every one.
"""

import math
import sys

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.llama as L
from oracle import LlamaShape, OracleModel, bf16_bits_to_f64
from paper_2411_03519_amd import synth

SHAPES = {
    # GQA group 2, head dim 8
    "micro": dict(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn_dim=48, vocab=97,
                  rope_base=10000.0, rms_eps=1e-5),
    # group 4, head dim 16, Llama-3 RoPE base
    "wider": dict(n_layers=2, d_model=64, n_heads=8, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab=131,
                  rope_base=500000.0, rms_eps=1e-5),
}


# ----------------------------------------------------------------------------
# Independent evaluation of the contract in torch float64
# ----------------------------------------------------------------------------

def to_bf16(x: torch.Tensor) -> torch.Tensor:
    """float64 -> nearest bfloat16 (ties to even), returned as float64.

    float64 -> float32 rounded to odd keeps the sticky information of the
    discarded bits in the last float32 bit, so torch's float32 -> bfloat16
    round-to-nearest-even then gives the correctly rounded result."""
    x = x.to(torch.float64)
    f = x.to(torch.float32)                       # nearest float32
    inexact = f.to(torch.float64) != x
    away = f.to(torch.float64).abs() > x.abs()    # rounded away from zero: step back
    bits = f.view(torch.int32)
    bits = torch.where(inexact & away, bits - 1, bits)
    bits = torch.where(inexact, bits | 1, bits)
    return bits.view(torch.float32).to(torch.bfloat16).to(torch.float64)


def rope_complex(u: torch.Tensor, pos: torch.Tensor, base: float) -> torch.Tensor:
    """u [n, heads, hd]: the pair (u_i, u_{i+hd/2}) as one complex number turned
    by pos * base^(-2i/hd)."""
    hd = u.shape[-1]
    half = hd // 2
    inv = torch.tensor([base ** (-2.0 * i / hd) for i in range(half)], dtype=torch.float64)
    rot = torch.polar(torch.ones(len(pos), half, dtype=torch.float64), pos[:, None].double() * inv[None, :])
    z = torch.complex(u[..., :half], u[..., half:]) * rot[:, None, :]
    return torch.cat([z.real, z.imag], dim=-1)


def contract_logits(cfg: dict, weights: dict, tokens) -> np.ndarray:
    """Logits of every position of ``tokens`` under the precision contract."""
    w = lambda a: torch.tensor(bf16_bits_to_f64(a))  # noqa: E731  (bf16 values, exact in float64)
    d, nq, nkv, hd = cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    eps = cfg["rms_eps"]
    toks = torch.tensor(np.asarray(tokens), dtype=torch.int64)
    n = len(toks)
    pos = torch.arange(n)
    x = w(weights["embed"])[toks]
    for lw in weights["layers"]:
        h = to_bf16(F.rms_norm(x, (d,), w(lw["attn_norm"]), eps=eps))
        q = to_bf16(rope_complex((h @ w(lw["wq"]).T).view(n, nq, hd), pos, cfg["rope_base"]))
        k = to_bf16(rope_complex((h @ w(lw["wk"]).T).view(n, nkv, hd), pos, cfg["rope_base"]))
        v = to_bf16((h @ w(lw["wv"]).T).view(n, nkv, hd))
        g = nq // nkv
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.repeat_interleave(g, dim=1).transpose(0, 1),
                                           v.repeat_interleave(g, dim=1).transpose(0, 1), is_causal=True)
        o = to_bf16(o.transpose(0, 1).reshape(n, nq * hd))
        x = x + o @ w(lw["wo"]).T
        h2 = to_bf16(F.rms_norm(x, (d,), w(lw["ffn_norm"]), eps=eps))
        a = to_bf16(F.silu(h2 @ w(lw["wgate"]).T) * (h2 @ w(lw["wup"]).T))
        x = x + a @ w(lw["wdown"]).T
    hf = to_bf16(F.rms_norm(x, (d,), w(weights["final_norm"]), eps=eps))
    return (hf @ w(weights["lm_head"]).T).numpy()


def inputs(name: str, seed: int, n: int):
    cfg = SHAPES[name]
    W = synth.llama_weights(cfg, seed, norm="random")
    toks = np.random.default_rng(seed).integers(0, cfg["vocab"], n)
    return cfg, W, toks


def oracle_vs_contract(cfg, W, toks):
    """(relative error of the oracle's float64 logits, largest error of its
    float32 output in float32 ulps of the contract's logits).

    ``forward`` returns float32 logits, so the float64 values are taken from
    its blocks (``hidden_layers``) and the same head; the float32 output itself,
    final RMSNorm rounding included, must then be the contract's value to
    within one float32 rounding."""
    ref = contract_logits(cfg, W, toks)
    om = OracleModel(LlamaShape(**cfg), W)
    x = om.hidden_layers(om.new_cache(), toks, cfg["n_layers"])
    ours = om.q(L.rms_norm(x, om.final_norm, cfg["rms_eps"])) @ om.lm_head.T
    rel = float(np.max(np.abs(ours - ref)) / np.max(np.abs(ref)))
    out32 = om.forward(om.new_cache(), toks).astype(np.float64)
    ulps = float(np.max(np.abs(out32 - ref) / np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)))
    return rel, ulps


PIN_CASES = (("micro", 31, 23), ("wider", 32, 41))


def pin_holds() -> bool:
    for nm, seed, n in PIN_CASES:
        rel, ulps = oracle_vs_contract(*inputs(nm, seed, n))
        if not (rel < 1e-12 and ulps <= 1.0):
            return False
    return True


# ----------------------------------------------------------------------------
# The pin and the checks that make it trustworthy
# ----------------------------------------------------------------------------

def test_to_bf16_is_correctly_rounded():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))
    # float64 values just above and below bf16 midpoints: where double rounding
    # through float32 would go wrong
    b = torch.tensor(x[:2000]).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    _, e = np.frexp(b)
    mid = b + np.ldexp(1.0, e - 9)
    x = np.concatenate([x, mid, mid + np.ldexp(1.0, e - 40), mid - np.ldexp(1.0, e - 40), b])
    got = to_bf16(torch.tensor(x)).numpy()
    # brute force: of the bf16 neighbours of x, the nearer one (the even one on a tie)
    for xi, gi in zip(x[::7], got[::7]):
        m, ex = math.frexp(xi)
        ulp = math.ldexp(1.0, ex - 8)
        lo = math.floor(xi / ulp) * ulp
        hi = lo + ulp
        dl, dh = xi - lo, hi - xi
        if dl < dh:
            want = lo
        elif dh < dl:
            want = hi
        else:
            want = lo if (round(lo / ulp) % 2 == 0) else hi
        assert gi == want, (xi, gi, want)


def test_rope_complex_matches_rotate_half_by_hand():
    # hd = 4, position 2, base 100: pairs (0, 2) by angle 2, (1, 3) by angle 2/10
    u = torch.tensor([[[1.0, 2.0, 3.0, 4.0]]], dtype=torch.float64)
    got = rope_complex(u, torch.tensor([2]), 100.0)[0, 0].numpy()
    a0, a1 = 2.0, 0.2
    want = [math.cos(a0) - 3 * math.sin(a0), 2 * math.cos(a1) - 4 * math.sin(a1),
            math.sin(a0) + 3 * math.cos(a0), 2 * math.sin(a1) + 4 * math.cos(a1)]
    np.testing.assert_allclose(got, want, rtol=1e-15)


def test_contract_without_rounding_is_the_transformers_llama(monkeypatch):
    # with to_bf16 the identity, contract_logits is a plain float64 Llama:
    # it must agree with the independent transformers implementation
    from tests.test_oracle_pins import hf_logits
    cfg, W, toks = inputs("wider", 33, 29)
    monkeypatch.setattr(sys.modules[__name__], "to_bf16", lambda t: t)
    ours = contract_logits(cfg, W, toks)
    ref = hf_logits(cfg, W, toks)
    # transformers forms the rotary cos/sin tables in float32: agreement to ~1e-7
    assert np.max(np.abs(ours - ref)) / np.max(np.abs(ref)) < 1e-6


@pytest.mark.parametrize("name,seed,n", PIN_CASES)
def test_quantised_oracle_matches_the_contract(name, seed, n):
    rel, ulps = oracle_vs_contract(*inputs(name, seed, n))
    assert rel < 1e-12, rel
    assert ulps <= 1.0, ulps


def test_storage_points_are_not_a_no_op():
    # the pin has teeth: the contract differs from the unrounded network by
    # far more than its threshold
    cfg, W, toks = inputs("micro", 31, 23)
    om = OracleModel(LlamaShape(**cfg), W, quantize=False)
    x = om.hidden_layers(om.new_cache(), toks, cfg["n_layers"])
    exact = L.rms_norm(x, om.final_norm, cfg["rms_eps"]) @ om.lm_head.T
    ref = contract_logits(cfg, W, toks)
    assert np.max(np.abs(exact - ref)) / np.max(np.abs(ref)) > 1e-5


# ----------------------------------------------------------------------------
# Planted storage-point mistakes
# ----------------------------------------------------------------------------

def block_with(points: frozenset):
    """The oracle's decoder block with bf16 rounding at ``points`` only.

    Names: h (attention RMSNorm output), q_pre/k_pre (before RoPE), q/k (after
    RoPE), v, o, x_mid (residual after attention), h2 (FFN RMSNorm output),
    gate/up (separately), a (SwiGLU product), x_out (residual after the FFN),
    p (softmax weights)."""
    def block(self, li, x, cache, positions):
        S = self.shape
        W = self.layer(li)
        r = lambda name, t: self.q(t) if name in points else t  # noqa: E731
        n = x.shape[0]
        h = r("h", L.rms_norm(x, W["attn_norm"], S.rms_eps))
        q = r("q_pre", (h @ W["wq"].T).reshape(n, S.n_heads, S.head_dim))
        k = r("k_pre", (h @ W["wk"].T).reshape(n, S.n_kv_heads, S.head_dim))
        v = r("v", (h @ W["wv"].T).reshape(n, S.n_kv_heads, S.head_dim))
        q = r("q", L.rope_rotate(q, positions, S.rope_base))
        k = r("k", L.rope_rotate(k, positions, S.rope_base))
        cache.write(li, positions, k, v)
        kc, vc = cache.read(li)
        if "p" in points:
            soft = L.softmax_rows
            L.softmax_rows = lambda s: self.q(soft(s))
            try:
                att = L.causal_gqa_attention(q, kc, vc, positions)
            finally:
                L.softmax_rows = soft
        else:
            att = L.causal_gqa_attention(q, kc, vc, positions)
        o = r("o", att.reshape(n, S.n_heads * S.head_dim))
        x = r("x_mid", x + o @ W["wo"].T)
        h2 = r("h2", L.rms_norm(x, W["ffn_norm"], S.rms_eps))
        a = r("a", L.swiglu(r("gate", h2 @ W["wgate"].T), r("up", h2 @ W["wup"].T)))
        return r("x_out", x + a @ W["wdown"].T)
    return block


CONTRACT = frozenset({"h", "q", "k", "v", "o", "h2", "a"})

STORAGE_MUTATIONS = {
    "drop_h": CONTRACT - {"h"},
    "drop_q": CONTRACT - {"q"},
    "drop_k": CONTRACT - {"k"},
    "drop_v": CONTRACT - {"v"},
    "drop_o": CONTRACT - {"o"},
    "drop_h2": CONTRACT - {"h2"},
    "drop_swiglu_product": CONTRACT - {"a"},
    "move_qk_before_rope": (CONTRACT - {"q", "k"}) | {"q_pre", "k_pre"},
    "move_product_to_gate_and_up": (CONTRACT - {"a"}) | {"gate", "up"},
    "add_residual_after_attention": CONTRACT | {"x_mid"},
    "add_residual_after_ffn": CONTRACT | {"x_out"},
    "add_softmax_weights": CONTRACT | {"p"},
}


def test_block_builder_with_the_contract_is_the_oracle(monkeypatch):
    cfg, W, toks = inputs("micro", 31, 23)
    om = OracleModel(LlamaShape(**cfg), W)
    want = om.forward(om.new_cache(), toks)
    monkeypatch.setattr(L.OracleModel, "block", block_with(CONTRACT))
    om2 = OracleModel(LlamaShape(**cfg), W)
    np.testing.assert_array_equal(om2.forward(om2.new_cache(), toks), want)


@pytest.mark.parametrize("name", sorted(STORAGE_MUTATIONS))
def test_moved_dropped_or_added_storage_point_is_caught(name, monkeypatch):
    monkeypatch.setattr(L.OracleModel, "block", block_with(STORAGE_MUTATIONS[name]))
    assert not pin_holds(), f"storage-point mutation {name} passed the pin"


def test_dropped_final_norm_rounding_is_caught(monkeypatch):
    # the final RMSNorm output is rounded in forward(); the mistake planted there
    def forward_unrounded_head(self, cache, tokens, logits_for=None):
        tokens = np.asarray(tokens, dtype=np.int64)
        x = self.hidden_layers(cache, tokens, self.shape.n_layers)
        if logits_for is not None:
            x = x[logits_for]
        hf = L.rms_norm(x, self.final_norm, self.shape.rms_eps)
        return self.lm_head_logits(hf).astype(np.float32)

    monkeypatch.setattr(L.OracleModel, "forward", forward_unrounded_head)
    assert not pin_holds()
