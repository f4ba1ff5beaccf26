"""Plausible mistakes planted in the oracle (on the CPU) must fail a pin.

Each case swaps one oracle building block for a subtly wrong version (wrong
pairing, sign, index, operand, scale, mask or rounding) and checks that the
pin suite of ``test_oracle_pins.py`` notices.
"""

import numpy as np
import pytest

import oracle.llama as L
from paper_2411_03519_amd import synth
from tests.test_oracle_pins import MICRO, oracle_vs_hf_error
import tests.test_oracle_pins as pins


def rope_interleaved(u, positions, base):
    hd = u.shape[-1]
    theta = base ** (-2.0 * np.arange(hd // 2) / hd)
    phi = np.asarray(positions, float)[:, None] * theta[None, :]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    a, b = u[..., 0::2], u[..., 1::2]
    out = np.empty_like(u)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def rope_wrong_sign(u, positions, base):
    hd = u.shape[-1]
    half = hd // 2
    theta = base ** (-2.0 * np.arange(half) / hd)
    phi = np.asarray(positions, float)[:, None] * theta[None, :]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c + b * s, -a * s + b * c], axis=-1)


def rope_wrong_freq(u, positions, base):
    hd = u.shape[-1]
    half = hd // 2
    theta = base ** (-1.0 * np.arange(half) / hd)
    phi = np.asarray(positions, float)[:, None] * theta[None, :]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def attention_factory(kv_map=None, scale=None, strict_mask=False):
    def attn(q, k, v, q_pos):
        n, nq, hd = q.shape
        nkv = k.shape[1]
        group = nq // nkv
        ctx = k.shape[0]
        if strict_mask:
            visible = np.arange(ctx)[None, :] < np.asarray(q_pos)[:, None]
            visible[:, 0] = True
        else:
            visible = np.arange(ctx)[None, :] <= np.asarray(q_pos)[:, None]
        out = np.empty((n, nq, hd))
        for j in range(nq):
            kvh = kv_map(j, nq, nkv) if kv_map else j // group
            sc = (q[:, j] @ k[:, kvh].T) * (scale(hd) if scale else 1 / np.sqrt(hd))
            sc = np.where(visible, sc, -np.inf)
            out[:, j] = L.softmax_rows(sc) @ v[:, kvh]
        return out
    return attn


def rms_no_gain(x, g, eps):
    return x / np.sqrt(np.mean(x * x, -1, keepdims=True) + eps)


def rms_no_eps_mean_abs(x, g, eps):
    return x / (np.mean(np.abs(x), -1, keepdims=True) + eps) * g


def swiglu_swapped(gate, up):
    return L.silu(up) * gate


def softmax_no_norm(s):
    m = np.max(s, -1, keepdims=True)
    return np.exp(s - m) / (np.exp(s - m).sum(-1, keepdims=True) + 1.0)


def bf16_truncate(x):
    x = np.asarray(x, np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    return np.ldexp(np.trunc(np.ldexp(x, 8 - e)), e - 8)


def silu_sigmoid_only(z):
    return 1.0 / (1.0 + np.exp(-z))


MUTATIONS = {
    "rope_interleaved_pairs": ("rope_rotate", rope_interleaved),
    "rope_wrong_sign": ("rope_rotate", rope_wrong_sign),
    "rope_wrong_frequency": ("rope_rotate", rope_wrong_freq),
    "gqa_modulo_mapping": ("causal_gqa_attention", attention_factory(kv_map=lambda j, nq, nkv: j % nkv)),
    "attention_scale_1_over_hd": ("causal_gqa_attention", attention_factory(scale=lambda hd: 1.0 / hd)),
    "causal_mask_off_by_one": ("causal_gqa_attention", attention_factory(strict_mask=True)),
    "rmsnorm_drops_gain": ("rms_norm", rms_no_gain),
    "rmsnorm_mean_abs": ("rms_norm", rms_no_eps_mean_abs),
    "swiglu_operands_swapped": ("swiglu", swiglu_swapped),
    "softmax_bad_normaliser": ("softmax_rows", softmax_no_norm),
    "silu_is_sigmoid": ("silu", silu_sigmoid_only),
}


def _pins_fail(monkeypatch) -> bool:
    """True if any pin that covers the whole model or the patched block fails."""
    checks = [
        lambda: oracle_vs_hf_error(MICRO) < 1e-6,
        lambda: oracle_vs_hf_error(dict(MICRO, d_model=64, n_heads=8, n_kv_heads=2, head_dim=16,
                                        rope_base=500000.0), seed=12, n=40) < 1e-6,
    ]
    for fn in (pins.test_rope_as_complex_rotation, pins.test_attention_brute_force_loops,
               pins.test_rms_norm_matches_torch, pins.test_softmax_rows_sum_to_one_and_shift_invariance,
               pins.test_silu_matches_torch_and_limits, pins.test_attention_matches_torch_sdpa_with_prior_context):
        checks.append(lambda fn=fn: fn() is None)
    for c in checks:
        try:
            if not c():
                return True
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, bad = MUTATIONS[name]
    monkeypatch.setattr(L, attr, bad)
    monkeypatch.setattr(pins, attr, bad, raising=False)
    assert _pins_fail(monkeypatch), f"mutation {name} passed every pin"


def test_unmutated_oracle_passes_same_checks(monkeypatch):
    assert not _pins_fail(monkeypatch)


def test_truncating_bf16_is_caught(monkeypatch):
    monkeypatch.setattr(pins, "bf16_round", bf16_truncate)
    with pytest.raises(AssertionError):
        pins.test_bf16_round_matches_torch_on_float32_inputs()


def test_dropped_residual_is_caught(monkeypatch):
    orig = L.OracleModel.block

    def block_no_ffn_residual(self, li, x, cache, positions):
        y = orig(self, li, x, cache, positions)
        W = self.layers[li]
        # undo "x +": return only the FFN branch added to the attention output
        h2 = self.q(L.rms_norm(x, W["ffn_norm"], self.shape.rms_eps))
        return y - 0.5 * (self.q(L.swiglu(h2 @ W["wgate"].T, h2 @ W["wup"].T)) @ W["wdown"].T)

    monkeypatch.setattr(L.OracleModel, "block", block_no_ffn_residual)
    assert oracle_vs_hf_error(MICRO) > 1e-6


def test_transposed_weight_is_caught(monkeypatch):
    # square wq/wo in a d_model == n_heads*head_dim shape: a transposed operand still runs
    orig_init = L.OracleModel.__init__

    def init_t(self, shape, weights, quantize=True):
        orig_init(self, shape, weights, quantize)
        for lw in self.layers:
            lw["wo"] = lw["wo"].T.copy()

    monkeypatch.setattr(L.OracleModel, "__init__", init_t)
    assert oracle_vs_hf_error(MICRO) > 1e-6
    _ = synth  # inputs come from the shared generator
