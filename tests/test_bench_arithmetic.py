"""The algorithmic work bench.py divides by (CPU only).

The roofline fractions in the bench line are algorithmic bytes or flops over
measured time, so the arithmetic behind them is pinned here against figures
worked out independently from the model shapes and workload recipes: the
per-token KV bytes, the decode weight bytes of each shape, and the per-step
bytes and prefill flops of the benchmarked configurations (8B with 25 agents,
70B with 128 agents), with their stated tolerances of rounding.
"""

import numpy as np

import bench
from paper_2411_03519_amd import synth

S8, S70, ST = synth.LLAMA3_8B, synth.LLAMA3_70B, synth.TINY


def test_llama3_8b_layer_parameters_by_matrix():
    # q 4096x4096, k and v 1024x4096 each, o 4096x4096, gate, up and down 14336x4096 each
    per_layer = 4096 * 4096 + 2 * 1024 * 4096 + 4096 * 4096 + 3 * 14336 * 4096
    assert per_layer == 218_103_808
    assert bench.layer_params(S8) == per_layer
    # 70B: q 8192x8192, k and v 1024x8192, o 8192x8192, gate/up/down 28672x8192
    assert bench.layer_params(S70) == 2 * 8192 * 8192 + 2 * 1024 * 8192 + 3 * 28672 * 8192


def test_kv_bytes_per_token():
    # K and V, bf16, every layer: 2 layers x 2 heads x 64 (tiny), 32 x 8 x 128 (8B), 80 x 8 x 128 (70B)
    assert bench.kv_token_bytes(ST) == 1024
    assert bench.kv_token_bytes(S8) == 131_072
    assert bench.kv_token_bytes(S70) == 327_680


def test_decode_weight_bytes():
    # every projection and the LM head once per step (the embedding is a gather)
    assert abs(bench.decode_weight_bytes(S8) - 15.01e9) < 0.01e9
    assert abs(bench.decode_weight_bytes(S70) - 139.0e9) < 0.05e9
    assert abs(bench.decode_weight_bytes(ST) - 5.0e6) < 0.05e6


def test_decode_step_bytes_of_the_25_agent_batch():
    prompts, n_new = synth.llama8b_agent_batch(0)
    lens = np.array([len(p) for p in prompts])
    assert lens.sum() == 31527
    per_step = sum(bench.decode_step_bytes(S8, lens + k) for k in range(n_new - 1)) / (n_new - 1)
    assert abs(per_step - 19.26e9) < 0.01e9
    # the first step by its parts: weights, 31527 context tokens of KV read,
    # 25 tokens of KV written, 25 rows of fp32 logits
    first = bench.decode_step_bytes(S8, lens)
    assert first == bench.decode_weight_bytes(S8) + (31527 + 25) * 131_072 + 25 * 128_256 * 4


def test_prefill_flops_of_the_25_agent_batch():
    prompts, _ = synth.llama8b_agent_batch(0)
    items = [np.arange(len(p)) for p in prompts]
    flops = bench.prefill_flops(S8, items, 25)
    assert abs(flops - 4.52e14) < 0.01e14
    # 13.96 GFLOP of linear layers per token and 524,288 flop per (query,
    # visible key) pair (4 x 32 layers x 32 heads x 128), plus 25 LM-head rows
    keys = sum(int(L) * (int(L) + 1) // 2 for L in map(len, prompts))
    linear = 2 * 32 * 218_103_808 * 31527
    assert abs(linear / 31527 - 13.96e9) < 0.005e9
    assert flops == linear + 524_288 * keys + 2 * 25 * 128_256 * 4096


def test_decode_step_bytes_of_the_70b_batch():
    ctx, n_new = synth.llama70b_agent_batch(0)
    lens = np.array([len(c) for c in ctx])
    assert lens.min() >= 1024 and lens.max() <= 3072 and len(lens) == 128
    per_step = sum(bench.decode_step_bytes(S70, lens + k) for k in range(n_new - 1)) / (n_new - 1)
    # 139.0 GB of weights plus about 84 GB of KV for contexts averaging ~2000 tokens
    assert abs(per_step - 222.8e9) < 0.01 * 222.8e9


def test_code_only_drops_comments_and_keeps_literals():
    src = ('int a = 1;   // a note\n/* a block\n   comment */ const char* s = "x // y /* z */";\n'
           "char c = '\"'; char d = '\\''; asm(\"s_nop 0\");\n")
    assert bench.code_only(src) == ('int a = 1; const char* s = "x // y /* z */"; char c = \'"\'; '
                                    "char d = '\\''; asm(\"s_nop 0\");")


def test_source_hash_ignores_comment_edits(tmp_path, monkeypatch):
    """The hash that marks a traffic measurement stale follows code changes
    only: an edited comment keeps it, a changed expression does not."""
    a, b, c = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    a.write_text("// v1\nx = y + 1; /* note */\n")
    b.write_text("// v2, reworded\nx = y + 1;   /* other note */\n")
    c.write_text("// v1\nx = y + 2; /* note */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.source_hash(["a.hip"]) == bench.source_hash(["b.hip"])
    assert bench.source_hash(["a.hip"]) != bench.source_hash(["c.hip"])
