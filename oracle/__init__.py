"""Oracle for the batched agent-LLM forward pass — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product (the HIP library
``libmetro.so`` and its Python binding) never imports, links or calls it, and
this package imports nothing from the product.

What it computes
----------------
AI Metropolis (arXiv 2411.03519) spends about 95% of simulation time in LLM
inference (§1) and serves Llama-3 instruct models (8B and 70B) with a batching
engine, replaying fixed-length generations without an end-of-sequence stop
(§4.1).  The paper does not define the
network; the network computed here is the public Llama decoder:

* token embedding, untied LM head, no biases, causal self-attention;
* RMSNorm (Zhang & Sennrich 2019) before attention and before the FFN;
* grouped-query attention (Ainslie et al. 2023) with contiguous head groups;
* rotary position embedding (Su et al. 2021) in the rotate-half pairing
  ``(i, i + head_dim/2)`` used by the Llama reference code;
* SwiGLU feed-forward (Shazeer 2020): ``W_down(silu(W_gate h) * W_up h)``;
* greedy decoding: the lowest index among the maximal logits.

Precision contract
------------------
Arithmetic is float64, so the oracle's own rounding error is far below that of
an fp32-accumulating GPU path.  The values a bf16 implementation stores in bf16
are rounded to bf16 (round to nearest, ties to even) at exactly these points:
the weights; the normalised activation ``h`` that feeds a projection; q, k and v
after RoPE (so the KV cache holds bf16 values); the attention output ``o`` that
feeds ``W_o``; the SwiGLU product that feeds ``W_down``.  Everything else
(residual stream, RMS statistics, scores, softmax, attention accumulation)
stays in float64; logits are handed out rounded to float32 and the argmax is
taken on those float32 values.  ``quantize=False`` skips the bf16 points and
gives the plain float64 Llama function, the form compared with an independent
implementation in the tests.

Every function here is pinned by ``tests/test_oracle_*.py`` against closed
forms, invariants, brute force and independent library routines.
"""

from .llama import (  # noqa: F401
    LlamaShape,
    OracleModel,
    ContiguousKV,
    PagedKV,
    bf16_round,
    bf16_bits_to_f64,
    rms_norm,
    rope_rotate,
    softmax_rows,
    causal_gqa_attention,
    silu,
    swiglu,
    greedy_argmax,
)
