"""Plain float64 CPU Llama decoder: the oracle (test infrastructure only).

See the package docstring for what is computed and the precision contract.
The code follows the published definitions step by step, one sequence at a
time, with no batching, blocking or fusion.
"""

from __future__ import annotations

import math
import os
from dataclasses import dataclass

import numpy as np


# ----------------------------------------------------------------------------
# Shapes and number formats
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class LlamaShape:
    """Hyper-parameters of a Llama-style decoder (Llama-3 8B / 70B family)."""

    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads


def bf16_round(x) -> np.ndarray:
    """Round to the nearest bfloat16 value, ties to even; returned as float64.

    bfloat16 keeps 8 significant bits (1 implicit + 7 stored) and the float32
    exponent range.  Writing ``x = m * 2**e`` with ``0.5 <= |m| < 1`` the
    spacing of bf16 values near ``x`` is ``2**(e - 8)``; below the smallest
    normal ``2**-126`` (``e < -125``) it stays ``2**-133`` (subnormals).
    ``np.round`` rounds halfway cases to even.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    r = np.ldexp(np.round(np.ldexp(x, 8 - e)), e - 8)
    return np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, x), r)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Decode bfloat16 storage (uint16: the top half of a float32) exactly."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# Building blocks (each one a published definition)
# ----------------------------------------------------------------------------

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm (Zhang & Sennrich 2019) over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_rotate(u: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding (Su et al. 2021), rotate-half pairing.

    ``u`` is ``[n, heads, hd]``; token ``t`` sits at absolute position
    ``positions[t]``.  For ``i < hd/2`` the pair ``(u_i, u_{i+hd/2})`` is turned
    by the angle ``p * base**(-2i/hd)``.
    """
    hd = u.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * i / hd)
    phi = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    c = np.cos(phi)[:, None, :].astype(u.dtype)
    s = np.sin(phi)[:, None, :].astype(u.dtype)
    a = u[..., :half]
    b = u[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax with the row maximum subtracted first (rows of -inf excluded)."""
    m = np.max(s, axis=-1, keepdims=True)
    w = np.exp(s - m)
    return w / np.sum(w, axis=-1, keepdims=True)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         q_pos: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention for one sequence.

    ``q`` is ``[n, nq, hd]`` for queries at absolute positions ``q_pos``;
    ``k`` and ``v`` are ``[ctx, nkv, hd]`` holding positions ``0 .. ctx-1``.
    Query head ``j`` reads kv head ``j // (nq // nkv)`` (contiguous groups).
    A query at position ``p`` sees keys ``0 .. p``; scores are scaled by
    ``1/sqrt(hd)``.
    """
    n, nq, hd = q.shape
    ctx, nkv, _ = k.shape
    group = nq // nkv
    visible = np.arange(ctx)[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty((n, nq, hd), dtype=q.dtype)
    for j in range(nq):
        kvh = j // group
        s = (q[:, j, :] @ k[:, kvh, :].T) / math.sqrt(hd)
        s = np.where(visible, s, -np.inf)
        out[:, j, :] = softmax_rows(s) @ v[:, kvh, :]
    return out


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU / swish: z * sigmoid(z) = z / (1 + exp(-z))."""
    return z / (1.0 + np.exp(-z))


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """SwiGLU combination (Shazeer 2020): silu(gate) * up."""
    return silu(gate) * up


def greedy_argmax(logits: np.ndarray) -> np.ndarray:
    """Greedy choice per row: the lowest index among the maximal values."""
    return np.argmax(logits, axis=-1).astype(np.int64)


# ----------------------------------------------------------------------------
# KV caches: contiguous (the definition) and paged (same values, paged storage)
# ----------------------------------------------------------------------------

class ContiguousKV:
    """Per-sequence KV cache: for each layer, k and v as ``[ctx, nkv, hd]``."""

    def __init__(self, shape: LlamaShape):
        self.shape = shape
        self.k = [None] * shape.n_layers
        self.v = [None] * shape.n_layers
        self.length = 0

    def write(self, layer: int, positions: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
        if self.k[layer] is None:
            assert positions[0] == 0, "positions must append"
            self.k[layer], self.v[layer] = k.copy(), v.copy()
            return
        assert positions[0] == self.k[layer].shape[0], "positions must append"
        self.k[layer] = np.concatenate([self.k[layer], k], axis=0)
        self.v[layer] = np.concatenate([self.v[layer], v], axis=0)

    def read(self, layer: int):
        return self.k[layer], self.v[layer]

    def advance(self, n: int) -> None:
        self.length += n


class PagedKV:
    """KV cache in fixed-size pages of a shared pool, reached by a block table.

    Page ``b`` holds positions ``page*b .. page*b + page - 1`` of the sequence
    for every layer.  Pages are taken from ``free_pages`` in the given order,
    so a test can hand in a shuffled free list.  ``read`` gathers the pages of
    the block table back into ``[ctx, nkv, hd]`` arrays.
    """

    def __init__(self, shape: LlamaShape, n_pages: int, page: int, free_pages):
        self.shape = shape
        self.page = page
        self.pool = None  # allocated on first write, in the arithmetic dtype
        self.n_pages = n_pages
        self.free = list(free_pages)
        self.block_table: list[int] = []
        self.filled = [0] * shape.n_layers
        self.length = 0

    def write(self, layer: int, positions: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
        if self.pool is None:
            S = self.shape
            self.pool = np.zeros((self.n_pages, S.n_layers, 2, self.page, S.n_kv_heads, S.head_dim), dtype=k.dtype)
        for t, p in enumerate(positions):
            b, off = divmod(int(p), self.page)
            while b >= len(self.block_table):
                self.block_table.append(self.free.pop(0))
            pg = self.block_table[b]
            self.pool[pg, layer, 0, off] = k[t]
            self.pool[pg, layer, 1, off] = v[t]
        self.filled[layer] = max(self.filled[layer], int(positions[-1]) + 1)

    def read(self, layer: int):
        ctx = self.filled[layer]
        pages = self.pool[self.block_table, layer]              # [nb, 2, page, nkv, hd]
        k = pages[:, 0].reshape(-1, self.shape.n_kv_heads, self.shape.head_dim)[:ctx]
        v = pages[:, 1].reshape(-1, self.shape.n_kv_heads, self.shape.head_dim)[:ctx]
        return k, v

    def advance(self, n: int) -> None:
        self.length += n


# ----------------------------------------------------------------------------
# The model
# ----------------------------------------------------------------------------

_LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wgate", "wup", "wdown")


class OracleModel:
    """Llama-style decoder evaluated one sequence at a time.

    ``weights`` is a dict: ``embed [V,d]``, ``final_norm [d]``, ``lm_head [V,d]``
    and ``layers``: a list of dicts with ``attn_norm [d]``, ``wq [nq*hd, d]``,
    ``wk [nkv*hd, d]``, ``wv [nkv*hd, d]``, ``wo [d, nq*hd]``, ``ffn_norm [d]``,
    ``wgate [F, d]``, ``wup [F, d]``, ``wdown [d, F]`` (all ``[out, in]``).
    Arrays of dtype uint16 are read as bfloat16 bit patterns; any other dtype is
    taken as real values (rounded to bf16 when ``quantize``).

    ``dtype`` is the arithmetic: float64 (the oracle) or float32, the same
    function evaluated the way an fp32-accumulating implementation would; the
    difference between the two measures how far legitimate fp32 rounding alone
    moves the result (the noise floor a tolerance must allow for).
    """

    def __init__(self, shape: LlamaShape, weights: dict, quantize: bool = True, dtype=np.float64,
                 lazy: bool = False):
        """``lazy``: keep ``weights`` as given and convert each layer's matrices
        (and the embedding rows and LM-head rows in use) to the arithmetic dtype
        when they are used, so that a full-depth 8B or 70B model fits in host
        memory.  The values, and so every result, are the same either way."""
        self.shape = shape
        self.quantize = quantize
        self.dtype = np.dtype(dtype)
        self.lazy = lazy
        assert len(weights["layers"]) == shape.n_layers
        self.final_norm = self.load(weights["final_norm"])
        if lazy:
            self._raw = weights
            self._cur = (-1, None)
        else:
            self.embed = self.load(weights["embed"])
            self.lm_head = self.load(weights["lm_head"])
            self.layers = [{k: self.load(lw[k]) for k in _LAYER_KEYS} for lw in weights["layers"]]

    def load(self, a) -> np.ndarray:
        """Weights in the arithmetic dtype.  uint16 arrays are bf16 bit patterns,
        whose values bf16 rounding leaves unchanged; other arrays are real
        values, rounded to bf16 when ``quantize``."""
        a = np.asarray(a)
        if a.dtype != np.uint16:
            return self.q(a.astype(np.float64))
        if a.size < (1 << 22):
            return bf16_bits_to_f64(a).astype(self.dtype, copy=False)
        # large matrices: decode row blocks on several threads (numpy releases the GIL)
        from concurrent.futures import ThreadPoolExecutor
        out = np.empty(a.shape, dtype=self.dtype)
        rows = a.reshape(a.shape[0], -1)
        flat = out.reshape(a.shape[0], -1)
        step = max(1, rows.shape[0] // 64)

        def work(r0):
            flat[r0:r0 + step] = bf16_bits_to_f64(rows[r0:r0 + step])
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, range(0, rows.shape[0], step)))
        return out

    def layer(self, li: int) -> dict:
        if not self.lazy:
            return self.layers[li]
        if self._cur[0] != li:
            self._cur = (-1, None)  # free the previous layer first
            self._cur = (li, {k: self.load(self._raw["layers"][li][k]) for k in _LAYER_KEYS})
        return self._cur[1]

    def embed_rows(self, tokens) -> np.ndarray:
        if not self.lazy:
            return self.embed[tokens]
        return self.load(np.asarray(self._raw["embed"])[tokens])

    def lm_head_logits(self, hf) -> np.ndarray:
        """``hf @ W_lm^T``; in lazy mode one block of vocabulary rows at a time
        (each logit is the same dot product either way)."""
        if not self.lazy:
            return hf @ self.lm_head.T
        W = np.asarray(self._raw["lm_head"])
        out = np.empty((hf.shape[0], W.shape[0]), dtype=np.result_type(hf.dtype, self.dtype))
        for r0 in range(0, W.shape[0], 16384):
            out[:, r0:r0 + 16384] = hf @ self.load(W[r0:r0 + 16384]).T
        return out

    def q(self, x):
        """The bf16 storage points of the precision contract (identity if not
        quantize), returned in the arithmetic dtype."""
        return (bf16_round(x) if self.quantize else np.asarray(x)).astype(self.dtype, copy=False)

    def new_cache(self) -> ContiguousKV:
        return ContiguousKV(self.shape)

    # -- one decoder block ----------------------------------------------------
    def block(self, li: int, x: np.ndarray, cache, positions: np.ndarray) -> np.ndarray:
        S = self.shape
        W = self.layer(li)
        n = x.shape[0]
        h = self.q(rms_norm(x, W["attn_norm"], S.rms_eps))
        q = (h @ W["wq"].T).reshape(n, S.n_heads, S.head_dim)
        k = (h @ W["wk"].T).reshape(n, S.n_kv_heads, S.head_dim)
        v = (h @ W["wv"].T).reshape(n, S.n_kv_heads, S.head_dim)
        q = self.q(rope_rotate(q, positions, S.rope_base))
        k = self.q(rope_rotate(k, positions, S.rope_base))
        v = self.q(v)
        cache.write(li, positions, k, v)
        kc, vc = cache.read(li)
        o = self.q(causal_gqa_attention(q, kc, vc, positions).reshape(n, S.n_heads * S.head_dim))
        x = x + o @ W["wo"].T
        h2 = self.q(rms_norm(x, W["ffn_norm"], S.rms_eps))
        a = self.q(swiglu(h2 @ W["wgate"].T, h2 @ W["wup"].T))
        return x + a @ W["wdown"].T

    # -- forward over new tokens of one sequence --------------------------------
    def forward(self, cache, tokens, logits_for=None) -> np.ndarray:
        """Append ``tokens`` to the sequence held by ``cache``; return float32
        logits ``[len(tokens), V]`` for every new position, or only for the
        new positions indexed by ``logits_for``."""
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.arange(cache.length, cache.length + len(tokens))
        x = self.embed_rows(tokens)
        for li in range(self.shape.n_layers):
            x = self.block(li, x, cache, positions)
        cache.advance(len(tokens))
        if logits_for is not None:
            x = x[logits_for]
        hf = self.q(rms_norm(x, self.final_norm, self.shape.rms_eps))
        return self.lm_head_logits(hf).astype(np.float32)

    def forward_each(self, caches, token_lists, logits_for_lists, on_layer=None) -> list:
        """``forward(caches[a], token_lists[a], logits_for_lists[a])`` for every
        sequence ``a``, with the layer loop outside the loop over sequences so
        that lazy mode converts each layer's weights once.  Each sequence still
        goes through the same blocks on its own, so every result is bitwise that
        of the separate calls.  ``on_layer(li)`` is called after each layer
        (progress reports of long runs)."""
        toks = [np.asarray(t, dtype=np.int64) for t in token_lists]
        pos = [np.arange(c.length, c.length + len(t)) for c, t in zip(caches, toks)]
        xs = [self.embed_rows(t) for t in toks]
        for li in range(self.shape.n_layers):
            for a, c in enumerate(caches):
                xs[a] = self.block(li, xs[a], c, pos[a])
            if on_layer is not None:
                on_layer(li)
        out = []
        for a, c in enumerate(caches):
            c.advance(len(toks[a]))
            x = xs[a] if logits_for_lists[a] is None else xs[a][logits_for_lists[a]]
            hf = self.q(rms_norm(x, self.final_norm, self.shape.rms_eps))
            out.append(self.lm_head_logits(hf).astype(np.float32))
        return out

    def hidden_layers(self, cache, tokens, n_layers: int) -> np.ndarray:
        """Residual stream after the first ``n_layers`` blocks (for sampling the
        cost of the full model on the CPU; no logits)."""
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.arange(cache.length, cache.length + len(tokens))
        x = self.embed_rows(tokens)
        for li in range(n_layers):
            x = self.block(li, x, cache, positions)
        cache.advance(len(tokens))
        return x

    # -- generation ------------------------------------------------------------
    def prefill(self, cache, prompt, chunk: int | None = None) -> np.ndarray:
        """Prefill ``prompt`` (optionally in chunks); return the last position's logits."""
        prompt = np.asarray(prompt, dtype=np.int64)
        step = len(prompt) if chunk is None else chunk
        last = None
        for s in range(0, len(prompt), step):
            last = self.forward(cache, prompt[s:s + step], logits_for=[-1])[0]
        return last

    def generate(self, prompt, n_new: int, chunk: int | None = None):
        """Greedy fixed-length generation: ``n_new`` tokens from one prefill and
        ``n_new - 1`` decode steps (no end-of-sequence stop).

        Returns ``(tokens [n_new], logits [n_new, V] float32)``; row ``i`` of the
        logits is the distribution that produced token ``i``.
        """
        cache = self.new_cache()
        logits = [self.prefill(cache, prompt, chunk)]
        toks = [int(greedy_argmax(logits[-1]))]
        for _ in range(n_new - 1):
            logits.append(self.forward(cache, [toks[-1]])[0])
            toks.append(int(greedy_argmax(logits[-1])))
        return np.array(toks, dtype=np.int64), np.stack(logits)

    def teacher_forced(self, prompt, feed, chunk: int | None = None) -> np.ndarray:
        """Logits for the prompt's last position and then after each token of
        ``feed`` (decode steps), whatever tokens the model itself would choose."""
        cache = self.new_cache()
        rows = [self.prefill(cache, prompt, chunk)]
        for t in feed:
            rows.append(self.forward(cache, [int(t)])[0])
        return np.stack(rows)
