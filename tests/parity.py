"""Comparison rules between the HIP path and the oracle.

Logits: max-abs <= 2e-2 over all compared values and, per row,
||gpu - oracle||_2 / ||oracle||_2 <= 1e-2.

At Llama-3 widths these figures are below what fp32 arithmetic can reach:
every bf16 re-quantisation point (h, q/k/v, o, the SwiGLU product) turns a
perturbation of relative size delta into about sqrt(delta * ulp), so the
oracle evaluated in float32 already differs from its float64 evaluation by
max-abs ~3.4e-2 (rel-L2 ~5.6e-3) at 8B widths and depth 2, and by max-abs
~1.2e-1, rel-L2 ~2.1e-2 at full depth (32 layers).  Each bound is therefore
the larger of the fixed figure and twice that measured float32-vs-float64
spread of the oracle on the same inputs (``noise_floor``).

Greedy tokens: compared step by step under teacher forcing (both sides are fed
the oracle's tokens).  A different choice is a failure when the oracle's top-2
margin at that step is >= the max-abs bound; below it the two candidates are
tied within tolerance and the step is counted as a tie-divergence instead.
"""

from __future__ import annotations

import numpy as np

MAX_ABS = 2e-2
REL_L2 = 1e-2


def logits_errors(got: np.ndarray, want: np.ndarray):
    got = np.asarray(got, np.float64).reshape(-1, want.shape[-1])
    want = np.asarray(want, np.float64).reshape(-1, want.shape[-1])
    max_abs = float(np.max(np.abs(got - want)))
    rel = np.linalg.norm(got - want, axis=1) / np.linalg.norm(want, axis=1)
    return max_abs, float(np.max(rel))


def assert_logits_close(got, want, what="", max_abs_bound=MAX_ABS, rel_bound=REL_L2):
    assert np.all(np.isfinite(got)), f"{what}: non-finite logits"
    max_abs, rel = logits_errors(got, want)
    msg = (f"{what}: max-abs {max_abs:.3e} (bound {max_abs_bound:.3e}), "
           f"max rel-L2 {rel:.3e} (bound {rel_bound:.3e})")
    print(msg, flush=True)
    assert max_abs <= max_abs_bound and rel <= rel_bound, msg
    return max_abs, rel


def noise_floor(f64_logits, f32_logits):
    """(max-abs bound, rel-L2 bound) from the float32-vs-float64 spread of the
    oracle itself: each the larger of the fixed figure and twice the spread."""
    spread, rel = logits_errors(f32_logits, f64_logits)
    print(f"oracle float32 vs float64: max-abs {spread:.3e}, max rel-L2 {rel:.3e}", flush=True)
    return max(MAX_ABS, 2.0 * spread), max(REL_L2, 2.0 * rel)


def top2_margin(logits: np.ndarray) -> np.ndarray:
    s = np.sort(np.asarray(logits, np.float64), axis=-1)
    return s[..., -1] - s[..., -2]


def check_tokens(got_tok: np.ndarray, want_logits: np.ndarray, what="", tie=MAX_ABS) -> int:
    """Greedy choices of the GPU against the oracle's logits of the same step.
    Returns the number of tie-divergences; raises on a real mismatch."""
    want_tok = np.argmax(want_logits, axis=-1)
    margin = top2_margin(want_logits)
    diff = np.asarray(got_tok).reshape(want_tok.shape) != want_tok
    bad = diff & (margin >= tie)
    assert not np.any(bad), f"{what}: token mismatch at margin {margin[bad]}"
    return int(np.sum(diff))
