"""Writes tests/golden/tiny_seed0.json from the oracle alone.

The paper prints no numerical output of the transformer it serves, so this
fixture is a regression record of the oracle on the tiny Llama-style shape
(2 layers, d_model 256, 4/2 heads of 64, FFN 688, vocab 4096; 4 agent prompts
of 32..128 tokens, 16 greedy tokens each).  It calls only ``oracle`` and the
seeded input generator.  Run: ``python tests/golden/make_golden.py``.
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import LlamaShape, OracleModel  # noqa: E402
from paper_2411_03519_amd import synth  # noqa: E402


def compute(seed=0):
    model = OracleModel(LlamaShape(**synth.TINY), synth.llama_weights(synth.TINY, seed))
    prompts, n_new = synth.tiny_agent_batch(seed)
    out = []
    for p in prompts:
        toks, logits = model.generate(p, n_new)
        srt = np.sort(logits, axis=1)
        out.append({"prompt_len": int(len(p)), "tokens": [int(t) for t in toks],
                    "row_l2": [float(x) for x in np.linalg.norm(logits.astype(np.float64), axis=1)],
                    "top2_margin": [float(x) for x in (srt[:, -1] - srt[:, -2])],
                    "first8": [[float(x) for x in r[:8]] for r in logits]})
    return {"shape": synth.TINY, "weights_seed": seed, "prompt_seed": seed, "n_new": n_new, "agents": out}


if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_seed0.json")
    with open(path, "w") as f:
        json.dump(compute(0), f, indent=1)
    print("wrote", path)
