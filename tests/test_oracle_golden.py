"""The oracle still reproduces its committed regression record (tiny shape)."""
import json
import os

import numpy as np

from tests.golden.make_golden import compute


def test_oracle_matches_committed_golden(repo_root):
    with open(os.path.join(repo_root, "tests", "golden", "tiny_seed0.json")) as f:
        gold = json.load(f)
    now = compute(gold["weights_seed"])
    for a, b in zip(now["agents"], gold["agents"]):
        assert a["prompt_len"] == b["prompt_len"]
        assert a["tokens"] == b["tokens"]
        np.testing.assert_allclose(a["row_l2"], b["row_l2"], rtol=1e-6)
        np.testing.assert_allclose(a["first8"], b["first8"], rtol=1e-6, atol=1e-7)
