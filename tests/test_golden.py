"""The oracle against its stored runs (tests/golden/README.md): tokens exactly,
logits / hidden heads and log-probs to 1e-9."""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

from make_golden import run          # noqa: E402
from test_shapes import GOLDEN_SHAPES  # noqa: E402


def test_oracle_matches_stored_runs():
    with open(os.path.join(HERE, "golden", "oracle_chain_tiny.json")) as fh:
        stored = json.load(fh)
    assert sorted(stored) == sorted(GOLDEN_SHAPES)
    for name, (cfg, mode) in GOLDEN_SHAPES.items():
        now = run(cfg, mode)
        assert now["tokens"] == stored[name]["tokens"], name
        for key in ("logits_head", "hidden_head", "logp"):
            if key in stored[name]:
                assert np.max(np.abs(np.array(now[key]) - np.array(stored[name][key]))) < 1e-9, (name, key)
