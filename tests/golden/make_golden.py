"""Write oracle_chain_tiny.json from the CPU oracle (see README.md)."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import Oracle                                     # noqa: E402
from synth import make_inputs, make_weights, host_inputs, host_weights   # noqa: E402
from test_shapes import GOLDEN_SHAPES                         # noqa: E402


def run(cfg, mode):
    hw, hi = host_weights(make_weights(cfg)), host_inputs(make_inputs(cfg), cfg)
    orc = Oracle(cfg, hw)
    if mode == "greedy":
        out = orc.chain(hi)
    elif mode == "catchup":
        out = orc.chain(hi, catchup=True)
    else:
        out = orc.chain(hi, temperature=cfg.temperature, uniforms=hi["uniforms"])
    rec = {"tokens": out["tokens"].tolist(),
           "logits_head": out["logits"][:, :, :8].round(12).tolist(),
           "hidden_head": out["hidden"][:, :, :8].round(12).tolist()}
    if mode == "sampled":
        rec["logp"] = out["logp"].round(12).tolist()
    return rec


def main():
    res = {name: run(cfg, mode) for name, (cfg, mode) in GOLDEN_SHAPES.items()}
    with open(os.path.join(HERE, "oracle_chain_tiny.json"), "w") as fh:
        json.dump(res, fh, indent=1)


if __name__ == "__main__":
    main()
