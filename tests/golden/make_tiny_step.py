"""Writes tiny_step.json: the float64 oracle's result for one training step
of the tiny GPT-2 (2 layers, d_model 64, 4 heads, vocab 256, T 32, B 2;
AdamW lr 3e-4, betas 0.9/0.999, eps 1e-8, wd 0.1, t = 1, no clip) on the
seeded synthetic inputs.  Calls only the oracle and the seeded generators.

    python tests/golden/make_tiny_step.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import gpt2 as og  # noqa: E402
from paper_2606_24780_amd import synth  # noqa: E402


def tiny_inputs():
    cfg = synth.TINY
    params = synth.init_params(cfg, 1)
    rng = np.random.Generator(np.random.PCG64(1001))
    x = synth.uniform_tokens((2, 32), cfg.V, rng)
    y = synth.uniform_tokens((2, 32), cfg.V, rng)
    return cfg, params, x, y


def main():
    cfg, params, x, y = tiny_inputs()
    specs = synth.param_specs(cfg)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    out = og.train_step(cfg, synth.HP_TINY, specs, params, zeros, zeros, x, y, t=1)
    rec = {
        "_source": "float64 oracle, tests/golden/make_tiny_step.py",
        "loss": out["loss"],
        "grad_norm": out["norm"],
        "grad_maxabs": {n: float(np.abs(out["grads"][n]).max()) for n, _, _ in specs},
        "grad_sum": {n: float(out["grads"][n].sum()) for n, _, _ in specs},
        "param_sum": {n: float(out["params"][n].sum()) for n, _, _ in specs},
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_step.json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
    print("wrote", path, "loss", rec["loss"])


if __name__ == "__main__":
    main()
