"""Stored fixtures: the paper's hyper-parameter table (cited in the file)
and the oracle's tiny-step record (written by tests/golden/make_tiny_step.py)."""
import json
import math
import os

import numpy as np

from paper_2606_24780_amd import synth

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_124m_config_matches_paper_table():
    g = json.load(open(os.path.join(HERE, "hparams_124m.json")))
    c, hp = synth.GPT2_124M, synth.HP_124M
    assert (c.C, c.L, c.H, c.hd, c.F, c.max_T, c.V, c.Vp) == (
        g["d_model"], g["layers"], g["heads"], g["head_dim"], g["ffn_hidden"],
        g["context_length"], g["vocab"], g["vocab_padded"])
    assert (hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, hp.grad_clip) == (
        g["max_lr"], g["beta1"], g["beta2"], g["eps"], g["weight_decay"], g["grad_clip"])
    n = synth.num_params(c)
    # 124M with the padded vocabulary rows and 1024 positions
    assert round(n / 1e6) == g["param_count_millions"]
    assert n == 124475904 and synth.num_decay_params(c) == 124354560
    B, T, C = g["per_gpu_batch"]
    assert 8 * g["grad_accumulation"] * B * T == g["global_batch_tokens"]
    # residual-projection init std for 12 layers
    assert abs(0.02 / math.sqrt(2 * c.L) - 0.0040824829) < 1e-9


def test_tiny_step_regression():
    from tests.golden.make_tiny_step import tiny_inputs
    from oracle import gpt2 as og
    rec = json.load(open(os.path.join(HERE, "tiny_step.json")))
    cfg, params, x, y = tiny_inputs()
    specs = synth.param_specs(cfg)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    out = og.train_step(cfg, synth.HP_TINY, specs, params, zeros, zeros, x, y, t=1)
    assert abs(out["loss"] - rec["loss"]) < 1e-12
    assert abs(out["norm"] - rec["grad_norm"]) < 1e-12
    for n, _, _ in specs:
        assert abs(np.abs(out["grads"][n]).max() - rec["grad_maxabs"][n]) <= 1e-12 * max(1, rec["grad_maxabs"][n])
        assert abs(out["params"][n].sum() - rec["param_sum"][n]) <= 1e-9 * max(1, abs(rec["param_sum"][n]))
