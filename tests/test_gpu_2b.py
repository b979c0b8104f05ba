"""The 2.42B-parameter configuration (section "Largest trainable parameter
model": d_model 3072, 20 layers, 24 heads of dim 128, B = 2, T = 1024).

* a narrow model with the same head dim (C = 256, H = 2, L = 2, V = 256,
  T = 64) through the whole step against the float64 oracle (loss, every
  gradient, the AdamW update);
* the 2.42B model at B = 2, T = 1024 with both sequences copies of one: the
  batch-mean gradient equals the one-sequence gradient, so the oracle's
  forward and backward of that sequence give the loss, the per-position
  losses and every gradient of the full-size step; the AdamW update is checked
  by the oracle's AdamW applied to the GPU's own gradients (the float64
  optimizer state of 2.42B parameters would not fit next to the rest)."""
import numpy as np
import pytest

from oracle import gpt2 as og
from paper_2606_24780_amd import bt, synth
from tests.gpu_util import assert_close_maxabs, dev, host, say, torch_gpu
from tests.test_gpu_gpt2 import GRAD_TOL, LOSS_TOL, _check_end_to_end, _check_update, _gpu_step, _unflat

pytestmark = pytest.mark.gpu


def test_narrow_model_head_dim_128_step_vs_oracle():
    torch = torch_gpu()
    cfg, hp = synth.TINY_HD128, synth.HP_TINY
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 11)
    B, T = 2, cfg.max_T
    rng = np.random.Generator(np.random.PCG64(128))
    x, y = synth.shifted_pair(synth.uniform_tokens(B * T + 1, cfg.V, rng), B, T)
    say("narrow model, head dim 128: train step")
    model, loss = _gpu_step(torch, cfg, hp, params, x, y)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1)
    say(f"loss gpu={loss:.8f} oracle={ref['loss']:.8f}")
    assert abs(loss - ref["loss"]) <= LOSS_TOL * abs(ref["loss"])
    g = _unflat(cfg, model.grads)
    for name, _, _ in specs:
        assert_close_maxabs(g[name], ref["grads"][name], GRAD_TOL, f"grad {name}")
    p, m, v = _unflat(cfg, model.params), _unflat(cfg, model.m), _unflat(cfg, model.v)
    _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="hd128")
    _check_end_to_end(hp, specs, params, g, ref["grads"], p, ref["params"])


@pytest.mark.timeout(1200)
def test_gpt2_2_42b_replicated_sequence_step():
    torch = torch_gpu()
    cfg, hp = synth.GPT2_2_42B, synth.HP_124M
    specs = synth.param_specs(cfg)
    B, T = 2, cfg.max_T
    params = synth.init_params(cfg, 5)
    stream = synth.zipf_tokens(T + 1, cfg.V, 1.1, 42)
    x1, y1 = synth.shifted_pair(stream, 1, T)
    x, y = np.repeat(x1, B, axis=0), np.repeat(y1, B, axis=0)
    say("gpt2 2.42B B=2 T=1024 (two copies of one sequence): train step")
    model = bt.GPT2(cfg, hp, B, T)
    model.load_params(synth.flatten(cfg, params))
    d_loss = torch.zeros(1, device="cuda")
    rows = torch.zeros(B * T, device="cuda")
    model.fwd_bwd(dev(torch, x), dev(torch, y), 1.0 / (B * T), 0, d_loss, rows)
    loss_rows = host(rows).reshape(B, T)
    model.optimizer_step(1, hp.lr)
    torch.cuda.synchronize()
    g = _unflat(cfg, model.grads)
    say("oracle forward + backward of the sequence")
    loss_o, rows_o, g_o = og.fwd_bwd(cfg, params, x1, y1)
    assert np.array_equal(loss_rows[0], loss_rows[1])
    assert np.allclose(loss_rows[0], rows_o[0] if rows_o.ndim == 2 else rows_o, rtol=LOSS_TOL, atol=0)
    assert abs(float(d_loss.item()) - loss_o) <= LOSS_TOL * abs(loss_o)
    for name, _, _ in specs:
        assert_close_maxabs(g[name], g_o[name], GRAD_TOL, f"grad {name}")
    del g_o
    p, m, v = _unflat(cfg, model.params), _unflat(cfg, model.m), _unflat(cfg, model.v)
    _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="2.42B")
