"""Pins for the whole-model float64 oracle (CPU only).

* fourth-order central finite differences of the loss on the tiny model:
  >= 32 sampled entries of every tensor plus every entry of one LN gain;
* an independent torch-CPU float64 autograd model of the same definitions
  (tiny model, padded vocabulary, and the GPT-2 124M shapes on a short
  sequence);
* loss = ln(V) exactly when the token embedding is zero (tiny and 124M shapes);
* 4 micro-steps of B/4 equal one step of B in exact arithmetic;
* one-block forward/backward against torch autograd.
"""
import math

import numpy as np
import pytest

from oracle import gpt2 as og
from oracle import ops
from paper_2606_24780_amd import synth

CFG = synth.TINY


def _tiny_inputs(seed=1, zero_wte=False):
    params = synth.init_params(CFG, seed, zero_wte=zero_wte)
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    x = synth.uniform_tokens((2, 32), CFG.V, rng)
    y = synth.uniform_tokens((2, 32), CFG.V, rng)
    return params, x, y


def _loss(params64, x, y):
    return og.forward(CFG, params64, x, y)[0]


def test_finite_differences_tiny_model():
    params, x, y = _tiny_inputs()
    p64 = {k: v.astype(np.float64) for k, v in params.items()}
    # give LN gains/biases and linear biases non-trivial values so their
    # gradients exercise every term
    rng = np.random.Generator(np.random.PCG64(99))
    for k in p64:
        if k.endswith(("b", "bqkv", "bo", "bfc", "bfp")) or k.endswith("g"):
            p64[k] = p64[k] + 0.05 * rng.standard_normal(p64[k].shape)
    loss, _, grads = og.fwd_bwd(CFG, p64, x, y)
    assert math.isfinite(loss)
    for name, shape, _ in synth.param_specs(CFG):
        g = grads[name]
        scale = np.abs(g).max()
        if name == "wte":
            idx_all = [np.unravel_index(i, shape) for i in rng.choice(g.size, 32, replace=False)]
            idx_all += [(int(x[0, 3]), 5), (int(y[1, 7]), 9)]
        elif name == "h1.ln2g":
            idx_all = [(j,) for j in range(shape[0])]
        else:
            idx_all = [np.unravel_index(i, shape) for i in rng.choice(g.size, 32, replace=False)]
        for idx in idx_all:
            th = p64[name]
            old = th[idx]
            # fourth-order central stencil: truncation O(h^4), round-off
            # ~ eps * loss / h, both far below the tolerance at h = 1e-3
            h = 1e-3 * max(1.0, abs(old))
            f = {}
            for s in (-2, -1, 1, 2):
                th[idx] = old + s * h
                f[s] = _loss(p64, x, y)
            th[idx] = old
            fd = (8 * (f[1] - f[-1]) - (f[2] - f[-2])) / (12 * h)
            assert abs(fd - g[idx]) <= 1e-6 * scale + 1e-12, (name, idx, fd, g[idx])


def _torch_model(torch, cfg, params, x, y):
    F = torch.nn.functional
    P = {k: torch.tensor(v.astype(np.float64), requires_grad=True) for k, v in params.items()}
    B, T = x.shape
    tok = torch.tensor(x.astype(np.int64))
    h = P["wte"][tok] + P["wpe"][:T][None]
    for l in range(cfg.L):
        q = lambda n: P[f"h{l}.{n}"]
        u = F.layer_norm(h, (cfg.C,), q("ln1g"), q("ln1b"), eps=cfg.ln_eps)
        qkv = u @ q("Wqkv") + q("bqkv")
        qkv = qkv.view(B, T, 3, cfg.H, cfg.hd)
        qq, kk, vv = (qkv[:, :, i].transpose(1, 2) for i in range(3))
        a = F.scaled_dot_product_attention(qq, kk, vv, is_causal=True)
        a = a.transpose(1, 2).reshape(B, T, cfg.C)
        h = h + a @ q("Wo") + q("bo")
        u = F.layer_norm(h, (cfg.C,), q("ln2g"), q("ln2b"), eps=cfg.ln_eps)
        h = h + F.gelu(u @ q("Wfc") + q("bfc"), approximate="tanh") @ q("Wfp") + q("bfp")
    u = F.layer_norm(h, (cfg.C,), P["lnfg"], P["lnfb"], eps=cfg.ln_eps)
    logits = u @ P["wte"].T
    loss = F.cross_entropy(logits[..., : cfg.V].reshape(-1, cfg.V),
                           torch.tensor(y.astype(np.int64)).reshape(-1))
    loss.backward()
    return loss.item(), {k: v.grad.numpy() for k, v in P.items()}


def test_tiny_model_vs_torch_autograd(torch_cpu):
    params, x, y = _tiny_inputs(seed=7)
    rng = np.random.Generator(np.random.PCG64(5))
    for k in params:
        if not k.startswith(("wte", "wpe")) and params[k].ndim == 1:
            params[k] = params[k] + 0.05 * rng.standard_normal(params[k].shape).astype(np.float32)
    loss, _, grads = og.fwd_bwd(CFG, params, x, y)
    tl, tg = _torch_model(torch_cpu, CFG, params, x, y)
    assert abs(loss - tl) < 1e-12
    for name in grads:
        assert np.allclose(grads[name], tg[name], rtol=1e-9, atol=1e-13 * max(1, np.abs(tg[name]).max())), name


def test_padded_vocab_model_vs_torch(torch_cpu):
    cfg = synth.GPT2Config(V=50, Vp=56, max_T=8, L=1, H=2, C=16)
    params = synth.init_params(cfg, 3)
    rng = np.random.Generator(np.random.PCG64(4))
    x = synth.uniform_tokens((3, 8), cfg.V, rng)
    y = synth.uniform_tokens((3, 8), cfg.V, rng)
    loss, _, grads = og.fwd_bwd(cfg, params, x, y)
    tl, tg = _torch_model(torch_cpu, cfg, params, x, y)
    assert abs(loss - tl) < 1e-12
    for name in grads:
        assert np.allclose(grads[name], tg[name], rtol=1e-9, atol=1e-14), name
    # padded rows of the tied embedding receive exactly zero gradient
    assert np.all(grads["wte"][cfg.V:] == 0)


@pytest.mark.slow
def test_124m_model_vs_torch_autograd(torch_cpu):
    """The oracle's forward and backward at the GPT-2 124M shapes (12 layers,
    768 wide, 12 heads, vocabulary 50,257 padded to 50,304) on one 16-token
    sequence, every 1-D parameter perturbed so that no term vanishes."""
    cfg = synth.GPT2_124M
    params = synth.init_params(cfg, 9)
    rng = np.random.Generator(np.random.PCG64(10))
    for k in params:
        if params[k].ndim == 1:
            params[k] = params[k] + 0.05 * rng.standard_normal(params[k].shape).astype(np.float32)
    stream = synth.zipf_tokens(16 + 1, cfg.V, 1.1, 41)
    x, y = synth.shifted_pair(stream, 1, 16)
    loss, _, grads = og.fwd_bwd(cfg, params, x, y)
    tl, tg = _torch_model(torch_cpu, cfg, params, x, y)
    assert abs(loss - tl) < 1e-12 * abs(tl)
    for name in grads:
        assert np.allclose(grads[name], tg[name], rtol=1e-9, atol=1e-13 * max(1, np.abs(tg[name]).max())), name
    assert np.all(grads["wte"][cfg.V:] == 0)


def test_zero_wte_loss_is_ln_V_tiny():
    params, x, y = _tiny_inputs(zero_wte=True)
    loss, rows, _ = og.forward(CFG, params, x, y)
    assert np.allclose(rows, math.log(CFG.V), rtol=0, atol=1e-13)


@pytest.mark.slow
def test_zero_wte_loss_is_ln_V_124m():
    cfg = synth.GPT2_124M
    params = synth.init_params(cfg, 4, zero_wte=True)
    stream = synth.zipf_tokens(2 * 8 + 1, cfg.V, 1.1, 40)
    x, y = synth.shifted_pair(stream, 2, 8)
    loss, rows, _ = og.forward(cfg, params, x, y)
    assert np.allclose(rows, math.log(50257), rtol=0, atol=1e-12)
    assert abs(loss - 10.824905) < 1e-6  # ln 50257; ln 50304 would be 10.825840


def test_accumulation_equals_large_batch():
    cfg = synth.GPT2Config(V=64, Vp=64, max_T=16, L=1, H=2, C=16)
    params = synth.init_params(cfg, 11)
    specs = synth.param_specs(cfg)
    stream = synth.zipf_tokens(8 * 16 + 1, cfg.V, 1.1, 12)
    x, y = synth.shifted_pair(stream, 8, 16)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    hp = synth.HP_124M
    big = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1, accum=1)
    acc = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1, accum=4)
    assert abs(big["loss"] - acc["loss"]) < 1e-12
    for n in big["grads"]:
        assert np.allclose(big["grads"][n], acc["grads"][n], rtol=0, atol=1e-12)
        assert np.allclose(big["params"][n], acc["params"][n], rtol=0, atol=1e-12)


def test_block_vs_torch(torch_cpu):
    torch = torch_cpu
    F = torch.nn.functional
    C, H, B, T = 32, 4, 2, 12
    p = synth.block_params(C, H, 3)
    rng = np.random.Generator(np.random.PCG64(3))
    x = rng.standard_normal((B, T, C))
    dy = rng.standard_normal((B, T, C)) * 1e-3
    y, cache = og.block_fwd(x, p, H)
    dx, gr = og.block_bwd(dy, p, cache)
    P = {k: torch.tensor(v.astype(np.float64), requires_grad=True) for k, v in p.items()}
    xt = torch.tensor(x, requires_grad=True)
    u = F.layer_norm(xt, (C,), P["ln1g"], P["ln1b"], eps=1e-5)
    qkv = (u @ P["Wqkv"] + P["bqkv"]).view(B, T, 3, H, C // H)
    q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))
    a = F.scaled_dot_product_attention(q, k, v, is_causal=True).transpose(1, 2).reshape(B, T, C)
    h = xt + a @ P["Wo"] + P["bo"]
    u = F.layer_norm(h, (C,), P["ln2g"], P["ln2b"], eps=1e-5)
    yt = h + F.gelu(u @ P["Wfc"] + P["bfc"], approximate="tanh") @ P["Wfp"] + P["bfp"]
    yt.backward(torch.tensor(dy))
    assert np.allclose(y, yt.detach().numpy(), atol=1e-12)
    assert np.allclose(dx, xt.grad.numpy(), atol=1e-15)
    for k in gr:
        assert np.allclose(gr[k], P[k].grad.numpy(), rtol=1e-9, atol=1e-15), k


def test_train_step_adamw_t1_closed_form():
    params, x, y = _tiny_inputs()
    specs = synth.param_specs(CFG)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    hp = synth.HP_TINY
    out = og.train_step(CFG, hp, specs, params, zeros, zeros, x, y, t=1)
    for name, _, dec in specs:
        g = out["grads"][name]
        p0 = params[name].astype(np.float64)
        exp = p0 - hp.lr * (hp.weight_decay * p0 * (1.0 if dec else 0.0) + g / (np.abs(g) + hp.eps))
        assert np.allclose(out["params"][name], exp, rtol=0, atol=1e-15), name
