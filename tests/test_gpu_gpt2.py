"""Composed training step (bt_gpt2_*) against the float64 oracle.

* tiny GPT-2 (2 layers, d 64, 4 heads, vocab 256, T 32, B 2): loss, every
  gradient tensor and the AdamW update;
* zero token embedding: loss = ln V;
* determinism: two identical steps are bitwise equal;
* 4 micro-steps of B/4 with accumulation equal one step of B;
* GPT-2 124M at B=16, T=1024 in the benchmark's launch configuration:
  per-position losses of sampled sequences against the oracle run on those
  sequences alone, and a batch of 16 copies of one sequence, whose full
  gradient and update the oracle computes from that one sequence.

Bars (stated for this path): loss relative error <= 1e-5; each gradient
tensor <= 1e-4 of its max-abs; post-AdamW parameters <= 1e-5 of their
max-abs, with the oracle's AdamW fed the GPU's own gradients (at t = 1 the
update g/(|g|+eps) amplifies gradient rounding where |g| ~ eps, so the
end-to-end comparison is reported and checked against that sensitivity
instead)."""
import math

import numpy as np
import pytest

from oracle import gpt2 as og
from oracle import ops
from paper_2606_24780_amd import bt, synth
from tests.golden.make_tiny_step import tiny_inputs
from tests.gpu_util import assert_close_maxabs, dev, host, progress, say, torch_gpu

pytestmark = pytest.mark.gpu

LOSS_TOL, GRAD_TOL, PARAM_TOL = 1e-5, 1e-4, 1e-5


def _gpu_step(torch, cfg, hp, params, x, y, max_B=None):
    B, T = x.shape
    model = bt.GPT2(cfg, hp, max_B or B, T)
    model.load_params(synth.flatten(cfg, params))
    loss = model.train_step(dev(torch, x), dev(torch, y))
    torch.cuda.synchronize()
    return model, loss


def _unflat(cfg, t):
    return synth.unflatten(cfg, host(t))


def _check_update(cfg, hp, specs, params0, g_gpu, p_gpu, m_gpu, v_gpu, t, coef_gpu_norm=None, what=""):
    """Reading of the post-AdamW bar: the oracle's AdamW applied to the GPU's
    own gradients (and the clip coefficient of their norm) must match."""
    flat_g = np.concatenate([g_gpu[n].ravel() for n, _, _ in specs])
    norm = ops.grad_norm(flat_g)
    coef = ops.clip_coef(norm, hp.grad_clip)
    for name, _, dec in specs:
        rp, rm, rv = ops.adamw(params0[name], g_gpu[name], np.zeros_like(g_gpu[name]), np.zeros_like(g_gpu[name]),
                               t, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, 1.0 if dec else 0.0, coef)
        assert_close_maxabs(p_gpu[name], rp, PARAM_TOL, f"{what} param {name}")
        assert_close_maxabs(m_gpu[name], rm, 1e-5, f"{what} m {name}")
        assert_close_maxabs(v_gpu[name], rv, 1e-5, f"{what} v {name}")
    return norm, coef


def _check_end_to_end(hp, specs, params0, g_gpu, g_or, p_gpu, p_or, c_gpu=1.0, c_or=1.0):
    """End-to-end params: elementwise within 1e-5 max-abs, or within the
    t = 1 sensitivity of the update u(x) = x / (|x| + eps) of the clipped
    gradient x = c g: lr * eps * |x_gpu - x_or| / (min|x| + eps)^2 (mean-value
    bound on an interval of one sign)."""
    worst = 0.0
    for name, _, _ in specs:
        d = np.abs(p_gpu[name] - p_or[name])
        scale = np.abs(p_or[name]).max()
        xg, xo = c_gpu * g_gpu[name], c_or * g_or[name]
        xmin = np.minimum(np.abs(xg), np.abs(xo))
        bound = hp.lr * hp.eps * np.abs(xg - xo) / (xmin + hp.eps) ** 2 + PARAM_TOL * scale
        same_sign = np.sign(xg) == np.sign(xo)
        bound = np.where(same_sign, bound, 2 * hp.lr + PARAM_TOL * scale)
        assert (d <= bound * (1 + 1e-6) + 1e-12).all(), f"end-to-end {name}"
        worst = max(worst, float(d.max() / scale))
    say(f"[parity] end-to-end params worst max-abs-rel {worst:.3e}")


def test_tiny_step_vs_oracle():
    torch = torch_gpu()
    cfg, params, x, y = tiny_inputs()
    hp = synth.HP_TINY
    specs = synth.param_specs(cfg)
    say("gpt2 tiny step")
    model, loss = _gpu_step(torch, cfg, hp, params, x, y)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1)
    say(f"loss gpu={loss:.8f} oracle={ref['loss']:.8f}")
    assert abs(loss - ref["loss"]) <= LOSS_TOL * abs(ref["loss"])
    g = _unflat(cfg, model.grads)
    for name, _, _ in specs:
        assert_close_maxabs(g[name], ref["grads"][name], GRAD_TOL, f"grad {name}")
    p = _unflat(cfg, model.params)
    m = _unflat(cfg, model.m)
    v = _unflat(cfg, model.v)
    _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="tiny")
    _check_end_to_end(hp, specs, params, g, ref["grads"], p, ref["params"])
    assert model.step_count == 1


def test_tiny_zero_wte_loss_is_ln_V():
    torch = torch_gpu()
    cfg, _, x, y = tiny_inputs()
    params = synth.init_params(cfg, 1, zero_wte=True)
    say("gpt2 tiny zero wte")
    _, loss = _gpu_step(torch, cfg, synth.HP_TINY, params, x, y)
    assert abs(loss - math.log(cfg.V)) <= 1e-6 * math.log(cfg.V)


def test_tiny_step_deterministic():
    torch = torch_gpu()
    cfg, params, x, y = tiny_inputs()
    say("gpt2 tiny determinism")
    m1, l1 = _gpu_step(torch, cfg, synth.HP_TINY, params, x, y)
    m2, l2 = _gpu_step(torch, cfg, synth.HP_TINY, params, x, y)
    assert l1 == l2
    assert torch.equal(m1.grads, m2.grads) and torch.equal(m1.params, m2.params)
    assert torch.equal(m1.opt_state, m2.opt_state)


def test_step_profiler_counts_and_intervals():
    """The step profiler (HIP events around every library call, the end of
    one call shared with the start of the next): per-class call counts follow
    the model's structure, GEMM flops are sum 2MNK, and the intervals add up to
    no more than the steps' own event-timed duration (nothing counted twice)."""
    torch = torch_gpu()
    cfg, params, x, y = tiny_inputs()
    B, T = x.shape
    L, C, F, Vp = cfg.L, cfg.C, 4 * cfg.C, cfg.Vp
    say("gpt2 tiny step profiler")
    model = bt.GPT2(cfg, synth.HP_TINY, B, T)
    model.load_params(synth.flatten(cfg, params))
    xd, yd = dev(torch, x), dev(torch, y)
    model.train_step(xd, yd)
    model.profile_enable(True)
    model.profile_read(reset=True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(model.stream)
    steps = 2
    for _ in range(steps):
        model.train_step(xd, yd)
    e1.record(model.stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    prof = model.profile_read(reset=True)
    model.profile_enable(False)
    # LayerNorm backward: 2L+1 row passes and one batched sum of their dgamma / dbeta partials
    expect = {"gemm": 12 * L + 3, "attn_fwd": L, "attn_bwd": L, "ln_fwd": 2 * L + 1, "ln_bwd": 2 * L + 2,
              "xent": 1, "emb_fwd": 1, "emb_bwd": 1, "grad_norm": 1, "adamw": 1}
    for name, n in expect.items():
        assert prof[name]["launches"] == steps * n, (name, prof[name]["launches"])
        assert prof[name]["ms"] > 0, name
    M = B * T
    shapes = [(M, 3 * C, C), (M, C, C), (M, F, C), (M, C, F)]
    flops = L * sum(2 * m * n * k * 3 for m, n, k in shapes) + 3 * 2 * M * Vp * C
    assert prof["gemm"]["flops"] == pytest.approx(steps * flops, rel=1e-12)
    assert sum(v["ms"] for v in prof.values()) <= total_ms * 1.001


def test_tiny_multi_step_losses():
    torch = torch_gpu()
    cfg, params, x, y = tiny_inputs()
    hp = synth.HP_TINY
    specs = synth.param_specs(cfg)
    say("gpt2 tiny 3 steps")
    model = bt.GPT2(cfg, hp, 2, 32)
    model.load_params(synth.flatten(cfg, params))
    xd, yd = dev(torch, x), dev(torch, y)
    p = {k: v.astype(np.float64) for k, v in params.items()}
    m = {k: np.zeros_like(v) for k, v in p.items()}
    v = {k: np.zeros_like(val) for k, val in p.items()}
    for t in range(1, 4):
        loss = model.train_step(xd, yd)
        ref = og.train_step(cfg, hp, specs, p, m, v, x, y, t=t)
        p, m, v = ref["params"], ref["m"], ref["v"]
        say(f"step {t}: gpu {loss:.8f} oracle {ref['loss']:.8f}")
        assert abs(loss - ref["loss"]) <= 1e-4 * abs(ref["loss"])


def test_tiny_accumulation_equals_large_batch():
    torch = torch_gpu()
    cfg = synth.TINY
    hp = synth.HP_124M  # with clipping
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 5)
    stream = synth.zipf_tokens(8 * 32 + 1, cfg.V, 1.1, 50)
    x, y = synth.shifted_pair(stream, 8, 32)
    say("gpt2 tiny accumulation 4 x 2 vs 8")
    big, loss_big = _gpu_step(torch, cfg, hp, params, x, y)
    acc = bt.GPT2(cfg, hp, 2, 32)
    acc.load_params(synth.flatten(cfg, params))
    d_loss = torch.zeros(1, device="cuda")
    for k in range(4):
        acc.fwd_bwd(dev(torch, x[2 * k:2 * k + 2]), dev(torch, y[2 * k:2 * k + 2]), 1.0 / (8 * 32), k > 0, d_loss)
    acc.optimizer_step(1, hp.lr)
    torch.cuda.synchronize()
    assert abs(float(d_loss.item()) - loss_big) <= 1e-6 * abs(loss_big)
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1, accum=4)
    ga, gb = _unflat(cfg, acc.grads), _unflat(cfg, big.grads)
    for name, _, _ in specs:
        assert_close_maxabs(ga[name], gb[name], GRAD_TOL, f"accum vs big {name}")
        assert_close_maxabs(ga[name], ref["grads"][name], GRAD_TOL, f"accum vs oracle {name}")
    _check_update(cfg, hp, specs, params, ga, _unflat(cfg, acc.params), _unflat(cfg, acc.m), _unflat(cfg, acc.v), 1,
                  what="accum")


def test_deep_narrow_accumulation_vs_oracle():
    """17 layers: the step's 35 LayerNorm dgamma / dbeta sums take two batched
    launches (at most 32 per launch), and with two accumulating micro-steps
    the second adds into the first's parameter gradients."""
    torch = torch_gpu()
    cfg = synth.GPT2Config(V=256, Vp=256, max_T=32, L=17, H=4, C=64)
    hp = synth.HP_124M
    specs = synth.param_specs(cfg)
    # LayerNorm gains and biases away from 1 / 0, so that their gradients are not special
    params = synth.init_params(cfg, 7)
    rng = np.random.Generator(np.random.PCG64(70))
    for name in params:
        if name.endswith(("ln1g", "ln2g", "lnfg")):
            params[name] = (1.0 + 0.2 * rng.standard_normal(params[name].shape)).astype(np.float32)
        elif name.endswith(("ln1b", "ln2b", "lnfb")):
            params[name] = (0.2 * rng.standard_normal(params[name].shape)).astype(np.float32)
    stream = synth.zipf_tokens(4 * 32 + 1, cfg.V, 1.1, 71)
    x, y = synth.shifted_pair(stream, 4, 32)
    say("gpt2 deep narrow (L=17) accumulation 2 x 2 vs oracle")
    acc = bt.GPT2(cfg, hp, 2, 32)
    acc.load_params(synth.flatten(cfg, params))
    d_loss = torch.zeros(1, device="cuda")
    for k in range(2):
        acc.fwd_bwd(dev(torch, x[2 * k:2 * k + 2]), dev(torch, y[2 * k:2 * k + 2]), 1.0 / (4 * 32), k > 0, d_loss)
    acc.optimizer_step(1, hp.lr)
    torch.cuda.synchronize()
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1, accum=2)
    assert abs(float(d_loss.item()) - ref["loss"]) <= LOSS_TOL * abs(ref["loss"])
    ga = _unflat(cfg, acc.grads)
    for name, _, _ in specs:
        assert_close_maxabs(ga[name], ref["grads"][name], GRAD_TOL, f"deep accum vs oracle {name}")
    _check_update(cfg, hp, specs, params, ga, _unflat(cfg, acc.params), _unflat(cfg, acc.m), _unflat(cfg, acc.v), 1,
                  what="deep accum")


@pytest.mark.parametrize("B,T", [(3, 100), (4, 37)])
def test_ragged_step_vs_oracle(B, T):
    """The composed step at a sequence length below the model's maximum and a
    multiple of no tile.  The model is narrow: C = 96, three heads of 32, and
    a vocabulary of 300 padded to 304.  M = B*T = 300 uses the stored-dS
    attention backward.  With T = 37 (not a multiple of 4) the backward
    recomputes instead.  Loss, every gradient and the clipped AdamW update
    are checked against the oracle.  The gradient buffer starts filled with a
    sentinel, and the step must overwrite all of it: the rows of wpe beyond T
    and the padded rows of wte come out exactly zero."""
    torch = torch_gpu()
    cfg = synth.GPT2Config(V=300, Vp=304, max_T=128, L=2, H=3, C=96)
    hp = synth.HP_124M
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 12)
    rng = np.random.Generator(np.random.PCG64(120))
    for name in params:
        if name.endswith(("ln1g", "ln2g", "lnfg")):
            params[name] = (1.0 + 0.2 * rng.standard_normal(params[name].shape)).astype(np.float32)
        elif params[name].ndim == 1:
            params[name] = (0.2 * rng.standard_normal(params[name].shape)).astype(np.float32)
    stream = synth.zipf_tokens(B * T + 1, cfg.V, 1.1, 13)
    x, y = synth.shifted_pair(stream, B, T)
    say(f"gpt2 ragged step B={B} T={T} (max_T={cfg.max_T}, Vp={cfg.Vp})")
    model = bt.GPT2(cfg, hp, B, T)
    model.load_params(synth.flatten(cfg, params))
    model.grads.fill_(7.25)  # a step that does not accumulate writes every gradient element
    loss = model.train_step(dev(torch, x), dev(torch, y))
    torch.cuda.synchronize()
    zeros = {k: np.zeros_like(v, dtype=np.float64) for k, v in params.items()}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1)
    say(f"loss gpu={loss:.8f} oracle={ref['loss']:.8f}")
    assert abs(loss - ref["loss"]) <= LOSS_TOL * abs(ref["loss"])
    g = _unflat(cfg, model.grads)
    for name, _, _ in specs:
        assert_close_maxabs(g[name], ref["grads"][name], GRAD_TOL, f"grad {name}")
    assert np.all(g["wte"][cfg.V:] == 0) and np.all(g["wpe"][T:] == 0)
    p, m, v = _unflat(cfg, model.params), _unflat(cfg, model.m), _unflat(cfg, model.v)
    norm, coef = _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="ragged")
    _check_end_to_end(hp, specs, params, g, ref["grads"], p, ref["params"], c_gpu=coef, c_or=ref["coef"])


# ---------------------------------------------------------------- GPT-2 124M
def _inputs_124m(B=16, T=1024):
    cfg = synth.GPT2_124M
    params = synth.init_params(cfg, 4)
    stream = synth.zipf_tokens(B * T + 1, cfg.V, 1.1, 40)
    x, y = synth.shifted_pair(stream, B, T)
    return cfg, params, x, y


@pytest.mark.timeout(600)
def test_gpt2_124m_loss_rows_sampled():
    torch = torch_gpu()
    cfg, params, x, y = _inputs_124m()
    hp = synth.HP_124M
    B, T = x.shape
    say("gpt2 124M B=16 T=1024 fwd_bwd loss rows")
    model = bt.GPT2(cfg, hp, B, T)
    model.load_params(synth.flatten(cfg, params))
    d_loss = torch.zeros(1, device="cuda")
    rows = torch.zeros(B * T, device="cuda")
    model.fwd_bwd(dev(torch, x), dev(torch, y), 1.0 / (B * T), 0, d_loss, rows)
    lr_gpu = host(rows).reshape(B, T)
    assert np.isfinite(lr_gpu).all()
    assert abs(float(d_loss.item()) - lr_gpu.mean()) <= 1e-5 * lr_gpu.mean()
    for b in (0, 11):
        say(f"oracle forward of sequence {b}")
        _, rr, _ = og.forward(cfg, params, x[b:b + 1], y[b:b + 1])
        err = np.abs(lr_gpu[b] - rr).max() / np.abs(rr).max()
        say(f"[parity] loss rows seq {b}: max rel {err:.3e}")
        assert np.allclose(lr_gpu[b], rr, rtol=LOSS_TOL, atol=0)


@pytest.mark.timeout(900)
def test_gpt2_124m_replicated_sequence_full_step():
    """16 copies of one sequence: the batch-mean gradient equals the
    one-sequence gradient, so the oracle run on that sequence alone gives
    every gradient and the clipped AdamW update of the full-size step."""
    torch = torch_gpu()
    cfg, params, x, y = _inputs_124m()
    hp = synth.HP_124M
    specs = synth.param_specs(cfg)
    B, T = x.shape
    xr = np.repeat(x[3:4], B, axis=0)
    yr = np.repeat(y[3:4], B, axis=0)
    say("gpt2 124M replicated-sequence train step")
    model, loss = _gpu_step(torch, cfg, hp, params, xr, yr)
    g = _unflat(cfg, model.grads)
    p = _unflat(cfg, model.params)
    m = _unflat(cfg, model.m)
    v = _unflat(cfg, model.v)
    _, norm_gpu, coef_gpu = model.read_scalars()
    del model
    say("oracle step on the single sequence")
    zeros = {k: np.zeros(s, dtype=np.float64) for k, s, _ in specs}
    ref = og.train_step(cfg, hp, specs, params, zeros, zeros, x[3:4], y[3:4], t=1)
    say(f"loss gpu={loss:.8f} oracle={ref['loss']:.8f}; norm gpu={norm_gpu:.6f} oracle={ref['norm']:.6f}")
    assert abs(loss - ref["loss"]) <= LOSS_TOL * abs(ref["loss"])
    assert abs(norm_gpu - ref["norm"]) <= 1e-4 * ref["norm"]
    for name, _, _ in specs:
        assert_close_maxabs(g[name], ref["grads"][name], GRAD_TOL, f"grad {name}")
    norm, coef = _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="124M")
    assert abs(coef - coef_gpu) <= 1e-6 * coef
    _check_end_to_end(hp, specs, params, g, ref["grads"], p, ref["params"], coef_gpu, ref["coef"])


@pytest.mark.timeout(900)
def test_gpt2_124m_distinct_sequences_full_step():
    """The benchmark's own batch: 16 different Zipf sequences of 1024 tokens
    through the full-size step, against the oracle run one sequence at a time
    and summed (micro-steps of the data-parallel training-step algorithm,
    each scaled by 1/(B*T)): the loss, every gradient tensor, the gradient
    norm and clip coefficient, and the clipped AdamW update."""
    torch = torch_gpu()
    cfg, params, x, y = _inputs_124m()
    hp = synth.HP_124M
    specs = synth.param_specs(cfg)
    B, T = x.shape
    assert len({tuple(r) for r in x}) == B, "the batch must hold distinct sequences"
    progress("gpt2 124M distinct-sequence train step (B=16, T=1024) on the GPU")
    model, loss = _gpu_step(torch, cfg, hp, params, x, y)
    g = _unflat(cfg, model.grads)
    p = _unflat(cfg, model.params)
    m = _unflat(cfg, model.m)
    v = _unflat(cfg, model.v)
    _, norm_gpu, coef_gpu = model.read_scalars()
    del model
    torch.cuda.empty_cache()
    scale = 1.0 / (B * T)
    grads, loss_or = None, 0.0
    for b in range(B):
        lb, _, cache = og.forward(cfg, params, x[b:b + 1], y[b:b + 1])
        gb = og.backward(cfg, params, cache, scale)
        del cache
        loss_or += lb / B
        if grads is None:
            grads = gb
        else:
            for n in grads:
                grads[n] += gb[n]
        progress(f"oracle sequence {b + 1}/{B} done")
    zeros = {k: np.zeros(s_, dtype=np.float64) for k, s_, _ in specs}
    p_or, _, _, norm_or, coef_or = og.optimizer_step(params, grads, zeros, zeros, 1, hp, specs)
    say(f"loss gpu={loss:.8f} oracle={loss_or:.8f}; norm gpu={norm_gpu:.6f} oracle={norm_or:.6f}")
    assert abs(loss - loss_or) <= LOSS_TOL * abs(loss_or)
    assert abs(norm_gpu - norm_or) <= 1e-4 * norm_or
    assert abs(coef_gpu - coef_or) <= 1e-4 * coef_or
    for name, _, _ in specs:
        assert_close_maxabs(g[name], grads[name], GRAD_TOL, f"grad {name}")
    _, coef = _check_update(cfg, hp, specs, params, g, p, m, v, 1, what="124M distinct")
    assert abs(coef - coef_gpu) <= 1e-6 * coef
    _check_end_to_end(hp, specs, params, g, grads, p, p_or, coef_gpu, coef_or)
    progress("gpt2 124M distinct-sequence step checked")


@pytest.mark.timeout(900)
def test_gpt2_124m_b64_equals_4x16_accumulation():
    """Large-batch path: one step at B=64 against 4 micro-steps of 16 rows
    with gradient accumulation (same tokens); gradients to the gradient bar,
    each update to the oracle's AdamW of its own gradients, and the two
    updates to each other within the t = 1 sensitivity of AdamW.  Also the
    per-position losses of one sequence of the big batch against the oracle."""
    torch = torch_gpu()
    cfg = synth.GPT2_124M
    hp = synth.HP_124M
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 4)
    stream = synth.zipf_tokens(64 * 1024 + 1, cfg.V, 1.1, 50)
    x, y = synth.shifted_pair(stream, 64, 1024)
    say("gpt2 124M B=64 step")
    torch.cuda.reset_peak_memory_stats()
    big = bt.GPT2(cfg, hp, 64, 1024)
    big.load_params(synth.flatten(cfg, params))
    rows = torch.zeros(64 * 1024, device="cuda")
    d_loss = torch.zeros(1, device="cuda")
    big.fwd_bwd(dev(torch, x), dev(torch, y), 1.0 / (64 * 1024), 0, d_loss, rows)
    big.optimizer_step(1, hp.lr)
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() / 2**30
    progress(f"peak device memory at B=64: {peak:.2f} GiB")
    # the large-batch step fits comfortably in the 288 GB of one MI355X: parameters,
    # gradients and moments (2 GB) plus about 0.85 GiB of activations per 1024 tokens
    assert 40.0 < peak < 80.0, peak
    g64 = _unflat(cfg, big.grads)
    p64, m64, v64 = _unflat(cfg, big.params), _unflat(cfg, big.m), _unflat(cfg, big.v)
    rows64 = host(rows).reshape(64, 1024)
    loss64 = float(d_loss.item())
    del big
    torch.cuda.empty_cache()
    say("gpt2 124M 4 x 16 accumulation")
    acc = bt.GPT2(cfg, hp, 16, 1024)
    acc.load_params(synth.flatten(cfg, params))
    d_loss2 = torch.zeros(1, device="cuda")
    for k in range(4):
        acc.fwd_bwd(dev(torch, x[16 * k:16 * k + 16]), dev(torch, y[16 * k:16 * k + 16]), 1.0 / (64 * 1024),
                    k > 0, d_loss2)
    acc.optimizer_step(1, hp.lr)
    torch.cuda.synchronize()
    assert abs(float(d_loss2.item()) - loss64) <= 1e-5 * loss64
    ga = _unflat(cfg, acc.grads)
    for name, _, _ in specs:
        assert_close_maxabs(ga[name], g64[name], GRAD_TOL, f"4x16 vs 64 grad {name}")
    _, c64 = _check_update(cfg, hp, specs, params, g64, p64, m64, v64, 1, what="B=64")
    _, cacc = _check_update(cfg, hp, specs, params, ga, _unflat(cfg, acc.params), _unflat(cfg, acc.m),
                            _unflat(cfg, acc.v), 1, what="4x16")
    _check_end_to_end(hp, specs, params, ga, g64, _unflat(cfg, acc.params), p64, cacc, c64)
    say("oracle forward of sequence 37 of the big batch")
    _, rr, _ = og.forward(cfg, params, x[37:38], y[37:38])
    assert np.allclose(rows64[37], rr, rtol=LOSS_TOL, atol=0)
