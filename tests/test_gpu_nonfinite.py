"""Failure handling of the composed step on the GPU (numerical values only,
no faults): a non-finite gradient norm skips the AdamW update and is
reported, and a target outside the vocabulary turns its row's loss and
gradient into NaN in every cross-entropy entry point (so a step over it is
reported and skipped rather than trained toward a wrong class)."""
import dataclasses
import math

import numpy as np
import pytest

from paper_2606_24780_amd import bt, synth
from tests.golden.make_tiny_step import tiny_inputs
from tests.gpu_util import dev, host, say, torch_gpu

pytestmark = pytest.mark.gpu


def _model(torch, hp=None):
    cfg = synth.TINY
    hp = hp or synth.HP_TINY
    _, params, x, y = tiny_inputs()
    model = bt.GPT2(cfg, hp, x.shape[0], x.shape[1])
    model.load_params(synth.flatten(cfg, params))
    return model, dev(torch, x), dev(torch, y)


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
@pytest.mark.parametrize("clip", [0.0, 1.0])
def test_optimizer_step_skips_non_finite_gradient(bad, clip):
    torch = torch_gpu()
    say(f"non-finite gradient {bad} clip={clip}")
    hp = dataclasses.replace(synth.HP_TINY, grad_clip=clip)
    model, x, y = _model(torch, hp)
    d_loss = torch.zeros(1, device="cuda")
    model.fwd_bwd(x, y, 1.0 / x.numel(), 0, d_loss)
    # a first, finite step gives nonzero moments to protect
    model.optimizer_step(1, hp.lr)
    model.fwd_bwd(x, y, 1.0 / x.numel(), 0, d_loss)
    g = model.grads
    g[g.numel() // 3] = bad
    p0, s0 = model.params.clone(), model.opt_state.clone()
    model.optimizer_step(2, hp.lr)
    torch.cuda.synchronize()
    assert torch.equal(model.params, p0), "parameters changed by a skipped step"
    assert torch.equal(model.opt_state, s0), "moments changed by a skipped step"
    _, norm, coef = model.read_scalars()
    assert not math.isfinite(norm) and math.isnan(coef)


def test_train_step_reports_non_finite_and_keeps_state():
    torch = torch_gpu()
    say("train step with an out-of-vocabulary target")
    model, x, y = _model(torch)
    loss1 = model.train_step(x, y)
    assert math.isfinite(loss1) and model.step_count == 1
    p0, s0 = model.params.clone(), model.opt_state.clone()
    y_bad = y.clone()
    y_bad[0, 5] = synth.TINY.V  # outside [0, V)
    with pytest.raises(bt.BTNonFiniteError) as ei:
        model.train_step(x, y_bad)
    assert "non-finite gradient norm" in str(ei.value)
    assert bt.lib().bt_last_status() == bt.BT_ENONFINITE
    torch.cuda.synchronize()
    assert torch.equal(model.params, p0) and torch.equal(model.opt_state, s0)
    assert model.step_count == 1
    # the next valid step proceeds from the unchanged state, and clears the status
    loss2 = model.train_step(x, y)
    assert math.isfinite(loss2) and model.step_count == 2
    assert bt.lib().bt_last_status() == 0 and bt.lib().bt_last_error() == b""


@pytest.mark.parametrize("M,V,Vp", [(6, 50257, 50304), (5, 300, 300), (4, 13, 16)])
def test_xent_invalid_target_rows_are_nan(M, V, Vp):
    torch = torch_gpu()
    say(f"xent invalid targets M={M} V={V}")
    rng = np.random.Generator(np.random.PCG64(7))
    z = (rng.standard_normal((M, Vp)) * 2).astype(np.float32)
    y = rng.integers(0, V, M).astype(np.int32)
    y[1], y[3] = -1, V  # rows 1 and 3 invalid
    scale = 1.0 / M
    zd, yd = dev(torch, z), dev(torch, y)
    loss = torch.empty(M, device="cuda")
    lse = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fwd(zd, yd, loss, lse, M, V, Vp)
    dz = torch.empty_like(zd)
    bt.bt_softmax_xent_bwd(zd, lse, yd, dz, scale, M, V, Vp)
    loss2 = torch.empty(M, device="cuda")
    lse2 = torch.empty(M, device="cuda")
    zf = zd.clone()
    bt.bt_softmax_xent_fused(zf, yd, loss2, lse2, scale, M, V, Vp)
    good = np.array([r not in (1, 3) for r in range(M)])
    for name, l_, g_ in (("unfused", host(loss), host(dz)), ("fused", host(loss2), host(zf))):
        assert np.isnan(l_[~good]).all() and np.isfinite(l_[good]).all(), name
        assert np.isnan(g_[~good, :V]).all(), f"{name}: invalid rows must be NaN in columns < V"
        assert (g_[:, V:] == 0).all(), f"{name}: padded columns must be 0"
        assert np.isfinite(g_[good]).all(), name
    # the two paths agree on the valid rows
    assert np.allclose(host(dz)[good], host(zf)[good], rtol=0, atol=1e-6 * scale)
