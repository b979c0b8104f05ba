"""Float64 GPT-2 training step (oracle; test infrastructure only).

Model: GPT-2 architecture figure caption (pre-normalised decoder blocks,
masked multi-head self-attention, GELU feed-forward sublayer, residual
connections, weight-tied embeddings) and the "Training hyperparameters" table.
Step: Algorithm "Distributed Data Parallel Training Step" on one rank --
micro-steps of forward, cross-entropy against the target and backward, with
gradients summed over micro-steps, then one optimizer step.

The backward is written out by hand from the chain rule; the optimizer is
AdamW with optional global-norm clipping.

Parameters are a dict name -> array with the names of the canonical flat
layout (token embedding "wte" [Vp, C], positions "wpe" [max_T, C], per layer
"h{l}.Wqkv" [C, 3C], "h{l}.Wo" [C, C], "h{l}.Wfc" [C, 4C], "h{l}.Wfp" [4C, C]
stored [in, out], biases and LN gains/biases, final "lnfg"/"lnfb").
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from . import ops

F64 = np.float64


def _p(params, name):
    return np.asarray(params[name], F64)


# --------------------------------------------------------------------------
# One pre-LN block:  x1 = x + Attn(LN1(x)) ;  y = x1 + MLP(LN2(x1))
#   Attn(u) = attention(u Wqkv + bqkv) Wo + bo
#   MLP(u)  = gelu(u Wfc + bfc) Wfp + bfp
# --------------------------------------------------------------------------
def block_fwd(x, p: Dict[str, np.ndarray], H: int, eps: float = 1e-5):
    """x [B, T, C] -> (y [B, T, C], cache)."""
    x = np.asarray(x, F64)
    B, T, C = x.shape
    ln1, mu1, rs1 = ops.layernorm_fwd(x, p["ln1g"], p["ln1b"], eps)
    qkv = ops.gemm(ln1.reshape(-1, C), p["Wqkv"]) + np.asarray(p["bqkv"], F64)
    att, lse = ops.attention_fwd(qkv.reshape(B, T, 3 * C), H)
    att = att.reshape(B * T, C)
    x1 = x + (ops.gemm(att, p["Wo"]) + np.asarray(p["bo"], F64)).reshape(B, T, C)
    ln2, mu2, rs2 = ops.layernorm_fwd(x1, p["ln2g"], p["ln2b"], eps)
    h = ops.gemm(ln2.reshape(-1, C), p["Wfc"]) + np.asarray(p["bfc"], F64)
    g = ops.gelu_fwd(h)
    y = x1 + (ops.gemm(g, p["Wfp"]) + np.asarray(p["bfp"], F64)).reshape(B, T, C)
    cache = dict(x=x, ln1=ln1, mu1=mu1, rs1=rs1, qkv=qkv, att=att, lse=lse, x1=x1,
                 ln2=ln2, mu2=mu2, rs2=rs2, h=h, g=g, H=H)
    return y, cache


def block_bwd(dy, p: Dict[str, np.ndarray], cache) -> Tuple[np.ndarray, Dict[str, np.ndarray]]:
    """dy [B, T, C] -> (dx [B, T, C], grads of the block's parameters)."""
    dy = np.asarray(dy, F64)
    B, T, C = dy.shape
    H = cache["H"]
    d2 = dy.reshape(-1, C)
    gr: Dict[str, np.ndarray] = {}
    # MLP down-projection
    gr["Wfp"] = ops.gemm(cache["g"], d2, trans_a=True)
    gr["bfp"] = d2.sum(axis=0)
    dg = ops.gemm(d2, p["Wfp"], trans_b=True)
    dh = ops.gelu_bwd(cache["h"], dg)
    # MLP up-projection
    gr["Wfc"] = ops.gemm(cache["ln2"].reshape(-1, C), dh, trans_a=True)
    gr["bfc"] = dh.sum(axis=0)
    dln2 = ops.gemm(dh, p["Wfc"], trans_b=True).reshape(B, T, C)
    dx1_ln, gr["ln2g"], gr["ln2b"] = ops.layernorm_bwd(dln2, cache["x1"], p["ln2g"],
                                                       cache["mu2"], cache["rs2"])
    dx1 = dy + dx1_ln
    d1 = dx1.reshape(-1, C)
    # attention output projection
    gr["Wo"] = ops.gemm(cache["att"], d1, trans_a=True)
    gr["bo"] = d1.sum(axis=0)
    datt = ops.gemm(d1, p["Wo"], trans_b=True)
    dqkv = ops.attention_bwd(datt.reshape(B, T, H, C // H),
                             cache["qkv"].reshape(B, T, 3 * C), H).reshape(-1, 3 * C)
    # QKV projection
    gr["Wqkv"] = ops.gemm(cache["ln1"].reshape(-1, C), dqkv, trans_a=True)
    gr["bqkv"] = dqkv.sum(axis=0)
    dln1 = ops.gemm(dqkv, p["Wqkv"], trans_b=True).reshape(B, T, C)
    dx_ln, gr["ln1g"], gr["ln1b"] = ops.layernorm_bwd(dln1, cache["x"], p["ln1g"],
                                                      cache["mu1"], cache["rs1"])
    return dx1 + dx_ln, gr


_BLOCK_KEYS = ("Wqkv", "Wo", "Wfc", "Wfp", "ln1g", "ln1b", "bqkv", "bo",
               "ln2g", "ln2b", "bfc", "bfp")


def _layer(params, l):
    return {k: _p(params, f"h{l}.{k}") for k in _BLOCK_KEYS}


# --------------------------------------------------------------------------
# Whole model
# --------------------------------------------------------------------------
def forward(cfg, params, tokens, targets):
    """Returns (mean loss, per-position loss rows, cache)."""
    tokens = np.asarray(tokens)
    B, T = tokens.shape
    x = ops.embedding_fwd(_p(params, "wte"), _p(params, "wpe"), tokens)
    caches = []
    for l in range(cfg.L):
        x, c = block_fwd(x, _layer(params, l), cfg.H, cfg.ln_eps)
        caches.append(c)
    lnf, muf, rsf = ops.layernorm_fwd(x, params["lnfg"], params["lnfb"], cfg.ln_eps)
    # tied LM head over every padded row; the loss uses the first V columns
    logits = ops.gemm(lnf.reshape(-1, cfg.C), _p(params, "wte"), trans_b=True)
    loss_rows, lse = ops.xent_fwd(logits, targets, cfg.V)
    cache = dict(tokens=tokens, targets=np.asarray(targets), caches=caches, xL=x,
                 lnf=lnf, muf=muf, rsf=rsf, logits=logits, B=B, T=T)
    return float(loss_rows.mean()), loss_rows, cache


def backward(cfg, params, cache, loss_scale: float):
    """Gradients of loss_scale * sum of per-position losses, as float64 dict.

    With loss_scale = 1/(B*T) this is the gradient of the mean loss; under
    k-step accumulation each micro-step uses 1/(B*T*k)."""
    B, T, C = cache["B"], cache["T"], cfg.C
    grads: Dict[str, np.ndarray] = {}
    dlogits = ops.xent_bwd(cache["logits"], cache["targets"], cfg.V, loss_scale)
    wte = _p(params, "wte")
    dlnf = ops.gemm(dlogits, wte).reshape(B, T, C)
    dwte_head = ops.gemm(dlogits, cache["lnf"].reshape(-1, C), trans_a=True)
    dx, grads["lnfg"], grads["lnfb"] = ops.layernorm_bwd(dlnf, cache["xL"], params["lnfg"],
                                                         cache["muf"], cache["rsf"])
    for l in reversed(range(cfg.L)):
        dx, gl = block_bwd(dx, _layer(params, l), cache["caches"][l])
        for k, v in gl.items():
            grads[f"h{l}.{k}"] = v
    dwte_emb, dwpe = ops.embedding_bwd(dx, cache["tokens"], cfg.Vp, cfg.max_T)
    grads["wte"] = dwte_head + dwte_emb
    grads["wpe"] = dwpe
    return grads


def fwd_bwd(cfg, params, tokens, targets, loss_scale=None):
    tokens = np.asarray(tokens)
    if loss_scale is None:
        loss_scale = 1.0 / tokens.size
    loss, rows, cache = forward(cfg, params, tokens, targets)
    return loss, rows, backward(cfg, params, cache, loss_scale)


def decay_mask(cfg, specs) -> Dict[str, float]:
    return {name: (1.0 if dec else 0.0) for name, _, dec in specs}


def optimizer_step(params, grads, m, v, t: int, hp, specs):
    """Global-norm clip (if hp.grad_clip > 0) then AdamW on every tensor.

    Returns (new params, new m, new v, grad norm, clip coefficient)."""
    names = [n for n, _, _ in specs]
    norm = ops.grad_norm(np.concatenate([np.asarray(grads[n], F64).ravel() for n in names]))
    coef = ops.clip_coef(norm, hp.grad_clip)
    np_, nm, nv = {}, {}, {}
    for name, _, dec in specs:
        np_[name], nm[name], nv[name] = ops.adamw(
            params[name], grads[name], m[name], v[name], t, hp.lr, hp.beta1, hp.beta2,
            hp.eps, hp.weight_decay, 1.0 if dec else 0.0, coef)
    return np_, nm, nv, norm, coef


def train_step(cfg, hp, specs, params, m, v, tokens, targets, t: int = 1, accum: int = 1):
    """Forward + backward over `accum` equal micro-batches (rows of tokens),
    summing gradients, then clip + AdamW.  Returns a dict with loss (mean
    over all positions), grads, params, m, v, norm, coef."""
    tokens = np.asarray(tokens)
    targets = np.asarray(targets)
    B = tokens.shape[0]
    assert B % accum == 0
    mb = B // accum
    scale = 1.0 / tokens.size
    grads = None
    loss = 0.0
    rows: List[np.ndarray] = []
    for k in range(accum):
        tk = tokens[k * mb:(k + 1) * mb]
        yk = targets[k * mb:(k + 1) * mb]
        lk, rk, cache = forward(cfg, params, tk, yk)
        gk = backward(cfg, params, cache, scale)
        del cache
        loss += lk / accum
        rows.append(rk)
        if grads is None:
            grads = gk
        else:
            for n in grads:
                grads[n] = grads[n] + gk[n]
    p1, m1, v1, norm, coef = optimizer_step(params, grads, m, v, t, hp, specs)
    return dict(loss=loss, loss_rows=np.concatenate(rows), grads=grads, params=p1,
                m=m1, v=v1, norm=norm, coef=coef)
