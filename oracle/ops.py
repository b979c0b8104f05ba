"""Per-operation float64 definitions (oracle; test infrastructure only).

Each function takes numpy arrays (any float dtype; promoted to float64) and
returns float64 arrays.  No blocking, fusion or reordering beyond the plain
definition of the operation.
"""
from __future__ import annotations

import math

import numpy as np

F64 = np.float64


def _f(x):
    return np.asarray(x, dtype=F64)


# --------------------------------------------------------------------------
# Dense products.  "Kernel Design and Optimization" and "Implementation:
# Native GEMM Library": C = op(A) op(B) for the QKV, attention-output and MLP
# projections in forward and both backward layouts.
# --------------------------------------------------------------------------
def gemm(a, b, trans_a: bool = False, trans_b: bool = False):
    """C = op(A) @ op(B) in float64 (library matmul as a single step)."""
    a = _f(a)
    b = _f(b)
    if trans_a:
        a = a.T
    if trans_b:
        b = b.T
    return a @ b


# --------------------------------------------------------------------------
# LayerNorm.  Pre-normalised blocks (GPT-2 architecture figure caption);
# stable mean/variance reductions ("Kernel Design": mathematically stable
# algorithms; Related Work cites Welford).  Reading: eps = 1e-5 inside the
# square root, biased variance (divide by C).
# --------------------------------------------------------------------------
def layernorm_fwd(x, gamma, beta, eps: float = 1e-5):
    """y = gamma * (x - mean) * rstd + beta over the last axis.

    Returns (y, mean, rstd)."""
    x = _f(x)
    mean = x.mean(axis=-1)
    xc = x - mean[..., None]
    var = (xc * xc).mean(axis=-1)
    rstd = 1.0 / np.sqrt(var + eps)
    y = xc * rstd[..., None] * _f(gamma) + _f(beta)
    return y, mean, rstd


def layernorm_bwd(dy, x, gamma, mean, rstd):
    """Gradient of layernorm_fwd.

    With xhat = (x - mean) * rstd and g = dy * gamma (per row of C):
      dx = rstd * (g - mean(g) - xhat * mean(g * xhat))
      dgamma = sum_rows dy * xhat,  dbeta = sum_rows dy.
    Returns (dx, dgamma, dbeta)."""
    dy = _f(dy)
    x = _f(x)
    xhat = (x - _f(mean)[..., None]) * _f(rstd)[..., None]
    g = dy * _f(gamma)
    dx = _f(rstd)[..., None] * (g - g.mean(axis=-1, keepdims=True)
                               - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    red = tuple(range(dy.ndim - 1))
    dgamma = (dy * xhat).sum(axis=red)
    dbeta = dy.sum(axis=red)
    return dx, dgamma, dbeta


# --------------------------------------------------------------------------
# GELU (GPT-2 architecture figure caption, "GELU feed-forward sublayer";
# Appendix "GELU Forward / Backward").  Reading: the tanh form.
# --------------------------------------------------------------------------
_K0 = math.sqrt(2.0 / math.pi)
_K1 = 0.044715


def gelu_fwd(x):
    """0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    x = _f(x)
    return 0.5 * x * (1.0 + np.tanh(_K0 * (x + _K1 * x ** 3)))


def gelu_grad(x):
    """d/dx of gelu_fwd."""
    x = _f(x)
    u = _K0 * (x + _K1 * x ** 3)
    t = np.tanh(u)
    du = _K0 * (1.0 + 3.0 * _K1 * x * x)
    return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * du


def gelu_bwd(x, dy):
    return _f(dy) * gelu_grad(x)


# --------------------------------------------------------------------------
# Causal multi-head self-attention (GPT-2 figure caption: masked multi-head
# self-attention; Appendix "Attention Forward / Backward", causal case).
# Reading: scale 1/sqrt(hd); key j is visible to query i iff j <= i; no
# dropout (hyper-parameter table: dropout 0).  qkv is laid out [B, T, 3, H, hd].
# --------------------------------------------------------------------------
def split_qkv(qkv, H: int):
    qkv = _f(qkv)
    qkv = qkv.reshape(qkv.shape[0], qkv.shape[1], 3, H, -1)
    q = qkv[:, :, 0].transpose(0, 2, 1, 3)  # [B, H, T, hd]
    k = qkv[:, :, 1].transpose(0, 2, 1, 3)
    v = qkv[:, :, 2].transpose(0, 2, 1, 3)
    return q, k, v


def causal_scores(q, k):
    """S = q k^T / sqrt(hd) with masked entries set to -inf."""
    hd = q.shape[-1]
    s = (q @ np.swapaxes(k, -1, -2)) / math.sqrt(hd)
    T = q.shape[-2]
    mask = np.triu(np.ones((T, T), dtype=bool), k=1)
    s = np.where(mask, -np.inf, s)
    return s


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def logsumexp_rows(s):
    m = s.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(s - m).sum(axis=-1, keepdims=True)))[..., 0]


def attention_fwd(qkv, H: int):
    """O = softmax(mask(Q K^T / sqrt(hd))) V per (batch, head).

    Returns (out [B, T, H, hd], lse [B, H, T]) where lse is the natural-log
    sum of exponentials of each masked score row."""
    q, k, v = split_qkv(qkv, H)
    s = causal_scores(q, k)
    p = softmax_rows(s)
    o = p @ v  # [B, H, T, hd]
    return o.transpose(0, 2, 1, 3), logsumexp_rows(s)


def attention_bwd(dout, qkv, H: int):
    """Gradient of attention_fwd with respect to qkv (layout [B, T, 3, H, hd]).

    Plain chain rule through the softmax Jacobian:
      dV = P^T dO, dP = dO V^T, dS_ij = P_ij (dP_ij - sum_k P_ik dP_ik),
      dQ = dS K / sqrt(hd), dK = dS^T Q / sqrt(hd)."""
    q, k, v = split_qkv(qkv, H)
    hd = q.shape[-1]
    s = causal_scores(q, k)
    p = softmax_rows(s)
    do = _f(dout).transpose(0, 2, 1, 3)
    dv = np.swapaxes(p, -1, -2) @ do
    dp = do @ np.swapaxes(v, -1, -2)
    ds = p * (dp - (p * dp).sum(axis=-1, keepdims=True))
    dq = ds @ k / math.sqrt(hd)
    dk = np.swapaxes(ds, -1, -2) @ q / math.sqrt(hd)
    B, _, T, _ = q.shape
    dqkv = np.empty((B, T, 3, H, hd), F64)
    dqkv[:, :, 0] = dq.transpose(0, 2, 1, 3)
    dqkv[:, :, 1] = dk.transpose(0, 2, 1, 3)
    dqkv[:, :, 2] = dv.transpose(0, 2, 1, 3)
    return dqkv


# --------------------------------------------------------------------------
# Sparse (integer-target) softmax cross-entropy (Algorithm "Distributed Data
# Parallel Training Step": loss = cross-entropy of FORWARD(x) against target;
# Appendix "Sparse Cross-Entropy Loss Forward / Backward").  Reading: the
# softmax runs over the first V columns only; padded columns (V..Vp) get zero
# gradient; the mean is over all positions, scaled by 1/k under k-step
# accumulation.
# --------------------------------------------------------------------------
def xent_fwd(logits, targets, V: int):
    """Per-row loss l_m = logsumexp(z_m[:V]) - z_m[y_m]; returns (loss_rows, lse)."""
    z = _f(logits)[:, :V]
    y = np.asarray(targets).reshape(-1).astype(np.int64)
    lse = logsumexp_rows(z)
    loss = lse - z[np.arange(z.shape[0]), y]
    return loss, lse


def xent_bwd(logits, targets, V: int, scale: float):
    """dz = (softmax(z[:V]) - onehot(y)) * scale; columns >= V are 0."""
    z = _f(logits)
    y = np.asarray(targets).reshape(-1).astype(np.int64)
    dz = np.zeros_like(z)
    p = softmax_rows(z[:, :V])
    p[np.arange(z.shape[0]), y] -= 1.0
    dz[:, :V] = p * scale
    return dz


# --------------------------------------------------------------------------
# Embeddings (GPT-2 figure caption: weight-tied embeddings; learned positions).
# --------------------------------------------------------------------------
def embedding_fwd(wte, wpe, tokens):
    tok = np.asarray(tokens)
    T = tok.shape[1]
    return _f(wte)[tok] + _f(wpe)[:T][None]


def embedding_bwd(dx0, tokens, Vp: int, max_T: int):
    """dwte[v] = sum over positions with token v of dx0; dwpe[t] = sum_b dx0[b, t]."""
    dx0 = _f(dx0)
    tok = np.asarray(tokens)
    B, T, C = dx0.shape
    dwte = np.zeros((Vp, C), F64)
    np.add.at(dwte, tok.reshape(-1), dx0.reshape(-1, C))
    dwpe = np.zeros((max_T, C), F64)
    dwpe[:T] = dx0.sum(axis=0)
    return dwte, dwpe


# --------------------------------------------------------------------------
# Global gradient-norm clip (hyper-parameter table: gradient clip 1.0).
# Reading: global L2 norm over every gradient after accumulation,
# coefficient min(1, clip / (norm + 1e-6)).
# --------------------------------------------------------------------------
def grad_norm(g):
    g = _f(g)
    return math.sqrt(float(np.dot(g.ravel(), g.ravel())))


def clip_coef(norm: float, clip: float) -> float:
    if clip <= 0:
        return 1.0
    return min(1.0, clip / (norm + 1e-6))


# --------------------------------------------------------------------------
# AdamW ("Implementation: Horizontal Tensor Fusion"; hyper-parameter table:
# beta1 0.9, beta2 0.95, eps 1e-8, weight decay 0.1).  Reading: decoupled
# decay from the pre-update parameter, applied to 2-D tensors only; bias
# corrections with the step count t starting at 1; eps outside the root.
# --------------------------------------------------------------------------
def adamw(p, g, m, v, t: int, lr: float, beta1: float, beta2: float, eps: float,
          weight_decay: float, decay_mask, grad_scale: float = 1.0):
    """One AdamW step; returns (p, m, v) as new float64 arrays."""
    p = _f(p)
    g = _f(g) * grad_scale
    m = beta1 * _f(m) + (1.0 - beta1) * g
    v = beta2 * _f(v) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    p = p - lr * weight_decay * p * _f(decay_mask) - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v
