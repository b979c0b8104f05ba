"""Pins for the per-operation oracle (CPU only).

Each check is chosen so that a plausible slip in the oracle (dropped term,
wrong sign or index, transposed operand) fails: naive loops, closed forms,
exact identities, central finite differences and independent library
routines (torch CPU float64) that do not share the oracle's code.
"""
import math

import numpy as np
import pytest

from oracle import ops

RNG = np.random.Generator(np.random.PCG64(1234))


def central_diff(f, x, idx, h=1e-6):
    xp = x.copy()
    xm = x.copy()
    xp[idx] += h
    xm[idx] -= h
    return (f(xp) - f(xm)) / (2 * h)


# ----------------------------------------------------------------------- GEMM
@pytest.mark.parametrize("ta,tb", [(False, False), (False, True), (True, False), (True, True)])
def test_gemm_naive_triple_loop(ta, tb):
    M, N, K = 5, 7, 9
    A = RNG.standard_normal((K, M) if ta else (M, K))
    B = RNG.standard_normal((N, K) if tb else (K, N))
    C = ops.gemm(A, B, ta, tb)
    for i in range(M):
        for j in range(N):
            s = 0.0
            for k in range(K):
                a = A[k][i] if ta else A[i][k]
                b = B[j][k] if tb else B[k][j]
                s += a * b
            assert abs(C[i, j] - s) <= 1e-12 * max(1.0, abs(s))


def test_gemm_identity_and_permutation():
    A = RNG.standard_normal((6, 6)).astype(np.float32)
    assert np.array_equal(ops.gemm(A, np.eye(6)), A.astype(np.float64))
    perm = RNG.permutation(6)
    P = np.eye(6)[perm]
    assert np.array_equal(ops.gemm(P, A), A[perm].astype(np.float64))
    assert np.array_equal(ops.gemm(A, P, trans_b=True), A[:, perm].astype(np.float64))


# ------------------------------------------------------------------ LayerNorm
def test_layernorm_moments():
    x = RNG.standard_normal((7, 33)) * 3 + 1.5
    eps = 1e-5
    y, mean, rstd = ops.layernorm_fwd(x, np.ones(33), np.zeros(33), eps)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-13)
    var = x.var(axis=1)
    assert np.allclose(y.var(axis=1), var / (var + eps), rtol=1e-12)
    # rows of a constant input normalise to exactly beta
    yc, _, _ = ops.layernorm_fwd(np.full((2, 8), 3.0), np.full(8, 2.0), np.arange(8.0), eps)
    assert np.allclose(yc, np.arange(8.0)[None], atol=1e-12)


def test_layernorm_bwd_invariants_and_fd():
    M, C = 5, 12
    x = RNG.standard_normal((M, C))
    g = 1 + 0.1 * RNG.standard_normal(C)
    b = 0.1 * RNG.standard_normal(C)
    dy = RNG.standard_normal((M, C))
    _, mean, rstd = ops.layernorm_fwd(x, g, b)
    dx, dg, db = ops.layernorm_bwd(dy, x, g, mean, rstd)
    # with gamma = 1 (and eps = 0, where sum(xhat^2) = C exactly) the input
    # gradient is orthogonal to 1 and to xhat
    _, m1, r1 = ops.layernorm_fwd(x, np.ones(C), np.zeros(C), 0.0)
    dx1, _, _ = ops.layernorm_bwd(dy, x, np.ones(C), m1, r1)
    xhat = (x - m1[:, None]) * r1[:, None]
    assert np.allclose(dx1.sum(axis=1), 0, atol=1e-12)
    assert np.allclose((dx1 * xhat).sum(axis=1), 0, atol=1e-12)

    def L(xx):
        return float((ops.layernorm_fwd(xx, g, b)[0] * dy).sum())

    for idx in [(0, 0), (2, 5), (4, 11)]:
        assert abs(central_diff(L, x, idx) - dx[idx]) < 1e-7
    Lg = lambda gg: float((ops.layernorm_fwd(x, gg, b)[0] * dy).sum())
    Lb = lambda bb: float((ops.layernorm_fwd(x, g, bb)[0] * dy).sum())
    for j in [0, 7, 11]:
        assert abs(central_diff(Lg, g, j) - dg[j]) < 1e-7
        assert abs(central_diff(Lb, b, j) - db[j]) < 1e-7


def test_layernorm_vs_torch(torch_cpu):
    torch = torch_cpu
    M, C = 6, 20
    x = RNG.standard_normal((M, C))
    g = 1 + 0.1 * RNG.standard_normal(C)
    b = 0.1 * RNG.standard_normal(C)
    dy = RNG.standard_normal((M, C))
    xt = torch.tensor(x, requires_grad=True)
    gt = torch.tensor(g, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = torch.nn.functional.layer_norm(xt, (C,), gt, bt, eps=1e-5)
    yt.backward(torch.tensor(dy))
    y, mean, rstd = ops.layernorm_fwd(x, g, b)
    dx, dg, db = ops.layernorm_bwd(dy, x, g, mean, rstd)
    assert np.allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(dg, gt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------- GELU
def test_gelu_identities():
    x = RNG.standard_normal(1000) * 4
    assert np.allclose(ops.gelu_fwd(x) - ops.gelu_fwd(-x), x, atol=1e-13)
    assert ops.gelu_fwd(np.array([0.0]))[0] == 0.0
    assert abs(ops.gelu_grad(np.array([0.0]))[0] - 0.5) < 1e-15
    # far tails: identity for large positive, zero for large negative
    assert abs(ops.gelu_fwd(np.array([30.0]))[0] - 30.0) < 1e-12
    assert abs(ops.gelu_fwd(np.array([-30.0]))[0]) < 1e-12


def test_gelu_grad_fd_and_torch(torch_cpu):
    torch = torch_cpu
    x = np.linspace(-6, 6, 101)
    h = 1e-6
    fd = (ops.gelu_fwd(x + h) - ops.gelu_fwd(x - h)) / (2 * h)
    assert np.allclose(ops.gelu_grad(x), fd, atol=1e-8)
    xt = torch.tensor(x, requires_grad=True)
    yt = torch.nn.functional.gelu(xt, approximate="tanh")
    dy = RNG.standard_normal(x.shape)
    yt.backward(torch.tensor(dy))
    assert np.allclose(ops.gelu_fwd(x), yt.detach().numpy(), rtol=1e-13, atol=1e-14)
    assert np.allclose(ops.gelu_bwd(x, dy), xt.grad.numpy(), rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ Attention
def _qkv(B, T, H, hd, scale=1.0):
    return RNG.standard_normal((B, T, 3, H, hd)) * scale


def test_attention_brute_force():
    B, T, H, hd = 2, 5, 2, 3
    qkv = _qkv(B, T, H, hd)
    out, lse = ops.attention_fwd(qkv, H)
    for b in range(B):
        for h in range(H):
            for i in range(T):
                s = [sum(qkv[b, i, 0, h, d] * qkv[b, j, 1, h, d] for d in range(hd)) / math.sqrt(hd)
                     for j in range(i + 1)]
                den = sum(math.exp(v) for v in s)
                assert abs(lse[b, h, i] - math.log(den)) < 1e-12
                for d in range(hd):
                    o = sum(math.exp(s[j]) / den * qkv[b, j, 2, h, d] for j in range(i + 1))
                    assert abs(out[b, i, h, d] - o) < 1e-12


def test_attention_closed_forms():
    B, T, H, hd = 1, 9, 3, 4
    qkv = _qkv(B, T, H, hd)
    qkv[:, :, 0] = 0.0  # Q = 0: uniform weights over the causal prefix
    out, lse = ops.attention_fwd(qkv, H)
    v = qkv[:, :, 2]
    prefix_mean = np.cumsum(v, axis=1) / np.arange(1, T + 1)[None, :, None, None]
    assert np.allclose(out, prefix_mean, atol=1e-13)
    assert np.allclose(lse, np.log(np.arange(1, T + 1))[None, None, :], atol=1e-13)
    # T = 1: output is V
    q1 = _qkv(2, 1, 2, 5)
    o1, _ = ops.attention_fwd(q1, 2)
    assert np.allclose(o1, q1[:, :, 2], atol=1e-14)


def test_attention_causality():
    B, T, H, hd = 1, 8, 2, 4
    qkv = _qkv(B, T, H, hd)
    out, _ = ops.attention_fwd(qkv, H)
    qkv2 = qkv.copy()
    qkv2[:, 5:] += RNG.standard_normal(qkv2[:, 5:].shape)
    out2, _ = ops.attention_fwd(qkv2, H)
    assert np.array_equal(out[:, :5], out2[:, :5])
    assert not np.allclose(out[:, 5:], out2[:, 5:])


def test_attention_bwd_fd_and_torch(torch_cpu):
    torch = torch_cpu
    B, T, H, hd = 2, 6, 2, 4
    qkv = _qkv(B, T, H, hd)
    dout = RNG.standard_normal((B, T, H, hd))
    dqkv = ops.attention_bwd(dout, qkv, H)

    def L(z):
        return float((ops.attention_fwd(z, H)[0] * dout).sum())

    for idx in [(0, 0, 0, 0, 0), (1, 3, 1, 1, 2), (0, 5, 2, 0, 3), (1, 2, 0, 1, 1)]:
        assert abs(central_diff(L, qkv, idx) - dqkv[idx]) < 1e-8
    t = torch.tensor(qkv, requires_grad=True)
    q = t[:, :, 0].transpose(1, 2)
    k = t[:, :, 1].transpose(1, 2)
    v = t[:, :, 2].transpose(1, 2)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    o.transpose(1, 2).backward(torch.tensor(dout))
    out, _ = ops.attention_fwd(qkv, H)
    assert np.allclose(out, o.transpose(1, 2).detach().numpy(), atol=1e-13)
    assert np.allclose(dqkv, t.grad.numpy(), atol=1e-12)


# --------------------------------------------------------------- Cross-entropy
def test_softmax_rows_sum_to_one():
    z = RNG.standard_normal((10, 37)) * 5
    p = ops.softmax_rows(z)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-14)
    assert (p > 0).all()


def test_xent_closed_forms():
    M, V, Vp = 4, 50257, 50304
    loss, lse = ops.xent_fwd(np.zeros((M, Vp)), np.array([0, 7, 50000, 50256]), V)
    assert np.allclose(loss, math.log(V), rtol=0, atol=1e-12)  # ln V, not ln Vp
    assert abs(math.log(V) - 10.824905) < 1e-6
    # one-hot peaked logits: l = ln(1 + (V-1) e^-a)
    V2 = 31
    for a in [-2.0, 0.0, 3.0, 12.0]:
        z = np.zeros((1, V2 + 3))
        z[0, 4] = a
        z[0, V2:] = 100.0  # padded columns must not enter the softmax
        l, _ = ops.xent_fwd(z, np.array([4]), V2)
        assert abs(l[0] - math.log1p((V2 - 1) * math.exp(-a))) < 1e-12


def test_xent_bwd_fd_and_torch(torch_cpu):
    torch = torch_cpu
    M, V, Vp = 6, 13, 16
    z = RNG.standard_normal((M, Vp)) * 2
    y = RNG.integers(0, V, M)
    scale = 1.0 / M
    dz = ops.xent_bwd(z, y, V, scale)
    assert np.allclose(dz[:, V:], 0)
    assert np.allclose(dz.sum(axis=1), 0, atol=1e-15)
    loss, _ = ops.xent_fwd(z, y, V)
    assert (loss >= 0).all()

    def L(zz):
        return float(ops.xent_fwd(zz, y, V)[0].sum() * scale)

    for idx in [(0, 0), (3, int(y[3])), (5, 12), (2, 14)]:
        assert abs(central_diff(L, z, idx) - dz[idx]) < 1e-9
    zt = torch.tensor(z[:, :V], requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="mean")
    lt.backward()
    assert abs(lt.item() - loss.mean()) < 1e-13
    assert np.allclose(dz[:, :V], zt.grad.numpy(), atol=1e-14)


# ------------------------------------------------------------------ Embedding
def test_embedding_brute_force():
    V, T, C, B = 11, 4, 3, 3
    wte = RNG.standard_normal((V, C))
    wpe = RNG.standard_normal((6, C))
    tok = RNG.integers(0, V, (B, T))
    tok[0, 0] = tok[1, 2] = tok[2, 3] = 5  # repeated id accumulates
    x0 = ops.embedding_fwd(wte, wpe, tok)
    dx0 = RNG.standard_normal((B, T, C))
    dwte, dwpe = ops.embedding_bwd(dx0, tok, V, 6)
    ewte = np.zeros((V, C))
    ewpe = np.zeros((6, C))
    for b in range(B):
        for t in range(T):
            assert np.array_equal(x0[b, t], wte[tok[b, t]] + wpe[t])
            ewte[tok[b, t]] += dx0[b, t]
            ewpe[t] += dx0[b, t]
    assert np.allclose(dwte, ewte, atol=1e-14)
    assert np.allclose(dwpe, ewpe, atol=1e-14)


# ---------------------------------------------------------------------- AdamW
def test_adamw_closed_form_t1():
    rng = np.random.default_rng(277)  # own stream: independent of test order
    n = 64
    p0 = rng.standard_normal(n)
    g = rng.standard_normal(n) * 1e-2
    g[3] = 0.0
    lr, wd, eps = 3e-4, 0.1, 1e-8
    mask = (np.arange(n) < 40).astype(float)
    p1, m1, v1 = ops.adamw(p0, g, np.zeros(n), np.zeros(n), 1, lr, 0.9, 0.999, eps, wd, mask)
    expect = p0 - lr * (wd * p0 * mask + g / (np.abs(g) + eps))
    # the closed form and the oracle's update order round differently: a few
    # ulps of the parameter
    ulp = np.finfo(np.float64).eps
    assert np.all(np.abs(p1 - expect) <= 4 * ulp * np.maximum(np.abs(p0), 1.0))
    # g = 0: only decay acts (p0 - lr wd p0 and p0 (1 - lr wd) differ only in rounding)
    assert abs(p1[3] - p0[3] * (1 - lr * wd)) <= 4 * ulp * abs(p0[3])
    # clip coefficient c scales g before the moments; at t=1 the update is
    # sign-like so only m and v see it
    _, mc, vc = ops.adamw(p0, g, np.zeros(n), np.zeros(n), 1, lr, 0.9, 0.999, eps, wd, mask, 0.25)
    assert np.allclose(mc, 0.25 * m1) and np.allclose(vc, 0.0625 * v1)


def test_adamw_vs_torch_multi_step(torch_cpu):
    torch = torch_cpu
    n_dec, n_nodec = 24, 8
    lr, b1, b2, eps, wd = 6e-4, 0.9, 0.95, 1e-8, 0.1
    p = RNG.standard_normal(n_dec + n_nodec)
    pd = torch.tensor(p[:n_dec].copy(), requires_grad=True)
    pn = torch.tensor(p[n_dec:].copy(), requires_grad=True)
    opt = torch.optim.AdamW([{"params": [pd], "weight_decay": wd},
                             {"params": [pn], "weight_decay": 0.0}],
                            lr=lr, betas=(b1, b2), eps=eps)
    mask = np.r_[np.ones(n_dec), np.zeros(n_nodec)]
    m = np.zeros_like(p)
    v = np.zeros_like(p)
    for t in range(1, 5):
        g = RNG.standard_normal(p.shape) * 0.5
        pd.grad = torch.tensor(g[:n_dec].copy())
        pn.grad = torch.tensor(g[n_dec:].copy())
        total = torch.nn.utils.clip_grad_norm_([pd, pn], 1.0)
        opt.step()
        norm = ops.grad_norm(g)
        assert abs(norm - total.item()) < 1e-12
        p, m, v = ops.adamw(p, g, m, v, t, lr, b1, b2, eps, wd, mask, ops.clip_coef(norm, 1.0))
    assert np.allclose(p[:n_dec], pd.detach().numpy(), rtol=0, atol=1e-14)
    assert np.allclose(p[n_dec:], pn.detach().numpy(), rtol=0, atol=1e-14)


def test_clip_coef():
    assert ops.clip_coef(0.5, 1.0) == 1.0
    assert abs(ops.clip_coef(4.0, 1.0) - 1.0 / (4.0 + 1e-6)) < 1e-16
    assert ops.clip_coef(100.0, 0.0) == 1.0
    assert ops.grad_norm(np.array([3.0, 4.0])) == 5.0
