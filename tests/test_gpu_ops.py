"""Parity of the memory-bound kernels against the float64 oracle:
LayerNorm fwd/bwd, GELU fwd/bwd, sparse cross-entropy (fwd, bwd, fused),
AdamW, global grad norm + clip, embeddings fwd/bwd and column sums.

Sizes span the GPT-2 124M shapes (16384 rows of 768, 50,304-column logits,
the 124.5M-element parameter arena) and small ragged ones.  Bars: 1e-5 of
max-abs for values, 1e-4 of max-abs for gradients of the model, 1e-6 of
max-abs for the AdamW update on identical inputs; integer/index results and
the zero gradient of padded columns exactly."""
import math

import numpy as np
import pytest

from oracle import ops
from paper_2606_24780_amd import bt, synth
from tests.gpu_util import assert_close_maxabs, dev, host, say, torch_gpu

pytestmark = pytest.mark.gpu
RNG = np.random.Generator(np.random.PCG64(4))


# ------------------------------------------------------------------ LayerNorm
# Row widths of 1, 2, 3, 4, 6, 8, 12 and 16 float4 per lane (each register
# case of the kernels; 4096 is the largest C), ragged row counts.
@pytest.mark.parametrize("M,C", [(1, 64), (37, 768), (16384, 768), (5, 4096), (9, 1000), (2048, 3072),
                                 (300, 2600), (33, 400), (17, 1300), (13, 1800), (9, 3500)])
def test_layernorm(M, C):
    torch = torch_gpu()
    say(f"layernorm M={M} C={C}")
    x = (RNG.standard_normal((M, C)) * 2 + 0.5).astype(np.float32)
    g = (1 + 0.1 * RNG.standard_normal(C)).astype(np.float32)
    b = (0.1 * RNG.standard_normal(C)).astype(np.float32)
    dy = RNG.standard_normal((M, C)).astype(np.float32)
    dx0 = RNG.standard_normal((M, C)).astype(np.float32)
    dg0 = RNG.standard_normal(C).astype(np.float32)
    db0 = RNG.standard_normal(C).astype(np.float32)
    xd, gd, bd = dev(torch, x), dev(torch, g), dev(torch, b)
    y = torch.empty_like(xd)
    mean = torch.empty(M, device="cuda")
    rstd = torch.empty(M, device="cuda")
    bt.bt_layernorm_fwd(xd, gd, bd, y, mean, rstd, M, C, 1e-5)
    ry, rm, rr = ops.layernorm_fwd(x, g, b, 1e-5)
    assert_close_maxabs(host(y), ry, 1e-5, "y")
    assert_close_maxabs(host(mean), rm, 1e-5, "mean")
    assert_close_maxabs(host(rstd), rr, 1e-5, "rstd")
    rdx, rdg, rdb = ops.layernorm_bwd(dy, x, g, rm, rr)
    for beta in (0.0, 1.0):
        dx, dgd, dbd = dev(torch, dx0), dev(torch, dg0), dev(torch, db0)
        bt.bt_layernorm_bwd(dev(torch, dy), xd, gd, mean, rstd, dx, dgd, dbd, beta, beta, M, C)
        assert_close_maxabs(host(dx), rdx + beta * dx0, 1e-5, f"dx beta={beta}")
        assert_close_maxabs(host(dgd), rdg + beta * dg0, 1e-5, f"dgamma beta={beta}")
        assert_close_maxabs(host(dbd), rdb + beta * db0, 1e-5, f"dbeta beta={beta}")


# ----------------------------------------------------------------------- GELU
@pytest.mark.parametrize("n", [4, 4 * 1001, 16384 * 3072])
def test_gelu(n):
    torch = torch_gpu()
    say(f"gelu n={n}")
    x = (RNG.standard_normal(n) * 3).astype(np.float32)
    dy = RNG.standard_normal(n).astype(np.float32)
    xd = dev(torch, x)
    y = torch.empty_like(xd)
    bt.bt_gelu_fwd(xd, y)
    assert_close_maxabs(host(y), ops.gelu_fwd(x), 1e-5, "gelu")
    dyd = dev(torch, dy)
    bt.bt_gelu_bwd(xd, dyd, dyd)  # in place over dy
    assert_close_maxabs(host(dyd), ops.gelu_bwd(x, dy), 1e-5, "gelu bwd (in place)")


# --------------------------------------------------------------- Cross-entropy
# Vocabularies of 1, 2, 4, 8, 13 and 16 float4 per thread of the row kernel
# (the last at the largest supported Vp, 65,536), ragged V < Vp; 50,304 takes
# the streaming kernel.
@pytest.mark.parametrize("M,V,Vp", [(5, 256, 256), (7, 50257, 50304), (3, 13, 16), (2, 1, 4),
                                    (3, 8189, 8192), (4, 16381, 16384), (3, 32765, 32768),
                                    (3, 39997, 40000), (2, 65533, 65536)])
def test_xent(M, V, Vp):
    torch = torch_gpu()
    say(f"xent M={M} V={V} Vp={Vp}")
    z = (RNG.standard_normal((M, Vp)) * 2).astype(np.float32)
    y = RNG.integers(0, V, M).astype(np.int32)
    y[-1] = V - 1
    scale = 1.0 / (M * 3)
    zd, yd = dev(torch, z), dev(torch, y)
    loss = torch.empty(M, device="cuda")
    lse = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fwd(zd, yd, loss, lse, M, V, Vp)
    rl, rlse = ops.xent_fwd(z, y, V)
    assert np.allclose(host(loss), rl, rtol=1e-5, atol=1e-5 * max(1.0, np.abs(rl).max()))
    assert np.allclose(host(lse), rlse, rtol=1e-6, atol=1e-6)
    rdz = ops.xent_bwd(z, y, V, scale)
    dz = torch.empty_like(zd)
    bt.bt_softmax_xent_bwd(zd, lse, yd, dz, scale, M, V, Vp)
    # the natural scale of dlogits is `scale` (with V = 1 the gradient is exactly 0)
    assert_close_maxabs(host(dz), rdz, 1e-5, "dlogits (bwd)", scale=max(np.abs(rdz).max(), scale))
    assert np.all(host(dz)[:, V:] == 0)
    loss2 = torch.empty(M, device="cuda")
    lse2 = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fused(zd, yd, loss2, lse2, scale, M, V, Vp)  # in place
    assert np.allclose(host(loss2), rl, rtol=1e-5, atol=1e-5 * max(1.0, np.abs(rl).max()))
    assert_close_maxabs(host(zd), rdz, 1e-5, "dlogits (fused, in place)", scale=max(np.abs(rdz).max(), scale))
    assert np.all(host(zd)[:, V:] == 0)
    # rows of (softmax - onehot) sum to zero
    assert np.abs(host(zd)[:, :V].sum(axis=1)).max() <= 1e-6 * scale * 10


def test_xent_zero_logits_is_ln_V():
    torch = torch_gpu()
    M, V, Vp = 64, 50257, 50304
    say("xent zero logits")
    z = torch.zeros((M, Vp), device="cuda")
    y = dev(torch, RNG.integers(0, V, M).astype(np.int32))
    loss = torch.empty(M, device="cuda")
    lse = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fwd(z, y, loss, lse, M, V, Vp)
    assert np.allclose(host(loss), math.log(V), rtol=1e-6, atol=0)


def test_xent_full_size_sampled():
    torch = torch_gpu()
    M, V, Vp = 16384, 50257, 50304
    say("xent full size fused")
    g = torch.Generator(device="cuda").manual_seed(4)
    z = torch.randn((M, Vp), generator=g, device="cuda") * 3
    y = dev(torch, synth.zipf_tokens(M, V, 1.1, 40))
    rows = np.sort(RNG.choice(M, 32, replace=False))
    zr = host(z[torch.from_numpy(rows).cuda()])
    loss = torch.empty(M, device="cuda")
    lse = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fused(z, y, loss, lse, 1.0 / M, M, V, Vp)
    yr = host(y).astype(np.int64)[rows]
    rl, _ = ops.xent_fwd(zr, yr, V)
    assert np.allclose(host(loss)[rows], rl, rtol=1e-5, atol=0)
    assert_close_maxabs(host(z[torch.from_numpy(rows).cuda()]), ops.xent_bwd(zr, yr, V, 1.0 / M), 1e-5,
                        "dlogits rows")


@pytest.mark.parametrize("M,V,Vp", [(600, 50257, 50304), (530, 53001, 53248)])
def test_xent_fused_several_rows_per_block(M, V, Vp):
    """The fused pass at vocabularies of 13 float4 per thread runs one block
    per CU over several rows each, with the next row prefetched: every row
    of a launch in which each block takes 2-3 rows against the oracle."""
    torch = torch_gpu()
    say(f"xent fused several rows per block M={M} V={V} Vp={Vp}")
    z = (RNG.standard_normal((M, Vp)) * 3).astype(np.float32)
    y = RNG.integers(0, V, M).astype(np.int32)
    y[0], y[-1] = 0, V - 1
    scale = 1.0 / M
    zd, yd = dev(torch, z), dev(torch, y)
    loss = torch.empty(M, device="cuda")
    lse = torch.empty(M, device="cuda")
    bt.bt_softmax_xent_fused(zd, yd, loss, lse, scale, M, V, Vp)
    rl, rlse = ops.xent_fwd(z, y, V)
    assert np.allclose(host(loss), rl, rtol=1e-5, atol=0)
    assert np.allclose(host(lse), rlse, rtol=1e-6, atol=1e-6)
    dz = host(zd)
    assert_close_maxabs(dz, ops.xent_bwd(z, y, V, scale), 1e-5, "dlogits (fused, several rows per block)")
    assert np.all(dz[:, V:] == 0)


# ---------------------------------------------------------------------- AdamW
@pytest.mark.parametrize("t,clip", [(1, None), (2, 0.37), (7, None)])
def test_adamw(t, clip):
    torch = torch_gpu()
    n, nd = 4 * 2501, 4 * 1600
    say(f"adamw t={t} clip={clip}")
    p = RNG.standard_normal(n).astype(np.float32)
    g = (RNG.standard_normal(n) * 1e-2).astype(np.float32)
    g[:5] = 0
    m = (RNG.standard_normal(n) * 1e-3).astype(np.float32)
    v = (RNG.random(n) * 1e-5).astype(np.float32)
    hp = synth.HP_124M
    pd, gd, md, vd = dev(torch, p), dev(torch, g), dev(torch, m), dev(torch, v)
    coef = None if clip is None else dev(torch, np.array([clip], np.float32))
    bt.bt_adamw_step(pd, gd, md, vd, n, nd, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, t, coef)
    mask = (np.arange(n) < nd).astype(np.float64)
    rp, rm, rv = ops.adamw(p, g, m, v, t, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, mask,
                           1.0 if clip is None else float(np.float32(clip)))
    assert_close_maxabs(host(pd), rp, 1e-6, "p")
    assert_close_maxabs(host(md), rm, 1e-6, "m")
    assert_close_maxabs(host(vd), rv, 1e-6, "v")


def test_grad_norm_full_arena():
    torch = torch_gpu()
    n = synth.num_params(synth.GPT2_124M)
    say(f"grad norm n={n}")
    g = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn(n, generator=g, device="cuda") * 1e-3
    out = torch.zeros(2, device="cuda")
    bt.bt_grad_norm_clip(x, n, 1.0, out[0:1], out[1:2])
    norm = ops.grad_norm(host(x))
    o = host(out)
    assert abs(o[0] - norm) <= 1e-6 * norm
    assert abs(o[1] - ops.clip_coef(norm, 1.0)) <= 1e-6
    bt.bt_grad_norm_clip(x * 1e-4, n, 1.0, out[0:1], out[1:2])
    assert host(out)[1] == 1.0  # norm below the threshold: no clipping


# ----------------------------------------------------------------- Embeddings
# The gather's register cases: rows of 1, 2, 3, 4, 6, 8 and 16 float4 per lane.
@pytest.mark.parametrize("B,T,C,Vp,V", [(2, 32, 64, 256, 256), (16, 1024, 768, 50304, 50257), (3, 7, 12, 20, 17),
                                        (2, 33, 400, 300, 290), (3, 17, 1000, 100, 97), (2, 9, 1300, 64, 60),
                                        (2, 5, 1800, 64, 64), (2, 3, 4096, 16, 16)])
def test_embedding(B, T, C, Vp, V):
    torch = torch_gpu()
    say(f"embedding B={B} T={T} C={C}")
    wte = RNG.standard_normal((Vp, C)).astype(np.float32)
    wpe = RNG.standard_normal((T + 3, C)).astype(np.float32)
    tok = synth.zipf_tokens(B * T, V, 1.1, 9).reshape(B, T)
    tokd = dev(torch, tok)
    x0 = torch.empty((B * T, C), device="cuda")
    bt.bt_embedding_fwd(tokd, dev(torch, wte), dev(torch, wpe), x0, B, T, C, Vp)
    assert np.array_equal(host(x0), (ops.embedding_fwd(wte, wpe, tok)).reshape(B * T, C).astype(np.float32))
    dx0 = RNG.standard_normal((B, T, C)).astype(np.float32)
    dwte0 = RNG.standard_normal((Vp, C)).astype(np.float32)
    dwpe0 = RNG.standard_normal((T + 3, C)).astype(np.float32)
    rwte, rwpe = ops.embedding_bwd(dx0, tok, Vp, T + 3)
    for beta in (0.0, 1.0):
        dwte = dev(torch, dwte0)
        dwpe = dev(torch, dwpe0)
        bt.bt_embedding_bwd(tokd, dev(torch, dx0), dwte, dwpe, beta, B, T, C, Vp)
        assert_close_maxabs(host(dwte), rwte + dwte0, 1e-5, f"dwte beta={beta}")
        exp_wpe = dwpe0.astype(np.float64).copy()
        exp_wpe[:T] = rwpe[:T] + beta * dwpe0[:T]
        assert_close_maxabs(host(dwpe), exp_wpe, 1e-5, f"dwpe beta={beta}")
        d2 = dev(torch, dwte0)
        bt.bt_embedding_bwd(tokd, dev(torch, dx0), d2, dev(torch, dwpe0), beta, B, T, C, Vp)
        assert torch.equal(d2, dwte), "embedding backward not deterministic"


def _emb_tokens(kind, B, T, V, Vp):
    M = B * T
    if kind == "zipf":
        return synth.zipf_tokens(M, V, 1.1, 11).reshape(B, T)
    if kind == "const":        # one run across every piece of the sorted list
        return np.full((B, T), 3, np.int32)
    if kind == "blocks64":     # runs of exactly 64 entries: every run boundary on a piece boundary
        return ((np.arange(M) // 64) % V).astype(np.int32).reshape(B, T)[:, ::-1].copy()
    if kind == "two_heavy":    # two long runs meeting inside a piece, plus singletons
        t = np.where(np.arange(M) % 3 == 0, 1, 2).astype(np.int32)
        t[::97] = np.arange(t[::97].size) % V
        return t.reshape(B, T)
    if kind == "clamp":        # ids outside [0, Vp) are clamped to the table
        t = synth.zipf_tokens(M, V, 1.1, 12)
        t[::5] = -7
        t[1::7] = Vp + 3
        return t.reshape(B, T)
    raise ValueError(kind)


# Backward from a separately built token index (the composed step builds it
# on a second stream during the forward) against the oracle, and against the
# self-indexing backward bitwise; forward with clamped ids.
@pytest.mark.parametrize("B,T,C,Vp,V,kind", [
    (16, 1024, 768, 50304, 50257, "zipf"),
    (64, 1024, 64, 50304, 50257, "zipf"),
    (4, 128, 68, 300, 300, "const"),
    (2, 512, 12, 64, 64, "blocks64"),
    (3, 700, 36, 1000, 1000, "two_heavy"),
    (3, 7, 12, 20, 17, "zipf"),
    (2, 300, 16, 100, 90, "clamp"),
    (1, 1, 4, 5, 5, "zipf"),
    (2, 4096, 20, 70000, 70000, "zipf"),   # 17-bit ids: three digit passes
])
def test_embedding_indexed(B, T, C, Vp, V, kind):
    torch = torch_gpu()
    say(f"embedding indexed B={B} T={T} C={C} Vp={Vp} {kind}")
    rng = np.random.Generator(np.random.PCG64(B * 1000 + T))
    tok = _emb_tokens(kind, B, T, V, Vp)
    tok_eff = np.clip(tok, 0, Vp - 1)
    wte = rng.standard_normal((Vp, C)).astype(np.float32)
    wpe = rng.standard_normal((T, C)).astype(np.float32)
    tokd = dev(torch, tok)
    index = torch.empty(bt.lib().bt_embedding_index_bytes(B, T), dtype=torch.uint8, device="cuda")
    x0 = torch.empty((B * T, C), device="cuda")
    bt.bt_embedding_fwd(tokd, dev(torch, wte), dev(torch, wpe), x0, B, T, C, Vp)
    assert np.array_equal(host(x0), ops.embedding_fwd(wte, wpe, tok_eff).reshape(B * T, C).astype(np.float32))
    bt.bt_embedding_index(tokd, index, B, T, Vp)
    dx0 = rng.standard_normal((B, T, C)).astype(np.float32)
    dwte0 = rng.standard_normal((Vp, C)).astype(np.float32)
    dwpe0 = rng.standard_normal((T, C)).astype(np.float32)
    rwte, rwpe = ops.embedding_bwd(dx0, tok_eff, Vp, T)
    dxd = dev(torch, dx0)
    for beta in (0.0, 1.0):
        dwte, dwpe = dev(torch, dwte0), dev(torch, dwpe0)
        bt.bt_embedding_bwd_indexed(index, dxd, dwte, dwpe, beta, B, T, C, Vp)
        assert_close_maxabs(host(dwte), rwte + dwte0, 1e-5, f"dwte beta={beta}")
        assert_close_maxabs(host(dwpe), rwpe + beta * dwpe0, 1e-5, f"dwpe beta={beta}")
        # untouched rows of dwte stay bitwise equal
        untouched = np.setdiff1d(np.arange(Vp), np.unique(tok_eff))
        assert np.array_equal(host(dwte)[untouched], dwte0[untouched].astype(np.float64))
        # the same index again (the arrival counters reset themselves), and the
        # self-indexing backward: bitwise equal
        d2, p2 = dev(torch, dwte0), dev(torch, dwpe0)
        bt.bt_embedding_bwd_indexed(index, dxd, d2, p2, beta, B, T, C, Vp)
        assert torch.equal(d2, dwte) and torch.equal(p2, dwpe), "indexed backward not deterministic"
        d3, p3 = dev(torch, dwte0), dev(torch, dwpe0)
        bt.bt_embedding_bwd(tokd, dxd, d3, p3, beta, B, T, C, Vp)
        assert torch.equal(d3, dwte) and torch.equal(p3, dwpe), "indexed and self-indexing backward differ"


# ---------------------------------------------------------------- Column sums
@pytest.mark.parametrize("M,N", [(16384, 3072), (37, 20), (1, 4), (16384, 2304)])
def test_colsum(M, N):
    torch = torch_gpu()
    say(f"colsum M={M} N={N}")
    X = RNG.standard_normal((M, N)).astype(np.float32)
    o0 = RNG.standard_normal(N).astype(np.float32)
    for beta in (0.0, 1.0):
        out = dev(torch, o0)
        bt.bt_colsum(dev(torch, X), M, N, N, out, beta)
        assert_close_maxabs(host(out), X.astype(np.float64).sum(0) + beta * o0, 1e-5, f"colsum beta={beta}")
