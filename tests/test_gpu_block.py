"""One transformer block at the GPT-2 124M shape, forward and backward
composed from the C-ABI calls in the order the model uses them.

Shape B = 16, T = 1024, C = 768, H = 12.  Every parameter is random:
weights and biases N(0, 0.02), LN gains 1 + N(0, 0.02), LN biases N(0, 0.02),
so every bias epilogue, LayerNorm gain/shift and bias gradient is exercised
(the model's own initialisation has zero biases, unit gains).  Block input
x ~ N(0, 1) and upstream gradient dy ~ N(0, 1e-3).

The 16 sequences are copies of one: the float64 oracle runs that one
sequence, every copy's activations and input gradient must match it, and each
parameter gradient is exactly 16 times the oracle's.  Bars: block output
<= 1e-5 of max-abs; dx and each parameter gradient <= 1e-4 of max-abs."""
import numpy as np
import pytest

from oracle import gpt2 as og
from paper_2606_24780_amd import bt, synth
from tests.gpu_util import assert_close_maxabs, dev, host, say, torch_gpu

pytestmark = pytest.mark.gpu


def test_block_gpt2_124m_replicated():
    torch = torch_gpu()
    B, T, C, H = 16, 1024, 768, 12
    hd, F, M = C // H, 4 * C, B * T
    say("block B=16 T=1024 C=768 H=12, random LN/bias parameters")
    p = synth.block_params(C, H, 3)
    rng = np.random.Generator(np.random.PCG64(3003))
    x1s = rng.standard_normal((1, T, C)).astype(np.float32)
    dy1 = (rng.standard_normal((1, T, C)) * 1e-3).astype(np.float32)
    d = {k: dev(torch, v) for k, v in p.items()}

    def f(*shape):
        return torch.empty(shape, dtype=torch.float32, device="cuda")

    X = dev(torch, np.ascontiguousarray(np.broadcast_to(x1s, (B, T, C)).reshape(M, C)))
    DY = dev(torch, np.ascontiguousarray(np.broadcast_to(dy1, (B, T, C)).reshape(M, C)))
    N, T_ = bt.OP_N, bt.OP_T

    # ---- forward
    ln1, mu1, rs1 = f(M, C), f(M), f(M)
    bt.bt_layernorm_fwd(X, d["ln1g"], d["ln1b"], ln1, mu1, rs1, M, C)
    qkv = f(M, 3 * C)
    bt.bt_gemm(N, N, M, 3 * C, C, ln1, C, d["Wqkv"], 3 * C, 0.0, qkv, 3 * C, bias=d["bqkv"], epi=bt.EPI_BIAS)
    att, lse = f(M, C), f(B, H, T)
    bt.bt_attention_fwd(qkv, att, lse, B, T, H, hd)
    x1 = f(M, C)
    bt.bt_gemm(N, N, M, C, C, att, C, d["Wo"], C, 0.0, x1, C, bias=d["bo"], epi=bt.EPI_BIAS, residual=X)
    ln2, mu2, rs2 = f(M, C), f(M), f(M)
    bt.bt_layernorm_fwd(x1, d["ln2g"], d["ln2b"], ln2, mu2, rs2, M, C)
    h, g = f(M, F), f(M, F)
    bt.bt_gemm(N, N, M, F, C, ln2, C, d["Wfc"], F, 0.0, g, F, bias=d["bfc"], epi=bt.EPI_BIAS_GELU, preact_out=h)
    y = f(M, C)
    bt.bt_gemm(N, N, M, C, F, g, F, d["Wfp"], C, 0.0, y, C, bias=d["bfp"], epi=bt.EPI_BIAS, residual=x1)

    # ---- backward
    gr = {}
    gr["Wfp"], gr["bfp"] = f(F, C), f(C)
    bt.bt_gemm(T_, N, F, C, M, g, F, DY, C, 0.0, gr["Wfp"], C, colsum_B=gr["bfp"])
    dh = f(M, F)   # dg = dy Wfp^T, times gelu'(h) in the epilogue
    bt.bt_gemm(N, T_, M, F, C, DY, C, d["Wfp"], C, 0.0, dh, F, epi=bt.EPI_DGELU, gelu_in=h)
    gr["Wfc"], gr["bfc"] = f(C, F), f(F)
    bt.bt_gemm(T_, N, C, F, M, ln2, C, dh, F, 0.0, gr["Wfc"], F, colsum_B=gr["bfc"])
    dln2 = f(M, C)
    bt.bt_gemm(N, T_, M, C, F, dh, F, d["Wfc"], F, 0.0, dln2, C)
    dx1 = DY.clone()
    gr["ln2g"], gr["ln2b"] = f(C), f(C)
    bt.bt_layernorm_bwd(dln2, x1, d["ln2g"], mu2, rs2, dx1, gr["ln2g"], gr["ln2b"], 1.0, 0.0, M, C)
    gr["Wo"], gr["bo"] = f(C, C), f(C)
    bt.bt_gemm(T_, N, C, C, M, att, C, dx1, C, 0.0, gr["Wo"], C, colsum_B=gr["bo"])
    datt = f(M, C)
    bt.bt_gemm(N, T_, M, C, C, dx1, C, d["Wo"], C, 0.0, datt, C)
    dqkv = f(M, 3 * C)
    bt.bt_attention_bwd(datt, qkv, att, lse, dqkv, B, T, H, hd)
    gr["Wqkv"], gr["bqkv"] = f(C, 3 * C), f(3 * C)
    bt.bt_gemm(T_, N, C, 3 * C, M, ln1, C, dqkv, 3 * C, 0.0, gr["Wqkv"], 3 * C, colsum_B=gr["bqkv"])
    dln1 = f(M, C)
    bt.bt_gemm(N, T_, M, C, 3 * C, dqkv, 3 * C, d["Wqkv"], 3 * C, 0.0, dln1, C)
    dx = dx1.clone()
    gr["ln1g"], gr["ln1b"] = f(C), f(C)
    bt.bt_layernorm_bwd(dln1, X, d["ln1g"], mu1, rs1, dx, gr["ln1g"], gr["ln1b"], 1.0, 0.0, M, C)
    torch.cuda.synchronize()

    # ---- oracle on one sequence
    y_o, cache = og.block_fwd(x1s, p, H)
    dx_o, gr_o = og.block_bwd(dy1, p, cache)
    yh, dxh = host(y).reshape(B, T, C), host(dx).reshape(B, T, C)
    for b in (0, B - 1):
        assert_close_maxabs(yh[b], y_o[0], 1e-5, f"block output, copy {b}")
        assert_close_maxabs(dxh[b], dx_o[0], 1e-4, f"block dx, copy {b}")
    for k, v in gr.items():
        assert_close_maxabs(host(v), B * gr_o[k], 1e-4, f"d{k}")
