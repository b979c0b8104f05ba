"""The no-allocation GEMM entry point (bt_gemm_noalloc) against bt_gemm with a
caller workspace: bitwise equal on split-K products (the weight-gradient
shapes of GPT-2 124M, whose partials go to the library's static scratch),
on two calls in a row with the second smaller, and with epilogues; shapes
whose scratch need exceeds the static array are rejected before launching."""
import ctypes

import numpy as np
import pytest

from paper_2606_24780_amd import bt
from tests.gpu_util import dev, say, torch_gpu

pytestmark = pytest.mark.gpu


def _pair(torch, opA, opB, M, N, K, epi=bt.EPI_NONE, beta=0.0, seed=0, colsum=False):
    g = torch.Generator(device="cuda").manual_seed(seed)
    A = torch.randn((M, K) if opA == bt.OP_N else (K, M), generator=g, device="cuda")
    B = torch.randn((K, N) if opB == bt.OP_N else (N, K), generator=g, device="cuda") * 0.02
    bias = torch.randn(N, generator=g, device="cuda") if epi in (bt.EPI_BIAS, bt.EPI_BIAS_GELU) else None
    gin = torch.randn((M, N), generator=g, device="cuda") if epi == bt.EPI_DGELU else None
    C0 = torch.randn((M, N), generator=g, device="cuda")
    lda, ldb = A.shape[1], B.shape[1]
    outs = []
    for noalloc in (False, True):
        C = C0.clone()
        cs = torch.randn(N, generator=torch.Generator(device="cuda").manual_seed(seed + 1), device="cuda") if colsum else None
        pre = torch.empty((M, N), device="cuda") if epi == bt.EPI_BIAS_GELU else None
        if noalloc:
            bt.bt_gemm_noalloc(opA, opB, M, N, K, A, lda, B, ldb, beta, C, N, bias=bias, epi=epi, preact_out=pre,
                               gelu_in=gin, colsum_B=cs)
        else:
            bt.bt_gemm(opA, opB, M, N, K, A, lda, B, ldb, beta, C, N, bias=bias, epi=epi, preact_out=pre,
                       gelu_in=gin, colsum_B=cs)
        torch.cuda.synchronize()
        outs.append((C, cs, pre))
    return outs


def test_noalloc_matches_workspace_path():
    torch = torch_gpu()
    L = bt.lib()
    cap = L.bt_gemm_noalloc_max_ws_bytes()
    # weight gradient of the MLP up-projection (split along K = 16384), then a
    # smaller one: the second call reuses the scratch the first one filled
    for (M, N, K, beta, colsum) in [(768, 3072, 16384, 0.0, True), (768, 768, 4096, 1.0, False)]:
        need = L.bt_gemm_ws_bytes(bt.OP_T, bt.OP_N, M, N, K, bt.EPI_NONE)
        say(f"gemm noalloc TN M={M} N={N} K={K} scratch {need} of {cap}")
        assert 0 < need <= cap
        (c_ws, s_ws, _), (c_na, s_na, _) = _pair(torch, bt.OP_T, bt.OP_N, M, N, K, beta=beta, colsum=colsum,
                                                  seed=M + K)
        assert torch.equal(c_ws, c_na), "noalloc product differs from the workspace path"
        if colsum:
            assert torch.equal(s_ws, s_na)
    # split products with epilogues, and a product that needs no scratch
    for (opA, opB, M, N, K, epi) in [(bt.OP_N, bt.OP_N, 256, 128, 8192, bt.EPI_BIAS_GELU),
                                     (bt.OP_N, bt.OP_T, 256, 256, 8192, bt.EPI_DGELU),
                                     (bt.OP_N, bt.OP_N, 1024, 768, 768, bt.EPI_BIAS)]:
        say(f"gemm noalloc M={M} N={N} K={K} epi={epi} scratch {L.bt_gemm_ws_bytes(opA, opB, M, N, K, epi)}")
        (c_ws, _, p_ws), (c_na, _, p_na) = _pair(torch, opA, opB, M, N, K, epi=epi, seed=K)
        assert torch.equal(c_ws, c_na)
        if p_ws is not None:
            assert torch.equal(p_ws, p_na)


def test_noalloc_rejects_products_beyond_the_scratch():
    torch = torch_gpu()
    L = bt.lib()
    M, N, K = 50304, 768, 16384  # tied LM head weight gradient at B = 16
    assert L.bt_gemm_ws_bytes(bt.OP_T, bt.OP_N, M, N, K, bt.EPI_NONE) > L.bt_gemm_noalloc_max_ws_bytes()
    C = torch.full((4, 4), 7.0, device="cuda")
    st = L.bt_gemm_noalloc(bt.OP_T, bt.OP_N, M, N, K, 0x10000, M, 0x10000, N, 0.0, C.data_ptr(), N, None, 0,
                           None, None, None, None, None)
    assert st == 4 and b"static scratch" in L.bt_last_error()
    torch.cuda.synchronize()
    assert (C == 7.0).all()
