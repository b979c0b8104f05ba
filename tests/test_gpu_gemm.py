"""GEMM parity: bt_gemm (FP32 MFMA) against the float64 oracle.

Small shapes span several 128 x 128 tiles with ragged tails, every layout
(NN, NT, TN, TT) and every epilogue; the GPT-2 124M shapes (M = B*T = 16384)
run in full and are checked on sampled rows / columns that the oracle
computes one by one.  Bar: |C - C_ref| <= 1e-5 * max|C_ref| (FP32 inputs,
FP32 accumulation; the error of a K-term FP32 dot product grows like
sqrt(K) * 6e-8 relative to the row scale)."""
import numpy as np
import pytest

from oracle import ops
from paper_2606_24780_amd import bt
from tests.gpu_util import assert_close_maxabs, dev, host, say, torch_gpu

pytestmark = pytest.mark.gpu
TOL = 1e-5
RNG = np.random.Generator(np.random.PCG64(2))


def _operands(M, N, K, ta, tb):
    A = RNG.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    B = RNG.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    return A, B


def _run(torch, ta, tb, M, N, K, A, B, **kw):
    Ad, Bd = dev(torch, A), dev(torch, B)
    C0 = kw.pop("C0", None)
    C = dev(torch, C0) if C0 is not None else torch.zeros((M, N), dtype=torch.float32, device="cuda")
    lda = M if ta else K
    ldb = K if tb else N
    bt.bt_gemm(int(ta), int(tb), M, N, K, Ad, lda, Bd, ldb, kw.pop("beta", 0.0), C, N, **kw)
    return C


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("M,N,K", [(260, 196, 132), (64, 64, 256), (4, 8, 4), (300, 388, 1000),
                                   (128, 128, 32), (132, 260, 36), (8, 12, 4096),
                                   (256, 384, 272), (384, 256, 1024)])
def test_gemm_layouts(ta, tb, M, N, K):
    torch = torch_gpu()
    say(f"gemm layout ta={ta} tb={tb} M={M} N={N} K={K}")
    A, B = _operands(M, N, K, ta, tb)
    C = _run(torch, ta, tb, M, N, K, A, B)
    assert_close_maxabs(host(C), ops.gemm(A, B, bool(ta), bool(tb)), TOL, f"gemm {ta}{tb} {M}x{N}x{K}")


# (260, 196, 132) has ragged tiles (operands staged through registers); the
# full-tile shape takes the direct global -> LDS copy path.
@pytest.mark.parametrize("M,N,K", [(260, 196, 132), (256, 256, 144)])
def test_gemm_epilogues(M, N, K):
    torch = torch_gpu()
    A, B = _operands(M, N, K, 0, 0)
    bias = RNG.standard_normal(N).astype(np.float32)
    res = RNG.standard_normal((M, N)).astype(np.float32)
    gin = (RNG.standard_normal((M, N)) * 2).astype(np.float32)
    C0 = RNG.standard_normal((M, N)).astype(np.float32)
    ref = ops.gemm(A, B)
    say("gemm epilogue BIAS + residual")
    C = _run(torch, 0, 0, M, N, K, A, B, bias=dev(torch, bias), epi=bt.EPI_BIAS, residual=dev(torch, res))
    assert_close_maxabs(host(C), ref + bias + res, TOL, "bias+residual")
    say("gemm epilogue BIAS_GELU + preact")
    pre = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    C = _run(torch, 0, 0, M, N, K, A, B, bias=dev(torch, bias), epi=bt.EPI_BIAS_GELU, preact_out=pre)
    assert_close_maxabs(host(pre), ref + bias, TOL, "preact")
    assert_close_maxabs(host(C), ops.gelu_fwd(ref + bias), TOL, "gelu(pre)")
    say("gemm epilogue DGELU")
    C = _run(torch, 0, 1, M, N, K, A, np.ascontiguousarray(B.T), epi=bt.EPI_DGELU, gelu_in=dev(torch, gin))
    assert_close_maxabs(host(C), ref * ops.gelu_grad(gin), TOL, "dgelu")
    say("gemm beta=1 accumulate (split-K path)")
    A2, B2 = _operands(64, 64, 2048, 1, 0)
    C02 = RNG.standard_normal((64, 64)).astype(np.float32)
    C = _run(torch, 1, 0, 64, 64, 2048, A2, B2, C0=C02, beta=1.0)
    assert_close_maxabs(host(C), ops.gemm(A2, B2, True) + C02, TOL, "beta=1 split")
    say("gemm K=0 with bias")
    C = _run(torch, 0, 0, 8, 8, 0, np.zeros((8, 0), np.float32), np.zeros((0, 8), np.float32),
             bias=dev(torch, bias[:8]), epi=bt.EPI_BIAS)
    assert np.array_equal(host(C), np.broadcast_to(bias[:8].astype(np.float64), (8, 8)))


# Every combination of epilogue and additive inputs in the tile epilogue
# (products that are not split): the plain GELU-backward, bias and residual /
# beta = 1 products stream their one input a block ahead of the stores; two
# inputs and the bias + GELU products take the general 4-row path.  Ragged
# (260, 196, 36) and full-tile (256, 256, 64) shapes, each in both B layouts.
@pytest.mark.parametrize("M,N,K", [(260, 196, 36), (256, 256, 64)])
@pytest.mark.parametrize("tb", [0, 1])
def test_gemm_tile_epilogue_combinations(M, N, K, tb):
    torch = torch_gpu()
    L = bt.lib()
    for epi in (bt.EPI_NONE, bt.EPI_BIAS, bt.EPI_BIAS_GELU, bt.EPI_DGELU):
        assert L.bt_gemm_ws_bytes(0, tb, M, N, K, epi) == 0, "shape must not be split"
    A, B = _operands(M, N, K, 0, tb)
    bias = RNG.standard_normal(N).astype(np.float32)
    res = RNG.standard_normal((M, N)).astype(np.float32)
    gin = (RNG.standard_normal((M, N)) * 2).astype(np.float32)
    C0 = RNG.standard_normal((M, N)).astype(np.float32)
    prod = ops.gemm(A, B, False, bool(tb))
    for epi in (bt.EPI_NONE, bt.EPI_BIAS, bt.EPI_BIAS_GELU, bt.EPI_DGELU):
        for with_res in (False, True):
            for beta in (0.0, 1.0):
                say(f"gemm tile epilogue {epi} residual={with_res} beta={beta} M={M} N={N} K={K} tb={tb}")
                kw = dict(beta=beta, epi=epi)
                if epi in (bt.EPI_BIAS, bt.EPI_BIAS_GELU):
                    kw["bias"] = dev(torch, bias)
                pre = None
                if epi == bt.EPI_BIAS_GELU:
                    pre = torch.zeros((M, N), dtype=torch.float32, device="cuda")
                    kw["preact_out"] = pre
                if epi == bt.EPI_DGELU:
                    kw["gelu_in"] = dev(torch, gin)
                if with_res:
                    kw["residual"] = dev(torch, res)
                C = _run(torch, 0, tb, M, N, K, A, B, C0=C0 if beta else None, **kw)
                v = prod.copy()
                if epi in (bt.EPI_BIAS, bt.EPI_BIAS_GELU):
                    v = v + bias
                if epi == bt.EPI_BIAS_GELU:
                    assert_close_maxabs(host(pre), v, TOL, "preact")
                    v = ops.gelu_fwd(v)
                if epi == bt.EPI_DGELU:
                    v = v * ops.gelu_grad(gin)
                if with_res:
                    v = v + res
                if beta:
                    v = v + C0
                assert_close_maxabs(host(C), v, TOL, f"epi={epi} residual={with_res} beta={beta}")


# Long K over few tiles splits the product; the epilogue (with residual and
# beta = 1) then runs in the reduction of the partials.  (260, 196, 4100)
# is ragged, (256, 256, 4096) takes the direct-copy tiles.
@pytest.mark.parametrize("M,N,K", [(260, 196, 4100), (256, 256, 4096)])
def test_gemm_epilogues_split(M, N, K):
    torch = torch_gpu()
    L = bt.lib()
    for epi in (bt.EPI_BIAS, bt.EPI_BIAS_GELU):
        assert L.bt_gemm_ws_bytes(0, 0, M, N, K, epi) > 0, "shape expected to split"
    assert L.bt_gemm_ws_bytes(0, 1, M, N, K, bt.EPI_DGELU) > 0, "shape expected to split"
    A, B = _operands(M, N, K, 0, 0)
    bias = RNG.standard_normal(N).astype(np.float32)
    res = RNG.standard_normal((M, N)).astype(np.float32)
    gin = (RNG.standard_normal((M, N)) * 2).astype(np.float32)
    C0 = RNG.standard_normal((M, N)).astype(np.float32)
    ref = ops.gemm(A, B)
    say(f"split gemm BIAS + residual + beta=1 M={M} N={N} K={K}")
    C = _run(torch, 0, 0, M, N, K, A, B, bias=dev(torch, bias), epi=bt.EPI_BIAS, residual=dev(torch, res),
             C0=C0, beta=1.0)
    assert_close_maxabs(host(C), ref + bias + res + C0, TOL, "split bias+residual+beta")
    say("split gemm BIAS_GELU + preact")
    pre = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    C = _run(torch, 0, 0, M, N, K, A, B, bias=dev(torch, bias), epi=bt.EPI_BIAS_GELU, preact_out=pre)
    assert_close_maxabs(host(pre), ref + bias, TOL, "split preact")
    assert_close_maxabs(host(C), ops.gelu_fwd(ref + bias), TOL, "split gelu(pre)")
    say("split gemm DGELU")
    C = _run(torch, 0, 1, M, N, K, A, np.ascontiguousarray(B.T), epi=bt.EPI_DGELU, gelu_in=dev(torch, gin))
    assert_close_maxabs(host(C), ref * ops.gelu_grad(gin), TOL, "split dgelu")


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_gemm_full_tiles_match_ragged_path(ta, tb):
    """A full-tile product (direct LDS copies) and the same data inside a
    ragged product (register staging) add the same terms in the same order,
    so the shared 256 x 256 block of C is bitwise equal.  Both shapes must be
    split along K the same way (asserted from their workspace sizes); the
    zero bias adds exactly 0."""
    torch = torch_gpu()
    say(f"gemm full vs ragged path ta={ta} tb={tb}")
    M, N, K = 256, 256, 512
    L = bt.lib()
    splits = [L.bt_gemm_ws_bytes(ta, tb, m, n, K, bt.EPI_BIAS) // (4 * (m * n + n)) for m, n in ((M, N), (M + 4, N + 4))]
    assert splits[0] == splits[1], splits
    A, B = _operands(M + 4, N + 4, K, ta, tb)
    zb = torch.zeros(N + 4, dtype=torch.float32, device="cuda")
    C_big = host(_run(torch, ta, tb, M + 4, N + 4, K, A, B, bias=zb, epi=bt.EPI_BIAS))
    A_s = np.ascontiguousarray(A[:, :M] if ta else A[:M])
    B_s = np.ascontiguousarray(B[:N] if tb else B[:, :N])
    C_small = host(_run(torch, ta, tb, M, N, K, A_s, B_s, bias=zb[:N], epi=bt.EPI_BIAS))
    assert np.array_equal(C_small, C_big[:M, :N])
    assert_close_maxabs(C_small, ops.gemm(A_s, B_s, bool(ta), bool(tb)), TOL, "full tiles")


@pytest.mark.parametrize("wide", ["A", "B"])
def test_gemm_wide_leading_dimension(wide):
    """An operand whose leading dimension reaches 2^22 floats (a 4.2M-float
    row stride) would overflow the 32-bit per-lane offsets of the direct LDS
    copies, so such a product takes the staged path: the result equals, bit
    for bit, the same product on compact operands (direct copies; the same
    terms in the same order) and matches the oracle."""
    torch = torch_gpu()
    say(f"gemm wide leading dimension of {wide}")
    M, N, K = 128, 128, 256
    wide_ld = (1 << 22) + 4
    A, B = _operands(M, N, K, 0, 1)  # A [M][K], B [N][K] (NT)
    Ad, Bd = dev(torch, A), dev(torch, B)
    C_ref = torch.empty((M, N), dtype=torch.float32, device="cuda")
    bt.bt_gemm(bt.OP_N, bt.OP_T, M, N, K, Ad, K, Bd, K, 0.0, C_ref, N)
    rows = M if wide == "A" else N
    big = torch.zeros((rows, wide_ld), dtype=torch.float32, device="cuda")
    big[:, :K] = Ad if wide == "A" else Bd
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    if wide == "A":
        bt.bt_gemm(bt.OP_N, bt.OP_T, M, N, K, big, wide_ld, Bd, K, 0.0, C, N)
    else:
        bt.bt_gemm(bt.OP_N, bt.OP_T, M, N, K, Ad, K, big, wide_ld, 0.0, C, N)
    torch.cuda.synchronize()
    del big
    assert torch.equal(C, C_ref)
    assert_close_maxabs(host(C), ops.gemm(A, B, False, True), TOL, "wide leading dimension")


def test_gemm_deterministic_split():
    torch = torch_gpu()
    say("gemm determinism (split-K)")
    A, B = _operands(768, 768, 16384, 1, 0)
    C1 = _run(torch, 1, 0, 768, 768, 16384, A, B)
    C2 = _run(torch, 1, 0, 768, 768, 16384, A, B)
    assert torch.equal(C1, C2)


# GPT-2 124M (K, N) pairs at M = 16384: QKV, attn-out, FC, FC-proj, LM head
FULL = [(768, 2304), (768, 768), (768, 3072), (3072, 768), (768, 50304)]


@pytest.mark.parametrize("K,N", FULL)
def test_gemm_gpt2_124m_shapes_sampled(K, N):
    torch = torch_gpu()
    M = 16384
    g = torch.Generator(device="cuda").manual_seed(2)
    say(f"gemm full-size K={K} N={N}")
    X = torch.randn((M, K), generator=g, device="cuda")
    W = torch.randn((K, N), generator=g, device="cuda") * 0.02
    dY = torch.randn((M, N), generator=g, device="cuda")
    rows = np.sort(RNG.choice(M, 48, replace=False))
    cols = np.sort(RNG.choice(N, 48, replace=False))
    Wh = host(W)
    # forward NN: Y = X W
    Y = torch.empty((M, N), device="cuda")
    bt.bt_gemm(0, 0, M, N, K, X, K, W, N, 0.0, Y, N)
    Xr = host(X[torch.from_numpy(rows).cuda()])
    assert_close_maxabs(host(Y)[rows], Xr @ Wh, TOL, f"NN {M}x{N}x{K}")
    # dX = dY W^T (NT, reduction over N)
    dX = torch.empty((M, K), device="cuda")
    bt.bt_gemm(0, 1, M, K, N, dY, N, W, N, 0.0, dX, K)
    dYr = host(dY[torch.from_numpy(rows).cuda()])
    assert_close_maxabs(host(dX)[rows], dYr @ Wh.T, TOL, f"NT {M}x{K}x{N}")
    del dX, Y
    # dW = X^T dY (TN, reduction over the 16384 tokens)
    dW = torch.empty((K, N), device="cuda")
    bt.bt_gemm(1, 0, K, N, M, X, K, dY, N, 0.0, dW, N)
    dYc = host(dY[:, torch.from_numpy(cols).cuda()])
    assert_close_maxabs(host(dW)[:, cols], host(X).T @ dYc, TOL, f"TN {K}x{N}x{M}")


@pytest.mark.parametrize("M,N,K", [(768, 768, 16384), (64, 192, 256), (260, 196, 132), (3072, 768, 4096)])
def test_gemm_weight_grad_with_bias_grad(M, N, K):
    """dW = X^T dY (TN) with the bias gradient sum_m dY[m, n] returned by the
    same product (split-K and single-pass shapes), overwrite and accumulate."""
    torch = torch_gpu()
    say(f"gemm TN + column sums M={M} N={N} K={K}")
    X = RNG.standard_normal((K, M)).astype(np.float32)
    dY = RNG.standard_normal((K, N)).astype(np.float32)
    C0 = RNG.standard_normal((M, N)).astype(np.float32)
    cs0 = RNG.standard_normal(N).astype(np.float32)
    for beta in (0.0, 1.0):
        C = dev(torch, C0)
        cs = dev(torch, cs0)
        bt.bt_gemm(1, 0, M, N, K, dev(torch, X), M, dev(torch, dY), N, beta, C, N, colsum_B=cs)
        assert_close_maxabs(host(C), ops.gemm(X, dY, True) + beta * C0, TOL, f"dW beta={beta}")
        assert_close_maxabs(host(cs), dY.astype(np.float64).sum(0) + beta * cs0, TOL, f"db beta={beta}")
