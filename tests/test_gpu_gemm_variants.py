"""Every GEMM kernel variant that bt_gemm can launch, against the oracle.

For each product, bt_gemm picks a block-tile depth (16 or 32) and a number
of K splits.  It also decides whether operand tiles are copied straight
into LDS (every tile full) or staged with bounds checks.  Beyond those, the
kernel is specialised by the operand layouts and the epilogue.
bt_gemm_plan reports the first three choices.  For each operand layout,
this test searches a grid of shapes for the cheapest one that reaches each
(depth, split, direct) combination the planner produces.  On that shape it
runs every epilogue: plain, bias, bias + GELU with the pre-activation,
GELU backward, the residual and beta = 1 additive inputs, and the
bias-gradient column sums where the layout allows them.  The results are
checked against the float64 oracle.  Small products are checked in full;
large ones on sampled rows and columns that the oracle computes one by
one."""
import itertools

import numpy as np
import pytest

from oracle import ops
from paper_2606_24780_amd import bt
from tests.gpu_util import assert_close_maxabs, host, say, torch_gpu

pytestmark = pytest.mark.gpu
TOL = 1e-5
MS = [4, 64, 128, 132, 256, 260, 384, 512, 1024, 1028, 2048, 2052, 3076, 4096]
KS = [4, 16, 32, 36, 64, 128, 256, 512, 1024, 2048, 4096, 8192, 8196, 16384, 32768, 32772, 50304]
FULL_CHECK_MACS = 1 << 27


def plans_for_layout(ta, tb):
    """{(depth, split, direct): cheapest (M, N, K) on the grid reaching it}."""
    best = {}
    for M, N, K in itertools.product(MS, MS, KS):
        d, sp, dr = bt.bt_gemm_plan(ta, tb, M, N, K, M if ta else K, K if tb else N)
        key = (d, sp > 1, dr)
        if key not in best or M * N * K < best[key][0] * best[key][1] * best[key][2]:
            best[key] = (M, N, K)
    return best


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_gemm_variants(ta, tb):
    torch = torch_gpu()
    for (depth, split, direct), shape in sorted(plans_for_layout(ta, tb).items()):
        _check_variant(torch, ta, tb, depth, split, direct, *shape)


def _check_variant(torch, ta, tb, depth, split, direct, M, N, K):
    say(f"gemm variant layout={ta}{tb} depth={depth} split={split} direct={direct} {M}x{N}x{K}")
    d, sp, dr = bt.bt_gemm_plan(ta, tb, M, N, K, M if ta else K, K if tb else N)
    assert (d, sp > 1, dr) == (depth, split, direct)
    g = torch.Generator(device="cuda").manual_seed(M * 7 + N * 3 + K + 11 * ta + 5 * tb)
    A = torch.randn((K, M) if ta else (M, K), generator=g, device="cuda")
    B = torch.randn((N, K) if tb else (K, N), generator=g, device="cuda")
    bias = torch.randn(N, generator=g, device="cuda")
    gin = torch.randn((M, N), generator=g, device="cuda")
    res = torch.randn((M, N), generator=g, device="cuda")
    C0 = torch.randn((M, N), generator=g, device="cuda")
    lda, ldb = (M if ta else K), (K if tb else N)

    full = M * N * K <= FULL_CHECK_MACS
    rng = np.random.Generator(np.random.PCG64(M + N + K))
    rows = np.arange(M) if full else np.sort(rng.choice(M, min(M, 16), replace=False))
    cols = np.arange(N) if full else np.sort(rng.choice(N, min(N, 16), replace=False))
    rt, ct = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    opA_rows = host(A[:, rt]).T if ta else host(A[rt])          # op(A)[rows, :]
    opB_cols = host(B[ct]).T if tb else host(B[:, ct])          # op(B)[:, cols]
    ref = ops.gemm(opA_rows, opB_cols)                           # float64 oracle product
    pick = lambda t: host(t[rt][:, ct])

    def run(epi=bt.EPI_NONE, beta=0.0, C_init=None, **kw):
        C = C_init.clone() if C_init is not None else torch.zeros((M, N), device="cuda")
        bt.bt_gemm(ta, tb, M, N, K, A, lda, B, ldb, beta, C, N, epi=epi, **kw)
        return C

    bh, gh, rh, ch = host(bias)[cols], pick(gin), pick(res), pick(C0)
    assert_close_maxabs(pick(run()), ref, TOL, "plain")
    assert_close_maxabs(pick(run(beta=1.0, C_init=C0, residual=res)), ref + rh + ch, TOL, "beta=1 + residual")
    assert_close_maxabs(pick(run(bt.EPI_BIAS, bias=bias)), ref + bh, TOL, "bias")
    assert_close_maxabs(pick(run(bt.EPI_BIAS, bias=bias, residual=res)), ref + bh + rh, TOL, "bias + residual")
    pre = torch.zeros((M, N), device="cuda")
    out = run(bt.EPI_BIAS_GELU, bias=bias, preact_out=pre)
    assert_close_maxabs(pick(pre), ref + bh, TOL, "bias + GELU pre-activation")
    assert_close_maxabs(pick(out), ops.gelu_fwd(ref + bh), TOL, "bias + GELU")
    assert_close_maxabs(pick(run(bt.EPI_DGELU, gelu_in=gin)), ref * ops.gelu_grad(gh), TOL, "GELU backward")
    if tb == 0:
        cs = torch.full((N,), 3.0, device="cuda")
        out = run(colsum_B=cs)
        assert_close_maxabs(pick(out), ref, TOL, "plain with column sums")
        want = opB_cols.sum(axis=0)
        assert_close_maxabs(host(cs)[cols], want, TOL, "column sums of op(B)")
