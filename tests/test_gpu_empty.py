"""Zero-size calls.  Every entry point that accepts an empty input writes
exactly what its definition gives for it: nothing, or the output scaled by
its beta.  The outputs start as sentinel-filled buffers, so a stray write
shows.  Where the empty input still has a value (the rows of dwpe, the
gradient norm of an empty arena), it is checked against the oracle on the
same empty input.  Attention needs B, T >= 1 and must reject B = 0 before
it launches anything."""
import numpy as np
import pytest

from oracle import ops
from paper_2606_24780_amd import bt
from tests.gpu_util import dev, host, say, torch_gpu

pytestmark = pytest.mark.gpu
SENT = 7.25
BT_ESHAPE = 2


def _sent(torch, *shape):
    return torch.full(shape, SENT, dtype=torch.float32, device="cuda")


def _untouched(t, what):
    assert np.all(host(t) == SENT), f"{what}: written by an empty call"


def test_empty_row_ops():
    torch = torch_gpu()
    C = 64
    say("empty: layernorm forward, M = 0")
    x, y = _sent(torch, 4, C), _sent(torch, 4, C)
    mean, rstd = _sent(torch, 4), _sent(torch, 4)
    gamma, beta = torch.ones(C, device="cuda"), torch.zeros(C, device="cuda")
    bt.bt_layernorm_fwd(x, gamma, beta, y, mean, rstd, 0, C)
    for t, w in ((y, "y"), (mean, "mean"), (rstd, "rstd")):
        _untouched(t, f"layernorm_fwd {w}")

    say("empty: layernorm backward, M = 0, param_beta 1 then 0")
    dy, dx = _sent(torch, 4, C), _sent(torch, 4, C)
    dg, db = _sent(torch, C), _sent(torch, C)
    bt.bt_layernorm_bwd(dy, x, gamma, mean, rstd, dx, dg, db, 0.0, 1.0, 0, C)
    for t, w in ((dx, "dx"), (dg, "dgamma"), (db, "dbeta")):
        _untouched(t, f"layernorm_bwd {w}")
    bt.bt_layernorm_bwd(dy, x, gamma, mean, rstd, dx, dg, db, 0.0, 0.0, 0, C)
    _untouched(dx, "layernorm_bwd dx")
    assert np.all(host(dg) == 0) and np.all(host(db) == 0), "param_beta = 0 over no rows must give zeros"

    say("empty: GELU forward / backward, n = 0")
    gy, gdx = _sent(torch, 16), _sent(torch, 16)
    bt.bt_gelu_fwd(x, gy, n=0)
    bt.bt_gelu_bwd(x, dy, gdx, n=0)
    _untouched(gy, "gelu_fwd y")
    _untouched(gdx, "gelu_bwd dx")

    say("empty: cross-entropy forward / backward / fused, M = 0")
    V, Vp = 13, 16
    logits = _sent(torch, 2, Vp)
    targets = torch.zeros(2, dtype=torch.int32, device="cuda")
    rows, lse, dl = _sent(torch, 2), _sent(torch, 2), _sent(torch, 2, Vp)
    bt.bt_softmax_xent_fwd(logits, targets, rows, lse, 0, V, Vp)
    bt.bt_softmax_xent_bwd(logits, lse, targets, dl, 1.0, 0, V, Vp)
    bt.bt_softmax_xent_fused(logits, targets, rows, lse, 1.0, 0, V, Vp)
    for t, w in ((rows, "loss_rows"), (lse, "lse"), (dl, "dlogits"), (logits, "logits (fused, in place)")):
        _untouched(t, f"xent {w}")

    say("empty: column sums, M = 0, beta 1 then 0")
    out = _sent(torch, C)
    bt.bt_colsum(x, 0, C, C, out, 1.0)
    _untouched(out, "colsum beta=1")
    bt.bt_colsum(x, 0, C, C, out, 0.0)
    assert np.all(host(out) == 0), "colsum beta = 0 over no rows must give zeros"

    say("empty: GEMM with M = 0 and with N = 0")
    Cm = _sent(torch, 4, 8)
    A, Bm = _sent(torch, 4, 4), _sent(torch, 4, 8)
    bt.bt_gemm(0, 0, 0, 8, 4, A, 4, Bm, 8, 0.0, Cm, 8)
    bt.bt_gemm(0, 0, 4, 0, 4, A, 4, Bm, 8, 0.0, Cm, 8)
    _untouched(Cm, "gemm C")


def test_empty_optimizer_inputs():
    torch = torch_gpu()
    say("empty: AdamW, n = 0")
    p, g, m, v = (_sent(torch, 8) for _ in range(4))
    bt.bt_adamw_step(p, g, m, v, 0, 0, 1e-3, 0.9, 0.95, 1e-8, 0.1, 1)
    for t, w in ((p, "p"), (m, "m"), (v, "v")):
        _untouched(t, f"adamw {w}")

    say("empty: gradient norm of an empty arena")
    out = _sent(torch, 2)
    bt.bt_grad_norm_clip(_sent(torch, 4), 0, 1.0, out[0:1], out[1:2])
    o = host(out)
    norm = ops.grad_norm(np.zeros(0))
    assert o[0] == norm == 0.0
    assert o[1] == ops.clip_coef(norm, 1.0) == 1.0


@pytest.mark.parametrize("B,T", [(0, 5), (3, 0)])
def test_empty_embedding(B, T):
    torch = torch_gpu()
    C, Vp, maxT = 8, 20, 8
    say(f"empty: embedding B={B} T={T}")
    tokens = torch.zeros(max(B * T, 1), dtype=torch.int32, device="cuda")
    wte, wpe = _sent(torch, Vp, C), _sent(torch, maxT, C)
    x0 = _sent(torch, 4, C)
    bt.bt_embedding_fwd(tokens, wte, wpe, x0, B, T, C, Vp)
    _untouched(x0, "embedding_fwd x0")

    # the oracle's sums over no positions: dwpe rows t < T get an empty batch sum
    _, ref_dwpe = ops.embedding_bwd(np.zeros((B, T, C)), np.zeros((B, T), np.int64), Vp, maxT)
    index = torch.empty(max(bt.lib().bt_embedding_index_bytes(B, T), 16), dtype=torch.uint8, device="cuda")
    bt.bt_embedding_index(tokens, index, B, T, Vp)
    for name, call in (("bwd", lambda dwte, dwpe, beta: bt.bt_embedding_bwd(
                            tokens, x0, dwte, dwpe, beta, B, T, C, Vp)),
                       ("bwd_indexed", lambda dwte, dwpe, beta: bt.bt_embedding_bwd_indexed(
                            index, x0, dwte, dwpe, beta, B, T, C, Vp))):
        for beta in (1.0, 0.0):
            dwte, dwpe = _sent(torch, Vp, C), _sent(torch, maxT, C)
            call(dwte, dwpe, beta)
            _untouched(dwte, f"embedding {name} dwte (beta {beta})")
            got = host(dwpe)
            assert np.all(got[T:] == SENT), f"embedding {name}: rows t >= T written"
            want = beta * SENT + ref_dwpe[:T]
            assert np.array_equal(got[:T], want), f"embedding {name}: dwpe rows t < T at beta {beta}"


def test_attention_rejects_empty_batch():
    torch = torch_gpu()
    say("empty: attention with B = 0 is a shape error")
    H, hd, T = 2, 16, 8
    qkv = _sent(torch, T, 3 * H * hd)
    out, lse = _sent(torch, T, H * hd), _sent(torch, H, T)
    with pytest.raises(bt.BTError) as e:
        bt.bt_attention_fwd(qkv, out, lse, 0, T, H, hd)
    assert e.value.status == BT_ESHAPE
    _untouched(out, "attention out")
    _untouched(lse, "attention lse")
