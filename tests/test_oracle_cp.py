"""Pins for the context-parallel (ring) attention oracle (CPU only).

What pins it, other than itself: a pure-Python loop over (query, key) pairs
for the block attention; closed forms at Q = 0 (every visible score is 0, so a
block's output is the mean of its visible values and its lse the log of their
count); the partition identity of the softmax (merging the results of two
disjoint key sets gives the result over their union); equality of the
emulated ring with the plain causal attention; central finite differences for
the ring backward; and exact counts of causal work per rank."""
import math

import numpy as np
import pytest

from oracle import context_parallel as cp
from oracle import ops

RNG = np.random.Generator(np.random.PCG64(2606))


def test_balanced_chunks_cover_sequence_and_equalise_causal_work():
    for T, W in [(16, 1), (32, 2), (64, 4), (96, 3), (256, 8)]:
        pos = [cp.rank_positions(T, W, r) for r in range(W)]
        assert np.array_equal(np.sort(np.concatenate(pos)), np.arange(T))
        # visible (query, key) pairs of a rank: each query at position p sees p + 1 keys
        work = [int(sum(p + 1 for p in ps)) for ps in pos]
        assert len(set(work)) == 1
        assert sum(work) == T * (T + 1) // 2
    assert cp.balanced_chunks(32, 4) == [(0, 7), (1, 6), (2, 5), (3, 4)]
    with pytest.raises(ValueError):
        cp.balanced_chunks(30, 4)


def test_shard_tokens_gathers_positions():
    tok = RNG.integers(0, 1000, size=(2, 64))
    for r in range(4):
        loc = cp.shard_tokens(tok, 4, r)
        c = 8
        assert np.array_equal(loc[:, :c], tok[:, r * c:(r + 1) * c])
        assert np.array_equal(loc[:, c:], tok[:, (7 - r) * c:(8 - r) * c])


def test_block_fwd_matches_pair_loop():
    B, H, Tq, Tk, hd = 1, 2, 5, 6, 3
    q, k, v = (RNG.standard_normal((B, H, n, hd)) for n in (Tq, Tk, Tk))
    q_pos = np.array([3, 9, 0, 14, 7])
    k_pos = np.array([2, 8, 9, 1, 20, 15])
    out, lse = cp.block_attention_fwd(q, k, v, q_pos, k_pos)
    for b in range(B):
        for h in range(H):
            for i in range(Tq):
                keys = [j for j in range(Tk) if k_pos[j] <= q_pos[i]]
                if not keys:
                    assert lse[b, h, i] == -math.inf
                    assert np.all(out[b, h, i] == 0)
                    continue
                sc = {j: sum(q[b, h, i, d] * k[b, h, j, d] for d in range(hd)) / math.sqrt(hd) for j in keys}
                z = sum(math.exp(s) for s in sc.values())
                assert abs(lse[b, h, i] - math.log(z)) <= 1e-13
                for d in range(hd):
                    o = sum(math.exp(sc[j]) / z * v[b, h, j, d] for j in keys)
                    assert abs(out[b, h, i, d] - o) <= 1e-13


def test_block_fwd_zero_queries_closed_form():
    B, H, Tq, Tk, hd = 2, 3, 7, 9, 4
    q = np.zeros((B, H, Tq, hd))
    k, v = RNG.standard_normal((B, H, Tk, hd)), RNG.standard_normal((B, H, Tk, hd))
    q_pos = RNG.integers(0, 12, size=Tq)
    k_pos = RNG.integers(0, 12, size=Tk)
    out, lse = cp.block_attention_fwd(q, k, v, q_pos, k_pos)
    for i in range(Tq):
        vis = k_pos <= q_pos[i]
        n = int(vis.sum())
        if n == 0:
            assert np.all(lse[:, :, i] == -np.inf)
            continue
        np.testing.assert_allclose(lse[:, :, i], math.log(n), rtol=0, atol=1e-14)
        np.testing.assert_allclose(out[:, :, i], v[:, :, vis].mean(axis=2), rtol=0, atol=1e-14)


def test_merge_of_disjoint_key_sets_is_attention_over_union():
    B, H, T, hd = 2, 2, 6, 5
    q = RNG.standard_normal((B, H, T, hd)) * 2
    k = RNG.standard_normal((B, H, 2 * T, hd))
    v = RNG.standard_normal((B, H, 2 * T, hd))
    q_pos = np.full(T, 100)
    k_pos = np.arange(2 * T)
    perm = RNG.permutation(2 * T)
    a, b = perm[:T - 2], perm[T - 2:]
    oa, la = cp.block_attention_fwd(q, k[:, :, a], v[:, :, a], q_pos, k_pos[a])
    ob, lb = cp.block_attention_fwd(q, k[:, :, b], v[:, :, b], q_pos, k_pos[b])
    ou, lu = cp.block_attention_fwd(q, k, v, q_pos, k_pos)
    for (o1, l1, o2, l2) in [(oa, la, ob, lb), (ob, lb, oa, la)]:
        om, lm = cp.lse_merge(o1, l1, o2, l2)
        np.testing.assert_allclose(lm, lu, rtol=1e-14, atol=1e-14)
        np.testing.assert_allclose(om, ou, rtol=0, atol=1e-13)


def test_merge_closed_form_and_empty_blocks():
    # Q = 0: a block is (mean of n values, log n); merging weights by counts
    m1, m2 = RNG.standard_normal((1, 4)), RNG.standard_normal((1, 4))
    n1, n2 = 3.0, 13.0
    om, lm = cp.lse_merge(m1, np.array([math.log(n1)]), m2, np.array([math.log(n2)]))
    np.testing.assert_allclose(lm, [math.log(n1 + n2)], rtol=0, atol=1e-15)
    np.testing.assert_allclose(om, (n1 * m1 + n2 * m2) / (n1 + n2), rtol=0, atol=1e-15)
    # an empty block leaves the state; an empty state takes the block
    o, l = RNG.standard_normal((3, 2)), np.array([0.5, -2.0, 7.0])
    e_o, e_l = np.zeros((3, 2)), np.full(3, -np.inf)
    ko, kl = cp.lse_merge(o, l, e_o, e_l)
    assert np.array_equal(ko, o) and np.array_equal(kl, l)
    to, tl = cp.lse_merge(e_o, e_l, o, l)
    assert np.array_equal(to, o) and np.array_equal(tl, l)
    zo, zl = cp.lse_merge(e_o, e_l, e_o, e_l)
    assert np.all(zl == -np.inf) and np.all(zo == 0)
    # extreme lse gap: no overflow, the larger side wins
    bo, bl = cp.lse_merge(o, np.full(3, -800.0), m1[:, :2].repeat(3, 0), np.full(3, 800.0))
    np.testing.assert_allclose(bo, m1[:, :2].repeat(3, 0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(bl, 800.0, rtol=0, atol=0)


@pytest.mark.parametrize("T,W", [(16, 1), (32, 2), (64, 4), (48, 3)])
def test_ring_fwd_equals_causal_attention(T, W):
    B, H, hd = 2, 2, 8
    qkv = RNG.standard_normal((B, T, 3, H, hd))
    out, lse = cp.ring_attention_fwd(qkv, H, W)
    r_out, r_lse = ops.attention_fwd(qkv, H)
    np.testing.assert_allclose(out, r_out, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, r_lse, rtol=0, atol=1e-13)


@pytest.mark.parametrize("T,W", [(32, 2), (64, 4)])
def test_ring_bwd_equals_causal_attention_bwd(T, W):
    B, H, hd = 1, 2, 8
    qkv = RNG.standard_normal((B, T, 3, H, hd))
    dout = RNG.standard_normal((B, T, H, hd))
    d = cp.ring_attention_bwd(dout, qkv, H, W)
    np.testing.assert_allclose(d, ops.attention_bwd(dout, qkv, H), rtol=0, atol=1e-12)


def test_ring_bwd_central_differences():
    B, T, H, hd, W = 1, 16, 1, 4, 2
    qkv = RNG.standard_normal((B, T, 3, H, hd))
    dout = RNG.standard_normal((B, T, H, hd))
    d = cp.ring_attention_bwd(dout, qkv, H, W)

    def loss(x):
        return float((cp.ring_attention_fwd(x, H, W)[0] * dout).sum())

    for idx in [(0, 0, 0, 0, 1), (0, 5, 1, 0, 2), (0, 15, 2, 0, 3), (0, 9, 0, 0, 0), (0, 2, 1, 0, 3), (0, 11, 2, 0, 1)]:
        h = 1e-6
        xp, xm = qkv.copy(), qkv.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (loss(xp) - loss(xm)) / (2 * h)
        assert abs(fd - d[idx]) <= 1e-7 * max(1.0, abs(fd)), (idx, fd, d[idx])
