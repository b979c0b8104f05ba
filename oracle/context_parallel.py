"""Context-parallel (ring) attention in float64 (oracle; test infrastructure only).

Section "Context Parallelism": the sequence is spread over W ranks as a ring
of local chunks.  Key/value shards travel around the ring; at every ring step
a rank attends its local queries to the shard it holds, which gives a partial
output (block_out) and its log-sum-exp (block_lse), and folds them into its
running (out, lse) with a sigmoid-scaled update.  Causal masking follows the
global token positions.  Token chunks are rearranged once, where the data is
loaded, so that every rank carries the same causal work.  The backward pass
recomputes the scores shard by shard (one rotator) and sends the key/value
gradients around the ring with their shard (a second rotator).

Readings where the section is silent (each one is listed in the design notes):
* load balancing: the sequence is cut into 2W equal chunks and rank r holds
  chunks r and 2W-1-r, in that order;
* ring order: at step i, rank r holds the shard of rank (r - i) mod W, so step
  0 is the rank's own shard;
* a query that sees no key of a shard gets block_lse = -inf and a zero
  block_out, and the update leaves its running state unchanged.

Every function works on [B, H, rows, hd] float64 arrays (the layout of
``ops.split_qkv``) with int position vectors; ``ring_attention_fwd`` and
``ring_attention_bwd`` take the full-sequence qkv [B, T, 3, H, hd] and emulate
all W ranks one after another.
"""
from __future__ import annotations

import math

import numpy as np

from . import ops

F64 = np.float64


def balanced_chunks(T: int, W: int):
    """Chunk ids held by each rank (load balancing, reading above): rank r holds
    chunks r and 2W-1-r of length T / (2W)."""
    if W < 1 or T % (2 * W):
        raise ValueError(f"T={T} must split into 2W={2 * W} equal chunks")
    return [(r, 2 * W - 1 - r) for r in range(W)]


def rank_positions(T: int, W: int, r: int):
    """Global token positions of rank r's local rows, in local row order."""
    c = T // (2 * W)
    a, b = balanced_chunks(T, W)[r]
    return np.concatenate([np.arange(a * c, (a + 1) * c), np.arange(b * c, (b + 1) * c)])


def shard_tokens(tokens, W: int, r: int):
    """The rearrangement at the data-loading boundary: rank r's tokens [B, T/W]."""
    tokens = np.asarray(tokens)
    return tokens[:, rank_positions(tokens.shape[1], W, r)]


def block_attention_fwd(q, k, v, q_pos, k_pos):
    """Attention of queries q [B, H, Tq, hd] to one shard k, v [B, H, Tk, hd].

    Key j is visible to query i iff k_pos[j] <= q_pos[i]; the scale is
    1/sqrt(hd).  Returns (block_out [B, H, Tq, hd], block_lse [B, H, Tq]) with
    block_lse the natural-log sum of exponentials of the visible scores; a
    query with no visible key gets a zero row and -inf."""
    q, k, v = (np.asarray(a, F64) for a in (q, k, v))
    hd = q.shape[-1]
    vis = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]  # [Tq, Tk]
    seen = vis.any(axis=1)                                            # [Tq]
    s = np.where(vis, (q @ np.swapaxes(k, -1, -2)) / math.sqrt(hd), -np.inf)
    m = np.where(seen, s.max(axis=-1, initial=-np.inf), 0.0)
    e = np.where(vis, np.exp(s - m[..., None]), 0.0)
    l = e.sum(axis=-1)
    lse = np.where(seen, m + np.log(np.where(seen, l, 1.0)), -np.inf)
    out = (e / np.where(seen, l, 1.0)[..., None]) @ v
    return out, lse


def _sigmoid(x):
    """1 / (1 + e^-x), evaluated without overflow."""
    x = np.asarray(x, F64)
    z = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + z), z / (1.0 + z))


def _log_sigmoid(x):
    """log(1 / (1 + e^-x)) = min(x, 0) - log(1 + e^-|x|)."""
    x = np.asarray(x, F64)
    return np.minimum(x, 0.0) - np.log1p(np.exp(-np.abs(x)))


def lse_merge(out, lse, block_out, block_lse):
    """The sigmoid-scaled update of the running state by one partial result:

        out <- out - sigmoid(block_lse - lse) * (out - block_out)
        lse <- lse - log sigmoid(lse - block_lse)

    (out [..., rows, hd], lse [..., rows]).  Where block_lse is -inf the row
    keeps its state; where lse is -inf it takes the block's.  Returns new
    arrays."""
    out, lse = np.asarray(out, F64), np.asarray(lse, F64)
    block_out, block_lse = np.asarray(block_out, F64), np.asarray(block_lse, F64)
    both = np.isfinite(lse) & np.isfinite(block_lse)
    a = np.where(both, lse, 0.0)
    b = np.where(both, block_lse, 0.0)
    sig = _sigmoid(b - a)[..., None]
    new_out = np.where(both[..., None], out - sig * (out - block_out), 0.0)
    new_lse = np.where(both, a - _log_sigmoid(a - b), -np.inf)
    take_block = ~np.isfinite(lse) & np.isfinite(block_lse)
    keep = ~np.isfinite(block_lse)
    new_out = np.where(take_block[..., None], block_out, new_out)
    new_lse = np.where(take_block, block_lse, new_lse)
    new_out = np.where(keep[..., None], out, new_out)
    new_lse = np.where(keep, lse, new_lse)
    return new_out, new_lse


def block_attention_bwd(dout, q, k, v, q_pos, k_pos, lse, D):
    """One shard's part of the attention gradient, given the final (merged) lse
    [B, H, Tq] and D = rowsum(dO o O) of the final output:

        P = exp(S - lse) on visible entries (0 elsewhere),  dV = P^T dO,
        dP = dO V^T,  dS = P o (dP - D),  dQ = dS K / sqrt(hd),
        dK = dS^T Q / sqrt(hd).

    Returns (dq [B, H, Tq, hd], dk, dv [B, H, Tk, hd]); summed over all
    shards they are the gradient of the full attention."""
    dout, q, k, v = (np.asarray(a, F64) for a in (dout, q, k, v))
    hd = q.shape[-1]
    vis = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    s = (q @ np.swapaxes(k, -1, -2)) / math.sqrt(hd)
    p = np.where(vis, np.exp(np.where(vis, s, 0.0) - np.asarray(lse, F64)[..., None]), 0.0)
    dv = np.swapaxes(p, -1, -2) @ dout
    dp = dout @ np.swapaxes(v, -1, -2)
    ds = p * (dp - np.asarray(D, F64)[..., None])
    dq = ds @ k / math.sqrt(hd)
    dk = np.swapaxes(ds, -1, -2) @ q / math.sqrt(hd)
    return dq, dk, dv


def ring_attention_fwd(qkv, H: int, W: int):
    """All W ranks of the forward ring, one after another.  Returns
    (out [B, T, H, hd], lse [B, H, T]) in global token order."""
    q, k, v = ops.split_qkv(qkv, H)
    T = q.shape[2]
    pos = [rank_positions(T, W, r) for r in range(W)]
    out = np.zeros(q.shape, F64)
    lse = np.full(q.shape[:3], -np.inf)
    for r in range(W):
        o_r = l_r = None
        for i in range(W):
            s = (r - i) % W
            bo, bl = block_attention_fwd(q[:, :, pos[r]], k[:, :, pos[s]], v[:, :, pos[s]], pos[r], pos[s])
            o_r, l_r = (bo, bl) if i == 0 else lse_merge(o_r, l_r, bo, bl)
        out[:, :, pos[r]] = o_r
        lse[:, :, pos[r]] = l_r
    return out.transpose(0, 2, 1, 3), lse


def ring_attention_bwd(dout, qkv, H: int, W: int):
    """All W ranks of the backward ring: each rank recomputes its scores
    against every shard with the final lse and D, keeps its dQ, and adds the
    shard's dK/dV to the gradient that travels with the shard.  Returns dqkv
    [B, T, 3, H, hd] in global token order."""
    q, k, v = ops.split_qkv(qkv, H)
    B, _, T, hd = q.shape
    out, lse = ring_attention_fwd(qkv, H, W)
    do = np.asarray(dout, F64).transpose(0, 2, 1, 3)
    D = (do * out.transpose(0, 2, 1, 3)).sum(axis=-1)
    pos = [rank_positions(T, W, r) for r in range(W)]
    dq = np.zeros(q.shape, F64)
    dk = np.zeros(q.shape, F64)
    dv = np.zeros(q.shape, F64)
    for r in range(W):
        pr = pos[r]
        for i in range(W):
            s = (r - i) % W
            ps = pos[s]
            bq, bk, bv = block_attention_bwd(do[:, :, pr], q[:, :, pr], k[:, :, ps], v[:, :, ps], pr, ps,
                                             lse[:, :, pr], D[:, :, pr])
            dq[:, :, pr] += bq
            dk[:, :, ps] += bk
            dv[:, :, ps] += bv
    dqkv = np.empty((B, T, 3, H, hd), F64)
    dqkv[:, :, 0] = dq.transpose(0, 2, 1, 3)
    dqkv[:, :, 1] = dk.transpose(0, 2, 1, 3)
    dqkv[:, :, 2] = dv.transpose(0, 2, 1, 3)
    return dqkv
