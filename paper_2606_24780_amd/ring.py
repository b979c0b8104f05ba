"""The ring schedule of context-parallel attention (section "Context
Parallelism") over libbt's per-step calls.

At ring step i rank r holds the key/value shard of rank (r - i) mod W: its
own at step 0, then the one its left neighbour held at step i - 1.

* Forward: step 0 writes (out, lse) from the rank's own shard (the causal
  diagonal: every query sees at least itself); each later step folds its
  shard into the running state with the sigmoid-form update.
* Backward: D = rowsum(dO o O) of the final output once, then at every step
  the rank adds its dQ and the shard's dK/dV.  The shard's gradient travels
  with the shard, so at step i it already holds the contributions of the i
  ranks that held the shard before; it is written at step 0 and added to at
  every later step, on every rank.

Moving shards between GPUs is the caller's (`kv_of` / `dkv_of` return the
buffers a rank holds at a step).  On one GPU every rank's tensors are
resident and `emulate` runs all ranks step by step in ring order, which gives
the dK/dV sums the same order as the real ring.  Argument marshalling only:
every step runs in libbt's kernels.
"""
from __future__ import annotations

from . import bt


def shard_at(rank: int, step: int, W: int) -> int:
    """Owner of the shard that rank `rank` holds at ring step `step`."""
    return (rank - step) % W


def forward_step(rank, step, W, T, B, H, hd, qkv, kv, kv_stride, out, lse, stream=None):
    """One rank's forward at one ring step; kv / kv_stride: the shard it holds."""
    segs = bt.bt_cp_rank_segments(T, W, rank, shard_at(rank, step, W))
    bt.bt_attention_block_fwd(qkv, kv, kv_stride, out, lse, step > 0, B, H, hd, segs, stream)


def backward_step(rank, step, W, T, B, H, hd, dout, qkv, kv, kv_stride, lse, D, dqkv, dkv, ws=None,
                  stream=None):
    """One rank's backward at one ring step: dQ into dqkv (the rank's), dK/dV
    into dkv (the gradient travelling with the shard).  ws: scratch for the
    stored-dS method (see ws_bytes), or None to recompute."""
    segs = bt.bt_cp_rank_segments(T, W, rank, shard_at(rank, step, W))
    acc = 3 if step > 0 else 0
    bt.bt_attention_block_bwd(dout, qkv, kv, kv_stride, lse, D, dqkv, dkv, acc, B, H, hd, segs, ws=ws,
                              stream=stream)


def ws_bytes(W, T, B, H, hd):
    """Scratch for the stored-dS backward of any step of the ring (every
    step of the load-balanced split has the same shape)."""
    return bt.bt_attention_block_bwd_ws_bytes(B, H, hd, bt.bt_cp_rank_segments(T, W, 0, 0))


def emulate(W, T, B, H, hd, qkv, out, lse, kv_of, dout=None, D=None, dqkv=None, dkv_of=None, ws=None,
            stream=None):
    """All W ranks on one GPU.  qkv, out, lse, dout, D, dqkv: per-rank lists
    (local rows, [B, T/W, ...]); kv_of(s) -> (tensor or pointer, stride) of
    shard s; dkv_of(s) -> its gradient buffer; ws: scratch for the stored-dS
    backward (reused by every step), or None.  Runs the forward ring, and the
    backward ring when dout is given."""
    Tl = T // W
    for i in range(W):
        for r in range(W):
            kv, ks = kv_of(shard_at(r, i, W))
            forward_step(r, i, W, T, B, H, hd, qkv[r], kv, ks, out[r], lse[r], stream)
    if dout is None:
        return
    for r in range(W):
        bt.bt_attention_rowdot(dout[r], out[r], D[r], B, Tl, H, hd, stream)
    for i in range(W):
        for r in range(W):
            s = shard_at(r, i, W)
            kv, ks = kv_of(s)
            backward_step(r, i, W, T, B, H, hd, dout[r], qkv[r], kv, ks, lse[r], D[r], dqkv[r], dkv_of(s), ws,
                          stream)
