"""The ring schedule (host logic, CPU only): which shard each rank holds at
each step, and the merge / accumulate flags of every call, checked with the
library calls replaced by recorders."""
from paper_2606_24780_amd import bt, ring


def test_shard_at_is_a_ring():
    for W in (1, 2, 3, 8):
        for r in range(W):
            held = [ring.shard_at(r, i, W) for i in range(W)]
            assert held[0] == r and sorted(held) == list(range(W))
            # what rank r holds at step i, its left neighbour held at step i - 1
            for i in range(1, W):
                assert held[i] == ring.shard_at((r - 1) % W, i - 1, W)


def test_emulate_issues_the_ring_in_order(monkeypatch):
    calls = []
    monkeypatch.setattr(bt, "bt_cp_rank_segments", lambda T, W, r, s: ("segs", r, s))
    monkeypatch.setattr(bt, "bt_attention_block_fwd",
                        lambda qkv, kv, ks, out, lse, merge, B, H, hd, segs, stream:
                        calls.append(("fwd", segs[1], segs[2], bool(merge), qkv, kv, out)))
    monkeypatch.setattr(bt, "bt_attention_rowdot",
                        lambda dout, out, D, B, T, H, hd, stream: calls.append(("D", dout, out, D, T)))
    monkeypatch.setattr(bt, "bt_attention_block_bwd",
                        lambda dout, qkv, kv, ks, lse, D, dqkv, dkv, acc, B, H, hd, segs, ws=None, stream=None:
                        calls.append(("bwd", segs[1], segs[2], acc, dqkv, dkv, ws)))
    W, T = 4, 4096
    names = lambda p: [f"{p}{r}" for r in range(W)]
    ring.emulate(W, T, 2, 12, 64, names("qkv"), names("out"), names("lse"), lambda s: (f"kv{s}", 2304),
                 dout=names("do"), D=names("D"), dqkv=names("dqkv"), dkv_of=lambda s: f"dkv{s}", ws="scratch")
    fwd = [c for c in calls if c[0] == "fwd"]
    bwd = [c for c in calls if c[0] == "bwd"]
    assert len(fwd) == W * W and len(bwd) == W * W
    for k, c in enumerate(fwd):
        i, r = divmod(k, W)
        s = (r - i) % W
        assert c[1:] == (r, s, i > 0, f"qkv{r}", f"kv{s}", f"out{r}")
    dcalls = [c for c in calls if c[0] == "D"]
    assert dcalls == [("D", f"do{r}", f"out{r}", f"D{r}", T // W) for r in range(W)]
    assert calls.index(dcalls[-1]) < calls.index(bwd[0])  # D before any backward step
    for k, c in enumerate(bwd):
        i, r = divmod(k, W)
        s = (r - i) % W
        assert c[1:] == (r, s, 3 if i else 0, f"dqkv{r}", f"dkv{s}", "scratch")
    # every shard gradient is written once (its owner, step 0) before it is added to
    first = {}
    for c in bwd:
        first.setdefault(c[5], c)
    assert all(c[3] == 0 and c[1] == c[2] for c in first.values())
