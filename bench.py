"""Benchmark: GPT-2 124M FP32 training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--batch 16] [--no-cpu-baseline]
    python bench.py --seq 16384            # long-context workload, B = 2
    python bench.py --model 2.42b          # largest-trainable-model workload, B = 2

One step = bt_gpt2_train_step: forward, backward, global-norm clip and AdamW
over all 124,475,904 parameters, B x T = 16 x 1024 tokens of a seeded Zipf
stream (a stand-in for the paper's FineWeb-Edu corpus), random-init weights
of the paper's initialisation.  Inputs are resident in HBM before timing.
The other two workloads print their own line (no CPU baseline: the float64
oracle's full step does not fit a bounded sample there).

Prints one JSON line: tokens/s over the K timed steps (HIP events on the
library's stream, synchronised on both sides), the live roofline of the
dominant kernel class (the FP32 MFMA GEMMs) from the step profiler's events
over the same timed region, a per-class breakdown, and the float64 CPU oracle
timed on a bounded sample of the same workload.
"""
import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_FP32_PEAK_TFLOPS = 157.3   # MI355X dense FP32 matrix peak
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E peak
PAPER_1GPU_TOKS = 54600         # paper, 1 GPU eager (RTX 6000 Ada): context only
PAPER_LONGCTX_TOKS = 17784      # paper, long-context table (RTX 6000 Ada, B=2, T=16384): context only
PAPER_2B_TOKS = 13600           # paper, largest-model table (RTX 6000 Ada, 2.42B, B=2, T=1024): context only


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--model", choices=["124m", "2.42b"], default="124m",
                    help="2.42b: the largest-trainable-model configuration (B = 2 by default)")
    ap.add_argument("--batch", type=int, default=None, help="default 16 (124M, T <= 1024), else 2")
    ap.add_argument("--seq", type=int, default=1024)
    ap.add_argument("--cp", type=int, default=0, metavar="W",
                    help="time one rank's share of context-parallel ring attention over W ranks "
                         "(GPT-2 124M attention at B=2, T=16384) instead of the training step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=2048)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run 3 plain device copies of 1 GiB (reference for HBM byte counters)")
    return ap.parse_args()


def code_sha256(path):
    """sha256 of a source file's code: // comments, trailing blanks and empty
    lines removed, so that comment edits do not count as kernel changes."""
    import hashlib
    import re
    lines = []
    for line in open(path, encoding="utf-8"):
        line = re.sub(r"//.*$", "", line).rstrip()
        if line:
            lines.append(line)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def gemm_traffic():
    """HBM bytes per GEMM launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE passes (scaled by a plain 1 GiB copy), or None when the GEMM
    code has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "gemm_f32_mfma_gpt2_124m_b16_traffic.json")
    src = os.path.join(ROOT, "paper_2606_24780_amd", "csrc", "gemm.hip")
    try:
        rec = json.load(open(path))
        sha = code_sha256(src)
    except (OSError, ValueError):
        return None, None
    if rec.get("gemm_source_sha256") != sha:
        return None, rec.get("algorithmic_bytes_per_launch")
    return rec.get("traffic_bytes_per_launch"), rec.get("algorithmic_bytes_per_launch")


def calibrate_copy():
    """A plain copy kernel of known size: the per-dispatch FETCH_SIZE and
    WRITE_SIZE counters it produces scale the counters of the path's kernels
    to bytes."""
    import torch
    n = (1 << 30) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "dispatches": 3}))


def copy_bandwidth(torch, nbytes=1 << 30, reps=5):
    """Achievable HBM bandwidth reference: a plain device-to-device copy of
    nbytes (read + write counted), best of `reps` timed with HIP events."""
    x = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    best = float("inf")
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        y.copy_(x)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del x, y
    return 2 * nbytes / (best / 1e3) / 1e9


def cpu_baseline(sample_tokens: int):
    """The float64 oracle, as it stands, on a bounded sample of the same
    workload: one full step (fwd + bwd + clip + AdamW over all parameters)
    of the 124M model on `sample_tokens` tokens of the same stream."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import gpt2 as og
    from paper_2606_24780_amd import synth

    cfg, hp = synth.GPT2_124M, synth.HP_124M
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 4)
    T = min(cfg.max_T, sample_tokens)
    B = max(1, sample_tokens // T)
    stream = synth.zipf_tokens(B * T + 1, cfg.V, 1.1, 40)
    x, y = synth.shifted_pair(stream, B, T)
    zeros = {k: np.zeros(s, dtype=np.float64) for k, s, _ in specs}
    t0 = time.perf_counter()
    og.train_step(cfg, hp, specs, params, zeros, zeros, x, y, t=1)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": B * T / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one full float64 step (fwd+bwd+clip+AdamW over all 124.5M params) of GPT-2 124M on "
                      f"{B}x{T} tokens of the benchmark's token stream; {dt:.1f} s wall",
            "seconds": dt, "host_cpus": os.cpu_count()}


def bench_cp(a):
    """One rank's share of context-parallel ring attention (section "Context
    Parallelism"): the attention of one GPT-2 124M layer (H = 12, hd = 64) at
    the long-context shape B = 2, T = 16384, spread over W ranks with the
    load-balanced two-chunk split.  A step is one rank's forward ring (W
    block forwards, merged) plus its backward ring (row sums, W block
    backwards); every rank is timed, all ranks' tensors resident on the one
    GPU.  The backward uses the stored-dS method (the recomputing one is
    timed beside it).  The shard exchange between GPUs is not part of this
    timing."""
    import numpy as np
    import torch

    from paper_2606_24780_amd import bt, ring

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    W, B, H, hd = a.cp, (a.batch or 2), 12, 64
    T = a.seq if a.seq != 1024 else 16384
    C = H * hd
    Tl = T // W
    bt.bt_cp_rank_segments(T, W, 0, 0)  # validates T against W
    g = torch.Generator(device="cuda").manual_seed(24780)
    qkv = [torch.randn((B * Tl, 3 * C), generator=g, device="cuda") for _ in range(W)]
    dout = [torch.randn((B * Tl, C), generator=g, device="cuda") for _ in range(W)]
    out = [torch.empty((B * Tl, C), device="cuda") for _ in range(W)]
    lse = [torch.empty((B, H, Tl), device="cuda") for _ in range(W)]
    D = [torch.empty((B, H, Tl), device="cuda") for _ in range(W)]
    dq = [torch.empty((B * Tl, 3 * C), device="cuda") for _ in range(W)]
    kv_of = lambda s: (qkv[s][:, C:], 3 * C)
    dkv_of = lambda s: dq[s][:, C:]
    # scratch of the stored-dS backward, shared by every step
    ws = torch.empty(ring.ws_bytes(W, T, B, H, hd), dtype=torch.uint8, device="cuda")
    ring.emulate(W, T, B, H, hd, qkv, out, lse, kv_of, dout=dout, D=D, dqkv=dq, dkv_of=dkv_of, ws=ws)
    torch.cuda.synchronize()

    def fwd(r):
        for i in range(W):
            kv, ks = kv_of(ring.shard_at(r, i, W))
            ring.forward_step(r, i, W, T, B, H, hd, qkv[r], kv, ks, out[r], lse[r])

    def bwd(r, scratch=ws):
        bt.bt_attention_rowdot(dout[r], out[r], D[r], B, Tl, H, hd)
        for i in range(W):
            s_ = ring.shard_at(r, i, W)
            kv, ks = kv_of(s_)
            ring.backward_step(r, i, W, T, B, H, hd, dout[r], qkv[r], kv, ks, lse[r], D[r], dq[r], dkv_of(s_),
                               scratch)

    def timed(fn, reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for r in range(W):
        for _ in range(a.warmup):
            fwd(r)
            bwd(r)
    torch.cuda.synchronize()
    fwd_ms = [timed(lambda: fwd(r), a.steps) for r in range(W)]
    bwd_ms = [timed(lambda: bwd(r), a.steps) for r in range(W)]
    bwd_recompute_ms = [timed(lambda: bwd(r, None), a.steps) for r in range(W)]
    del ws
    rank_ms = [f + b for f, b in zip(fwd_ms, bwd_ms)]
    # credited work: 4 hd FLOP per visible (query, key) pair forward, 8 hd
    # backward; the split gives every rank 1/W of the T (T + 1) / 2 pairs
    pairs = B * H * T * (T + 1) / 2 / W
    flops = 12 * hd * pairs
    tflops = [flops / (m / 1e3) / 1e12 for m in rank_ms]

    # the same layer's attention on one GPU over the whole sequence, / W
    full = torch.randn((B * T, 3 * C), generator=g, device="cuda")
    f_out = torch.empty((B * T, C), device="cuda")
    f_lse = torch.empty((B, H, T), device="cuda")
    f_do = torch.randn((B * T, C), generator=g, device="cuda")
    f_d = torch.empty_like(full)
    ws = torch.empty(bt.lib().bt_attention_bwd_ws_bytes(B, T, H, hd), dtype=torch.uint8, device="cuda")

    def whole():
        bt.bt_attention_fwd(full, f_out, f_lse, B, T, H, hd)
        bt.bt_attention_bwd(f_do, full, f_out, f_lse, f_d, B, T, H, hd, ws=ws)
    whole()
    whole_ms = timed(whole, max(1, a.steps // 2))
    del ws
    mean_ms = float(np.mean(rank_ms))
    tf = flops / (max(rank_ms) / 1e3) / 1e12
    rec = {
        "metric": "context-parallel ring attention, one rank's share: forward + backward TFLOP/s on 1 GPU",
        "value": round(tf, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(max(rank_ms), 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"one rank of W={W} context-parallel ring attention: GPT-2 124M attention layer "
                               f"(H={H}, hd={hd}), B={B}, T={T}, {Tl} local tokens in chunks of {Tl // 2}",
                   "W": W, "batch": B, "seq_len": T, "heads": H, "head_dim": hd},
        "roofline": {"kernel": "attn_fwd_kernel / attn_bwd_dq_kernel / attn_bwd_dkv_kernel (segmented), "
                               "slowest rank", "bound": "mfma", "achieved": round(tf, 2), "peak": 157.3,
                     "unit": "TFLOP/s", "frac": round(tf / 157.3, 4), "traffic": None,
                     "flops_per_rank": flops},
        "rank_fwd_ms": [round(x, 3) for x in fwd_ms], "rank_bwd_ms": [round(x, 3) for x in bwd_ms],
        "rank_bwd_recompute_ms": [round(x, 3) for x in bwd_recompute_ms],
        "rank_tflops": [round(x, 2) for x in tflops],
        "balance_max_over_min": round(max(rank_ms) / min(rank_ms), 4),
        "whole_sequence_one_gpu_ms": round(whole_ms, 3),
        "whole_sequence_over_W_ms": round(whole_ms / W, 3),
        "rank_mean_ms": round(mean_ms, 3),
    }
    print(json.dumps(rec))


def main():
    a = parse()
    if a.calibrate_copy:
        calibrate_copy()
        return
    if a.gpus != 1:
        print(f"bench.py: only --gpus 1 is supported by this build (got {a.gpus}); "
              "the multi-GPU data-parallel exchange is not implemented", file=sys.stderr)
        sys.exit(2)
    if a.cp:
        bench_cp(a)
        return
    import numpy as np
    import torch

    from paper_2606_24780_amd import bt, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    T = a.seq
    big = a.model == "2.42b"
    long_ctx = T > synth.GPT2_124M.max_T and not big
    B = a.batch if a.batch is not None else (2 if big or long_ctx else 16)
    # T above 1024: the long-context configuration (the 124M model with T
    # learned positions; section "Long-context training" runs B = 2, T = 16384)
    if big:
        cfg = dataclasses.replace(synth.GPT2_2_42B, max_T=max(T, synth.GPT2_2_42B.max_T))
    else:
        cfg = dataclasses.replace(synth.GPT2_124M, max_T=T) if long_ctx else synth.GPT2_124M
    hp = synth.HP_124M
    params = synth.init_params(cfg, 4)
    stream = synth.zipf_tokens(B * T + 1, cfg.V, 1.1, 40)
    x, y = synth.shifted_pair(stream, B, T)
    torch.cuda.reset_peak_memory_stats()
    model = bt.GPT2(cfg, hp, B, T)
    model.load_params(synth.flatten(cfg, params))
    xd = torch.from_numpy(x).cuda()
    yd = torch.from_numpy(y).cuda()
    torch.cuda.synchronize()

    for _ in range(a.warmup):
        model.train_step(xd, yd)
    torch.cuda.synchronize()

    model.profile_enable(True)
    model.profile_read(reset=True)
    s = model.stream
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(s)
    losses = []
    for _ in range(a.steps):
        losses.append(model.train_step(xd, yd))
    ev1.record(s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1)
    prof = model.profile_read(reset=True)
    model.profile_enable(False)

    tok_s = a.steps * B * T / (ms / 1e3)
    copy_gbs = copy_bandwidth(torch)
    g = prof["gemm"]
    gemm_tflops = g["flops"] / (g["ms"] / 1e3) / 1e12 if g["ms"] > 0 else 0.0
    kernels = {}
    for name, st in prof.items():
        if st["launches"] == 0:
            continue
        k = {"calls_per_step": st["launches"] / a.steps, "ms_per_step": st["ms"] / a.steps}
        if st["flops"] > 0 and name in ("gemm", "attn_fwd", "attn_bwd"):
            k["tflops"] = st["flops"] / (st["ms"] / 1e3) / 1e12
            k["frac_mfma_fp32"] = k["tflops"] / MFMA_FP32_PEAK_TFLOPS
        if st["bytes"] > 0 and name not in ("gemm", "attn_fwd", "attn_bwd"):
            k["gbs"] = st["bytes"] / (st["ms"] / 1e3) / 1e9
            k["frac_hbm"] = k["gbs"] / HBM_PEAK_GBS
            k["frac_copy"] = k["gbs"] / copy_gbs
        kernels[name] = k
    traffic, algo_bytes = gemm_traffic()
    if big or long_ctx or B != 16 or T != 1024:
        # the committed counters cover the B = 16, T = 1024 step only
        traffic, algo_bytes = None, None
    roofline = {
        "kernel": "gemm_f32_mfma (all bt_gemm calls of the step, incl. split-K reduction)",
        "bound": "mfma", "achieved": round(gemm_tflops, 3), "peak": MFMA_FP32_PEAK_TFLOPS,
        "unit": "TFLOP/s", "frac": round(gemm_tflops / MFMA_FP32_PEAK_TFLOPS, 4), "traffic": traffic,
        "traffic_unit": "bytes per launch (L2-to-memory FETCH_SIZE + WRITE_SIZE, copy-scaled)",
        "algorithmic_bytes_per_launch": algo_bytes,
        "launches": g["launches"], "avg_launch_ms": g["ms"] / max(1, g["launches"]),
        "flops_per_launch": g["flops"] / max(1, g["launches"]),
    }
    out = {
        "metric": ("GPT-2 2.42B FP32 train tokens/s on 1 GPU; GEMM fraction of FP32 MFMA peak" if big else
                   "GPT-2 124M FP32 long-context train tokens/s on 1 GPU; GEMM fraction of FP32 MFMA peak"
                   if long_ctx else "GPT-2 124M FP32 train tokens/s on 1 GPU; GEMM fraction of FP32 MFMA peak"),
        "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms / a.steps, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": ("GPT-2 2.42B FP32 train step (fwd+bwd+clip+AdamW), largest-trainable-model configuration"
                                if big else
                                f"GPT-2 124M FP32 long-context train step (fwd+bwd+clip+AdamW), {T} learned positions"
                                if long_ctx else
                                "GPT-2 124M FP32 train step (fwd+bwd+clip+AdamW), one GPU's data-parallel shard"),
                   "batch": B, "seq_len": T, "layers": cfg.L, "d_model": cfg.C, "heads": cfg.H,
                   "vocab": cfg.V, "vocab_padded": cfg.Vp, "params": model.P,
                   "tokens": "Zipf(1.1) synthetic stream, seed 40; params seed 4"},
        "roofline": roofline,
        "kernels": kernels,
        "wall_s": round(wall, 3),
        "loss_first_last": [losses[0], losses[-1]],
        "peak_mem_gib": round(torch.cuda.max_memory_allocated() / 2**30, 2),
        "hbm_copy_gbs": round(copy_gbs, 1),
        "paper_context_tokens_s": PAPER_2B_TOKS if big else PAPER_LONGCTX_TOKS if long_ctx else PAPER_1GPU_TOKS,
    }
    if not a.no_cpu_baseline and not (big or long_ctx):
        out["cpu_baseline"] = cpu_baseline(a.cpu_sample_tokens)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
