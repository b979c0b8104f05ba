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
library's stream between steps, synchronised on both sides; also the median
step), the roofline of the dominant kernel class (the FP32 MFMA GEMMs) and a
per-class breakdown from the step profiler's events over K further steps, and
the float64 CPU oracle timed on the same B = 16 step (a sample of its 16
sequences, extrapolated; see cpu_baseline).

Measurements under the paper's kernel-benchmark protocol (25 warm-up runs,
100 timed, median, caches flushed between runs), each its own JSON line:
    python bench.py --sweep gemm   # standalone GEMM sweep at GPT-2 124M shapes
    python bench.py --block        # one transformer block, forward + backward
    python bench.py --kernels      # attention, GELU, LayerNorm, cross-entropy,
                                   # reduce-sum, AdamW at T = 1024 and 2048
"""
import os

# BLAS / OpenMP threads of the float64 oracle (the CPU baseline), fixed before
# numpy is first imported: the cores this process may run on, capped by a
# thread limit the environment already sets (this process's share of its host).
_AFFINITY = len(os.sched_getaffinity(0))
_ENV_CAP = os.environ.get("OMP_NUM_THREADS")
ORACLE_THREADS = min(_AFFINITY, int(_ENV_CAP)) if (_ENV_CAP or "").isdigit() and int(_ENV_CAP) > 0 else _AFFINITY
for _v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_v] = str(ORACLE_THREADS)

import argparse  # noqa: E402
import dataclasses  # noqa: E402
import json  # noqa: E402
import sys  # noqa: E402
import time  # noqa: E402

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
    ap.add_argument("--cpu-sample-seqs", type=int, default=2,
                    help="sequences of the B = 16 batch whose float64 forward + backward the CPU baseline times "
                         "(the step time is extrapolated to all 16; --cpu-sample-seqs 16 runs the whole step)")
    ap.add_argument("--sweep", choices=["gemm"], default=None,
                    help="gemm: the standalone FP32 GEMM sweep at GPT-2 124M shapes (M = 16384), NN / NT / TN")
    ap.add_argument("--block", action="store_true",
                    help="one GPT-2 124M transformer block, forward + backward, B = 16, T = 1024")
    ap.add_argument("--kernels", action="store_true",
                    help="the appendix kernels (attention, GELU, LayerNorm, sparse cross-entropy, reduce-sum, "
                         "AdamW) at the T = 1024 and T = 2048 shapes")
    ap.add_argument("--reps", type=int, default=100, help="timed runs per kernel in --sweep/--block/--kernels")
    ap.add_argument("--warm", type=int, default=25, help="warm-up runs per kernel in --sweep/--block/--kernels")
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


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(sample_seqs: int):
    """The float64 oracle, as it stands, timed on the host cores on the
    benchmark's own B = 16, T = 1024 step, run the way the oracle runs a
    16-micro-step accumulation: one sequence's forward + backward at a time,
    gradients summed, then the clip and AdamW over all 124.5M parameters.
    `sample_seqs` of the 16 sequences are timed (all 16 when it is 16) and
    the step time is 16 x their mean + the optimizer's time."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import gpt2 as og
    from paper_2606_24780_amd import synth

    cfg, hp = synth.GPT2_124M, synth.HP_124M
    specs = synth.param_specs(cfg)
    params = synth.init_params(cfg, 4)
    B, T = 16, cfg.max_T
    stream = synth.zipf_tokens(B * T + 1, cfg.V, 1.1, 40)
    x, y = synth.shifted_pair(stream, B, T)
    n = max(1, min(B, sample_seqs))
    grads = None
    seq_s = []
    for b in range(n):
        t0 = time.perf_counter()
        _, _, cache = og.forward(cfg, params, x[b:b + 1], y[b:b + 1])
        gb = og.backward(cfg, params, cache, 1.0 / (B * T))
        del cache
        if grads is None:
            grads = gb
        else:
            for k in grads:
                grads[k] += gb[k]
        seq_s.append(time.perf_counter() - t0)
    zeros = {k: np.zeros(s_, dtype=np.float64) for k, s_, _ in specs}
    t0 = time.perf_counter()
    og.optimizer_step(params, grads, zeros, zeros, 1, hp, specs)
    opt_s = time.perf_counter() - t0
    step_s = B * float(np.mean(seq_s)) + opt_s
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    what = ("the whole step" if n == B else
            f"{n} of the 16 sequences' forward + backward timed, step = 16 x their mean + the optimizer")
    return {"value": round(B * T / step_s, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 oracle on GPT-2 124M, B=16 x T=1024 (one sequence per micro-step, gradients "
                      f"summed, clip + AdamW over all 124.5M parameters); {what}",
            "step_s": round(step_s, 2), "seq_fwd_bwd_s": [round(t, 2) for t in seq_s],
            "optimizer_s": round(opt_s, 2), "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "affinity_cpus": _AFFINITY, "blas_threads_set": ORACLE_THREADS}


# ------------------------------------------------------- kernel measurements
# The paper's benchmark protocol (appendix "Hardware and Benchmarking
# Methodology"): 25 warm-up runs, 100 timed runs, the median, the caches
# flushed between runs.  Here the flush reads a 1 GiB buffer (larger than the
# 8 x 4 MB of L2 and the 256 MB memory-side cache) before every run: the
# kernel under test finds none of its data cached, and no dirty lines of the
# flush itself are left for it to write back.  Each run is bracketed by HIP
# events on the stream the kernels use.
class Protocol:
    def __init__(self, torch, warm, reps):
        self.torch, self.warm, self.reps = torch, warm, reps
        self.flush_buf = torch.empty((1 << 30) // 4, dtype=torch.float32, device="cuda")

    def median_ms(self, fn):
        torch = self.torch
        for _ in range(self.warm):
            fn()
        evs = []
        self.flush_buf.fill_(1.0)
        for _ in range(self.reps):
            self.flush_sum = self.flush_buf.sum()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            evs.append((e0, e1))
        torch.cuda.synchronize()
        ts = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
        return ts[len(ts) // 2], ts[0]


def protocol_info(pr):
    return {"warmup": pr.warm, "timed": pr.reps, "statistic": "median",
            "flush": "1 GiB buffer read before every timed run", "timer": "HIP events on the kernels' stream"}


def bench_gemm_sweep(a):
    """Config 2: M = 16384 (B = 16, T = 1024); for each (K, N) of GPT-2 124M
    the forward Y = X W (NN), the input gradient dX = dY W^T (NT) and the
    weight gradient dW = X^T dY (TN); X, dY ~ N(0, 1), W ~ N(0, 0.02)."""
    import torch

    from paper_2606_24780_amd import bt

    torch.cuda.set_device(0)
    pr = Protocol(torch, a.warm, a.reps)
    L = bt.lib()
    M = 16384
    g = torch.Generator(device="cuda").manual_seed(2)
    rows = []
    pairs = [(768, 2304), (768, 768), (768, 3072), (3072, 768), (768, 50304)]
    ws = torch.empty(max(max(L.bt_gemm_ws_bytes(0, 0, M, N, K, 0), L.bt_gemm_ws_bytes(0, 1, M, K, N, 0),
                             L.bt_gemm_ws_bytes(1, 0, K, N, M, 0)) for K, N in pairs) + 256,
                     dtype=torch.uint8, device="cuda")
    for K, N in pairs:
        X = torch.randn((M, K), generator=g, device="cuda")
        W = torch.randn((K, N), generator=g, device="cuda") * 0.02
        dY = torch.randn((M, N), generator=g, device="cuda")
        Y, dX, dW = torch.empty((M, N), device="cuda"), torch.empty((M, K), device="cuda"), torch.empty((K, N), device="cuda")
        prods = {
            "NN": (bt.OP_N, bt.OP_N, M, N, K, X, K, W, N, Y, N),
            "NT": (bt.OP_N, bt.OP_T, M, K, N, dY, N, W, N, dX, K),
            "TN": (bt.OP_T, bt.OP_N, K, N, M, X, K, dY, N, dW, N),
        }
        for lay, (oa, ob, m, n, k, A, lda, Bm, ldb, Cm, ldc) in prods.items():
            fn = lambda: bt.bt_gemm(oa, ob, m, n, k, A, lda, Bm, ldb, 0.0, Cm, ldc, ws=ws)
            med, best = pr.median_ms(fn)
            tf = 2.0 * m * n * k / (med / 1e3) / 1e12
            rows.append({"K": K, "N": N, "layout": lay, "product": f"{m}x{n}x{k}", "median_ms": round(med, 4),
                         "min_ms": round(best, 4), "tflops": round(tf, 2),
                         "frac_fp32_mfma_peak": round(tf / MFMA_FP32_PEAK_TFLOPS, 4),
                         "split_k_ws_bytes": int(L.bt_gemm_ws_bytes(oa, ob, m, n, k, 0))})
            print(json.dumps({"progress": rows[-1]}), file=sys.stderr, flush=True)
        del X, W, dY, Y, dX, dW
    tot_f = sum(2.0 * int(r["product"].split("x")[0]) * int(r["product"].split("x")[1]) *
                int(r["product"].split("x")[2]) for r in rows)
    tot_ms = sum(r["median_ms"] for r in rows)
    agg = tot_f / (tot_ms / 1e3) / 1e12
    print(json.dumps({
        "metric": "standalone FP32 GEMM sweep at GPT-2 124M shapes: TFLOP/s and fraction of FP32 MFMA peak",
        "value": round(agg, 2), "unit": "TFLOP/s", "n_gpus": 1, "higher_is_better": True, "dtype": "f32",
        "data": "synthetic", "vs_baseline": None,
        "config": {"workload": "GEMM sweep, M = 16384 (B = 16, T = 1024), (K, N) in (768, 2304), (768, 768), "
                               "(768, 3072), (3072, 768), (768, 50304); NN forward, NT input gradient, "
                               "TN weight gradient; X, dY ~ N(0, 1), W ~ N(0, 0.02)"},
        "roofline": {"bound": "mfma", "achieved": round(agg, 2), "peak": MFMA_FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(agg / MFMA_FP32_PEAK_TFLOPS, 4), "traffic": None},
        "protocol": protocol_info(pr), "rows": rows}))


def bench_block(a):
    """Config 3: one GPT-2 124M transformer block, forward + backward, composed
    from the C-ABI calls in the model's order (B = 16, T = 1024, C = 768,
    H = 12); weights and biases N(0, 0.02), LN gains 1 + N(0, 0.02), LN
    biases N(0, 0.02), x ~ N(0, 1), upstream gradient N(0, 1e-3)."""
    import numpy as np
    import torch

    from paper_2606_24780_amd import bt, synth

    torch.cuda.set_device(0)
    pr = Protocol(torch, a.warm, a.reps)
    L = bt.lib()
    B, T, C, H = 16, 1024, 768, 12
    hd, F, M = C // H, 4 * C, B * T
    p = synth.block_params(C, H, 3)
    d = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in p.items()}
    g = torch.Generator(device="cuda").manual_seed(3)
    X = torch.randn((M, C), generator=g, device="cuda")
    DY = torch.randn((M, C), generator=g, device="cuda") * 1e-3
    f = lambda *sh: torch.empty(sh, dtype=torch.float32, device="cuda")
    ln1, mu1, rs1, qkv, att, lse = f(M, C), f(M), f(M), f(M, 3 * C), f(M, C), f(B, H, T)
    x1, ln2, mu2, rs2, h, gg, y = f(M, C), f(M, C), f(M), f(M), f(M, F), f(M, F), f(M, C)
    gr = {k: f(*v.shape) for k, v in d.items()}
    dh, dln2, dx1, datt, dqkv, dln1, dx = f(M, F), f(M, C), f(M, C), f(M, C), f(M, 3 * C), f(M, C), f(M, C)
    ws_b = max(L.bt_gemm_ws_bytes(1, 0, F, C, M, 0), L.bt_gemm_ws_bytes(1, 0, C, F, M, 0),
               L.bt_gemm_ws_bytes(1, 0, C, 3 * C, M, 0), L.bt_attention_bwd_ws_bytes(B, T, H, hd),
               L.bt_layernorm_bwd_ws_bytes(M, C))
    ws = torch.empty(ws_b + 256, dtype=torch.uint8, device="cuda")
    N_, T_ = bt.OP_N, bt.OP_T

    def step():
        bt.bt_layernorm_fwd(X, d["ln1g"], d["ln1b"], ln1, mu1, rs1, M, C)
        bt.bt_gemm(N_, N_, M, 3 * C, C, ln1, C, d["Wqkv"], 3 * C, 0.0, qkv, 3 * C, bias=d["bqkv"], epi=bt.EPI_BIAS, ws=ws)
        bt.bt_attention_fwd(qkv, att, lse, B, T, H, hd)
        bt.bt_gemm(N_, N_, M, C, C, att, C, d["Wo"], C, 0.0, x1, C, bias=d["bo"], epi=bt.EPI_BIAS, residual=X, ws=ws)
        bt.bt_layernorm_fwd(x1, d["ln2g"], d["ln2b"], ln2, mu2, rs2, M, C)
        bt.bt_gemm(N_, N_, M, F, C, ln2, C, d["Wfc"], F, 0.0, gg, F, bias=d["bfc"], epi=bt.EPI_BIAS_GELU,
                   preact_out=h, ws=ws)
        bt.bt_gemm(N_, N_, M, C, F, gg, F, d["Wfp"], C, 0.0, y, C, bias=d["bfp"], epi=bt.EPI_BIAS, residual=x1, ws=ws)
        bt.bt_gemm(T_, N_, F, C, M, gg, F, DY, C, 0.0, gr["Wfp"], C, colsum_B=gr["bfp"], ws=ws)
        bt.bt_gemm(N_, T_, M, F, C, DY, C, d["Wfp"], C, 0.0, dh, F, epi=bt.EPI_DGELU, gelu_in=h, ws=ws)
        bt.bt_gemm(T_, N_, C, F, M, ln2, C, dh, F, 0.0, gr["Wfc"], F, colsum_B=gr["bfc"], ws=ws)
        bt.bt_gemm(N_, T_, M, C, F, dh, F, d["Wfc"], F, 0.0, dln2, C, ws=ws)
        dx1.copy_(DY)
        bt.bt_layernorm_bwd(dln2, x1, d["ln2g"], mu2, rs2, dx1, gr["ln2g"], gr["ln2b"], 1.0, 0.0, M, C, ws=ws)
        bt.bt_gemm(T_, N_, C, C, M, att, C, dx1, C, 0.0, gr["Wo"], C, colsum_B=gr["bo"], ws=ws)
        bt.bt_gemm(N_, T_, M, C, C, dx1, C, d["Wo"], C, 0.0, datt, C, ws=ws)
        bt.bt_attention_bwd(datt, qkv, att, lse, dqkv, B, T, H, hd, ws=ws)
        bt.bt_gemm(T_, N_, C, 3 * C, M, ln1, C, dqkv, 3 * C, 0.0, gr["Wqkv"], 3 * C, colsum_B=gr["bqkv"], ws=ws)
        bt.bt_gemm(N_, T_, M, C, 3 * C, dqkv, 3 * C, d["Wqkv"], 3 * C, 0.0, dln1, C, ws=ws)
        dx.copy_(dx1)
        bt.bt_layernorm_bwd(dln1, X, d["ln1g"], mu1, rs1, dx, gr["ln1g"], gr["ln1b"], 1.0, 0.0, M, C, ws=ws)

    med, best = pr.median_ms(step)
    gemm_f = 3 * 2.0 * M * (3 * C * C + C * C + 4 * C * C + 4 * C * C)
    attn_f = 12.0 * hd * B * H * T * (T + 1) / 2
    tf = (gemm_f + attn_f) / (med / 1e3) / 1e12
    print(json.dumps({
        "metric": "one GPT-2 124M transformer block, forward + backward: tokens/s on 1 GPU",
        "value": round(M / (med / 1e3), 1), "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True,
        "ms_per_step": round(med, 4), "dtype": "f32", "data": "synthetic", "vs_baseline": None,
        "config": {"workload": "one transformer block fwd+bwd (LN, QKV, causal attention, out-proj + residual, LN, "
                               "MLP with tanh-GELU, residual), B = 16, T = 1024, C = 768, H = 12, random LN and "
                               "bias parameters"},
        "roofline": {"bound": "mfma", "achieved": round(tf, 2), "peak": MFMA_FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / MFMA_FP32_PEAK_TFLOPS, 4), "traffic": None,
                     "flops": gemm_f + attn_f, "note": "algorithmic FLOPs of the 9 products and the attention "
                                                       "(4 + 8 hd per causal pair) over the whole block time"},
        "min_ms": round(best, 4), "protocol": protocol_info(pr)}))


def bench_kernels(a):
    """The appendix's per-kernel benchmarks, at the GPT-2 124M layer shapes
    with 16384 tokens as B x T = 16 x 1024 and 8 x 2048: causal attention
    forward / backward (H = 12, hd = 64), GELU forward / backward over the MLP
    activations (M x 3072), LayerNorm forward / backward (M x 768), sparse
    cross-entropy forward and backward over the 50,304-column logits, the
    reduce-sum of bias gradients (M x 3072 column sums) and AdamW over the
    124.5M-parameter arena.  Achieved GB/s on algorithmic bytes (every operand
    read or written once), TFLOP/s for attention."""
    import numpy as np
    import torch

    from paper_2606_24780_amd import bt, synth

    torch.cuda.set_device(0)
    pr = Protocol(torch, a.warm, a.reps)
    L = bt.lib()
    g = torch.Generator(device="cuda").manual_seed(5)
    rows = []

    def add(name, shape, fn, bytes_=None, flops=None):
        med, best = pr.median_ms(fn)
        r = {"kernel": name, "shape": shape, "median_ms": round(med, 4), "min_ms": round(best, 4)}
        if bytes_:
            r["gbs"] = round(bytes_ / (med / 1e3) / 1e9, 1)
            r["frac_hbm"] = round(r["gbs"] / HBM_PEAK_GBS, 4)
        if flops:
            r["tflops"] = round(flops / (med / 1e3) / 1e12, 2)
            r["frac_fp32_mfma_peak"] = round(r["tflops"] / MFMA_FP32_PEAK_TFLOPS, 4)
        rows.append(r)
        print(json.dumps({"progress": r}), file=sys.stderr, flush=True)

    C, H, hd, F, Vp, V = 768, 12, 64, 3072, 50304, 50257
    for B, T in ((16, 1024), (8, 2048)):
        M = B * T
        qkv = torch.randn((M, 3 * C), generator=g, device="cuda")
        out, lse = torch.empty((M, C), device="cuda"), torch.empty((B, H, T), device="cuda")
        dout = torch.randn((M, C), generator=g, device="cuda")
        dqkv = torch.empty_like(qkv)
        aws = torch.empty(L.bt_attention_bwd_ws_bytes(B, T, H, hd), dtype=torch.uint8, device="cuda")
        pairs = B * H * T * (T + 1) / 2
        tag = f"B={B} T={T}"
        add("attention_fwd (causal)", f"{tag} H={H} hd={hd}", lambda: bt.bt_attention_fwd(qkv, out, lse, B, T, H, hd),
            flops=4.0 * hd * pairs)
        add("attention_bwd (causal)", f"{tag} H={H} hd={hd}",
            lambda: bt.bt_attention_bwd(dout, qkv, out, lse, dqkv, B, T, H, hd, ws=aws), flops=8.0 * hd * pairs)
        del qkv, out, lse, dout, dqkv, aws
        x = torch.randn((M, F), generator=g, device="cuda")
        y = torch.empty_like(x)
        dy = torch.randn((M, F), generator=g, device="cuda")
        add("gelu_fwd", f"{tag} x [{M}, {F}]", lambda: bt.bt_gelu_fwd(x, y), bytes_=8.0 * M * F)
        add("gelu_bwd", f"{tag} x [{M}, {F}]", lambda: bt.bt_gelu_bwd(x, dy, y), bytes_=12.0 * M * F)
        cs = torch.empty(F, device="cuda")
        cws = torch.empty(L.bt_colsum_ws_bytes(M, F), dtype=torch.uint8, device="cuda")
        add("reduce_sum (column sums)", f"{tag} [{M}, {F}]", lambda: bt.bt_colsum(dy, M, F, F, cs, 0.0, ws=cws),
            bytes_=4.0 * M * F + 4.0 * F)
        del x, y, dy, cs, cws
        x = torch.randn((M, C), generator=g, device="cuda")
        gam = 1 + 0.02 * torch.randn(C, generator=g, device="cuda")
        bet = 0.02 * torch.randn(C, generator=g, device="cuda")
        yl, mu, rs = torch.empty_like(x), torch.empty(M, device="cuda"), torch.empty(M, device="cuda")
        dyl, dxl = torch.randn((M, C), generator=g, device="cuda"), torch.empty_like(x)
        dg, db = torch.empty(C, device="cuda"), torch.empty(C, device="cuda")
        lws = torch.empty(L.bt_layernorm_bwd_ws_bytes(M, C), dtype=torch.uint8, device="cuda")
        add("layernorm_fwd", f"{tag} [{M}, {C}]", lambda: bt.bt_layernorm_fwd(x, gam, bet, yl, mu, rs, M, C),
            bytes_=8.0 * M * C + 8.0 * M)
        add("layernorm_bwd", f"{tag} [{M}, {C}]",
            lambda: bt.bt_layernorm_bwd(dyl, x, gam, mu, rs, dxl, dg, db, 0.0, 0.0, M, C, ws=lws),
            bytes_=12.0 * M * C + 8.0 * M)
        del x, yl, dyl, dxl, lws
        z = torch.randn((M, Vp), generator=g, device="cuda")
        tgt = torch.from_numpy(synth.zipf_tokens(M, V, 1.1, 40)).cuda()
        lr_, ls_ = torch.empty(M, device="cuda"), torch.empty(M, device="cuda")
        dz = torch.empty_like(z)
        add("sparse_xent_fwd", f"{tag} logits [{M}, {Vp}]",
            lambda: bt.bt_softmax_xent_fwd(z, tgt, lr_, ls_, M, V, Vp), bytes_=4.0 * M * Vp + 12.0 * M)
        add("sparse_xent_bwd", f"{tag} logits [{M}, {Vp}]",
            lambda: bt.bt_softmax_xent_bwd(z, ls_, tgt, dz, 1.0 / M, M, V, Vp), bytes_=8.0 * M * Vp + 8.0 * M)
        del z, dz
    P, ND = 124475904, 124354560
    pp = torch.randn(P, generator=g, device="cuda")
    gg = torch.randn(P, generator=g, device="cuda") * 1e-3
    mm, vv = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
    add("adamw (one launch, flat arena)", f"P={P}",
        lambda: bt.bt_adamw_step(pp, gg, mm, vv, P, ND, 6e-4, 0.9, 0.95, 1e-8, 0.1, 1), bytes_=28.0 * P)
    print(json.dumps({
        "metric": "appendix per-kernel benchmarks at GPT-2 124M shapes (T = 1024 and T = 2048)",
        "value": None, "unit": None, "n_gpus": 1, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "attention fwd/bwd (causal, H = 12, hd = 64), GELU fwd/bwd, LayerNorm fwd/bwd, sparse "
                               "cross-entropy fwd/bwd, column reduce-sum, AdamW; 16384 tokens as 16 x 1024 and 8 x 2048"},
        "peaks": {"hbm_gbs": HBM_PEAK_GBS, "fp32_mfma_tflops": MFMA_FP32_PEAK_TFLOPS},
        "protocol": protocol_info(pr), "rows": rows}))


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
        print(f"bench.py: the benchmark runs on one GPU; only --gpus 1 is supported (got {a.gpus}): "
              "the multi-GPU data-parallel gradient exchange is not implemented", file=sys.stderr)
        sys.exit(2)
    if a.cp:
        bench_cp(a)
        return
    if a.sweep == "gemm":
        bench_gemm_sweep(a)
        return
    if a.block:
        bench_block(a)
        return
    if a.kernels:
        bench_kernels(a)
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

    # timed region: K steps, an event on the library's stream between steps
    # (no step profiler), synchronised on both sides
    s = model.stream
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    evs[0].record(s)
    losses = []
    for i in range(a.steps):
        losses.append(model.train_step(xd, yd))
        evs[i + 1].record(s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = evs[0].elapsed_time(evs[-1])
    step_ms = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(a.steps))
    median_ms = step_ms[len(step_ms) // 2]

    # per-class breakdown and the roofline: the same number of steps again with
    # the step profiler's events around every library call
    model.profile_enable(True)
    model.profile_read(reset=True)
    for _ in range(a.steps):
        model.train_step(xd, yd)
    prof = model.profile_read(reset=True)
    model.profile_enable(False)

    tok_s = a.steps * B * T / (ms / 1e3)
    copy_gbs = copy_bandwidth(torch)
    g = prof["gemm"]
    gemm_tflops = g["flops"] / (g["ms"] / 1e3) / 1e12 if g["ms"] > 0 else 0.0
    kernels = {}
    # the embedding backward also reads and writes the dwte rows of the
    # distinct tokens of the batch, which the library cannot count at launch
    n_distinct = int(np.unique(x).size)
    prof["emb_bwd"]["bytes"] += prof["emb_bwd"]["launches"] * 2.0 * 4 * n_distinct * cfg.C
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
        "ms_per_step": round(ms / a.steps, 3), "median_ms_per_step": round(median_ms, 3),
        "min_ms_per_step": round(step_ms[0], 3), "higher_is_better": True, "scaling": "weak",
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
        out["cpu_baseline"] = cpu_baseline(a.cpu_sample_seqs)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
