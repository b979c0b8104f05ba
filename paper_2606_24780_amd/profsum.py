"""Summaries of rocprofv3 output for the GPT-2 124M FP32 training step (B=16, T=1024).

    python -m paper_2606_24780_amd.profsum stats STATS_CSV STEPS [--command CMD]
        kernel statistics (rocprofv3 --kernel-trace --stats) as a markdown table
        with the GEMM class's time and fraction of the FP32 matrix peak.
    python -m paper_2606_24780_amd.profsum ratio PMC_CSV NUM DEN FULL STEPS [--command CMD]
        per-kernel ratio of two counters of one --pmc pass (e.g. matrix-pipe busy
        cycles per GUI cycle, FULL being the value of a pipe busy every cycle).
    python -m paper_2606_24780_amd.profsum mode BENCH_JSON STATS_CSV [--command CMD ...]
        one of bench.py's protocol measurements (--sweep gemm, --block,
        --kernels): its table of medians beside the rocprofv3 kernel statistics
        of the same command.
    python -m paper_2606_24780_amd.profsum traffic COPY_FETCH COPY_WRITE STEP_FETCH STEP_WRITE STEPS \
        --stats STATS_CSV --json OUT.json --md OUT.md [--command CMD ...]
        HBM bytes per dispatch from the FETCH_SIZE / WRITE_SIZE passes (KiB per
        dispatch), scaled by what the same counters read for a plain 1 GiB copy:
        the GEMM class's bytes per bt_gemm call (JSON read by bench.py) and the
        memory-bound kernels' measured bytes against their algorithmic bytes.
    python -m paper_2606_24780_amd.profsum coverage LIBBT_SO STATS_CSV [--command CMD ...]
        which kernel instantiations of the built library a traced run (e.g. the
        GPU test suite under rocprofv3 --kernel-trace --stats) launched.

Reads the CSV files that rocprofv3 wrote (and, for coverage, the symbol
table of the library built here, through nm); runs nothing on the GPU.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
MFMA_FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0

# GPT-2 124M step at B = 16, T = 1024
M, C, F, VP, L = 16384, 768, 3072, 50304, 12


def gemm_products(M=M, C=C, L=L, VP=VP):
    """(m, n, k, extra m*n operands read or written by the epilogue) of the
    12 L + 3 bt_gemm calls of one step (M tokens, d_model C, MLP 4C, L
    layers, padded vocabulary VP), in call order."""
    F = 4 * C
    fwd = [(M, 3 * C, C, 0), (M, C, C, 1), (M, F, C, 1), (M, C, F, 1)]
    bwd = [(F, C, M, 0), (M, F, C, 1), (C, F, M, 0), (M, C, F, 0),
           (C, C, M, 0), (M, C, C, 0), (C, 3 * C, M, 0), (M, C, 3 * C, 0)]
    return fwd * L + [(M, VP, C, 0), (M, C, VP, 0), (VP, C, M, 0)] + bwd * L


def gemm_layouts(L=L):
    """Layout (NN forward, NT input gradient, TN weight gradient) of each
    product of gemm_products(), in the same order."""
    return ["NN"] * 4 * L + ["NT", "NN", "TN"] + ["TN", "NT"] * 4 * L


def gemm_layout_of(name: str):
    """Layout of a gemm_f32_mfma dispatch from its first two template
    arguments (K-contiguous A, K-contiguous B); None for other kernels."""
    n = short_name(name)
    if not n.startswith("gemm_f32_mfma<"):
        return None
    a, b = [x.strip() for x in n[len("gemm_f32_mfma<"):-1].split(",")[:2]]
    return {("true", "false"): "NN", ("true", "true"): "NT", ("false", "false"): "TN"}.get((a, b), "TT")


def gemm_flops_per_step(**dims):
    return sum(2.0 * m * n * k for m, n, k, _ in gemm_products(**dims))


def gemm_bytes_per_step():
    """A and B read once, C written once, epilogue operands (residual,
    pre-activation) touched once."""
    return sum(4.0 * (m * k + k * n + (1 + e) * m * n) for m, n, k, e in gemm_products())


# algorithmic HBM bytes per dispatch of the memory-bound kernels
LN_FWD_BYTES = 4.0 * (2 * M * C + 2 * M + 2 * C)
# dy, x read and dx written, plus dx read by the 24 accumulating calls of the 25
LN_BWD_BYTES = 4.0 * ((3 * M * C + 2 * M + C) + 24 * (4 * M * C + 2 * M + C)) / 25
XENT_BYTES = 8.0 * M * VP
P_124M = 124475904
ADAMW_BYTES = 28.0 * P_124M
SUMSQ_BYTES = 4.0 * P_124M
T_SEQ = 1024
# embedding forward: token ids, one wte row per token and the T wpe rows read,
# the M x C sum written
EMB_FWD_BYTES = 4.0 * (M + 2 * M * C + T_SEQ * C)
# token index: ids read, one (key, position) pair per token written
EMB_INDEX_BYTES = 4.0 * (M + 2 * M)


def emb_bwd_bytes(distinct: int) -> float:
    """Embedding backward (both kernels): the index pairs and dx0 read, dwpe
    written, and the dwte rows of the `distinct` tokens read and written
    (accumulated onto the LM head's contribution)."""
    return 4.0 * (2 * M + M * C + T_SEQ * C + 2 * distinct * C)


def short_name(name: str) -> str:
    n = re.sub(r"^void ", "", name)
    n = n.replace("bt::(anonymous namespace)::", "").replace("bt::", "")
    n = re.sub(r"\(.*\)$", "", n) if "rocprim" not in n else "rocprim (radix sort)"
    return n


def kernel_class(name: str) -> str:
    n = short_name(name)
    if n.startswith("gemm_f32_mfma<"):
        args = n[len("gemm_f32_mfma<"):-1].split(",")
        return "gemm" if args[-1].strip() == "0" else "attn_bwd"
    if n.startswith("splitk_reduce"):
        return "gemm"
    if n.startswith("attn_fwd"):
        return "attn_fwd"
    if n.startswith("attn_bwd"):
        return "attn_bwd"
    if n.startswith("ln_fwd"):
        return "ln_fwd"
    if n.startswith("ln_bwd") or n.startswith("sum_partials_batched"):
        return "ln_bwd"
    if n.startswith("xent"):
        return "xent"
    if n.startswith("adamw"):
        return "adamw"
    if n.startswith("sumsq") or n.startswith("norm_finish"):
        return "grad_norm"
    if n.startswith("emb_fwd"):
        return "emb_fwd"
    if n.startswith("emb_index"):
        return "emb_index"
    if n.startswith("emb_bwd") or n.startswith("emb_finish"):
        return "emb_bwd"
    return "other"


def read_stats(path):
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            rows.append(dict(name=r["Name"], calls=int(r["Calls"]), total_ns=float(r["TotalDurationNs"]),
                             avg_ns=float(r["AverageNs"]), pct=float(r["Percentage"])))
    return rows


def stats_markdown(path, steps, command=None, **dims):
    rows = read_stats(path)
    total = sum(r["total_ns"] for r in rows)
    out = []
    if command:
        out += ["Command (run from the repository root):", "", "```", command, "```", ""]
    out += [f"The profiled process runs {steps} training steps (warm-up, timed and profiled passes); per-step figures divide by "
            f"{steps}.", "", "| kernel | calls/step | ms/step | avg us | % of GPU time |", "|---|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        out.append(f"| `{short_name(r['name'])}` | {r['calls'] / steps:.6g} | {r['total_ns'] / steps / 1e6:.3f} | "
                   f"{r['avg_ns'] / 1e3:.1f} | {100 * r['total_ns'] / total:.1f} |")
    cls = defaultdict(float)
    for r in rows:
        cls[kernel_class(r["name"])] += r["total_ns"] / steps / 1e6
    g_ms = cls["gemm"]
    flops = gemm_flops_per_step(**dims)
    n_calls = len(gemm_products(**dims))
    tf = flops / (g_ms / 1e3) / 1e12
    out += ["", f"Total GPU kernel time per step: {total / steps / 1e6:.2f} ms.", "",
            "Per class (ms/step): " + ", ".join(f"{k} {v:.3f}" for k, v in sorted(cls.items(), key=lambda x: -x[1])),
            "", f"GEMM class (every `gemm_f32_mfma` instantiation with BMODE 0, i.e. the {n_calls} `bt_gemm` "
            "products of a step, plus their split-K reductions; the batched causal dQ product inside the attention "
            f"backward is attention): {g_ms:.2f} ms/step; algorithmic {flops:.4e} FLOP/step -> "
            f"{tf:.1f} TFLOP/s = {100 * tf / MFMA_FP32_PEAK_TFLOPS:.1f}% of the {MFMA_FP32_PEAK_TFLOPS} TFLOP/s "
            "FP32 matrix peak."]
    return "\n".join(out) + "\n"


def read_pmc(path, counter):
    """[(kernel name, value in KiB)] per dispatch, in dispatch order."""
    out = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    out.sort()
    return [(n, v) for _, n, v in out]


def copy_scale(path, counter, nbytes=1 << 30):
    """bytes per counter KiB, from the 1 GiB device copies of bench.py --calibrate-copy."""
    vals = [v for n, v in read_pmc(path, counter) if "copyBuffer" in n and v > 0]
    if not vals:
        raise SystemExit(f"{path}: no copy dispatch with {counter}")
    return nbytes / (max(vals) * 1024.0), max(vals)


def code_sha256(path):
    lines = []
    for line in open(path, encoding="utf-8"):
        line = re.sub(r"//.*$", "", line).rstrip()
        if line:
            lines.append(line)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def traffic(a):
    fs, fkib = copy_scale(a.copy_fetch, "FETCH_SIZE")
    ws, wkib = copy_scale(a.copy_write, "WRITE_SIZE")
    fetch = read_pmc(a.step_fetch, "FETCH_SIZE")
    write = read_pmc(a.step_write, "WRITE_SIZE")
    by = defaultdict(lambda: [0, 0.0, 0.0])  # class -> dispatches, fetch bytes, write bytes
    per_kernel = defaultdict(lambda: [0, 0.0, 0.0])
    for (n, v) in fetch:
        c = kernel_class(n)
        by[c][0] += 1
        by[c][1] += v * 1024 * fs
        k = short_name(n)
        per_kernel[k][0] += 1
        per_kernel[k][1] += v * 1024 * fs
    for (n, v) in write:
        by[kernel_class(n)][2] += v * 1024 * ws
        per_kernel[short_name(n)][2] += v * 1024 * ws
    steps = a.steps
    launches = 147 * steps
    g = by["gemm"]
    # per layout: product dispatches (split-K reductions listed on their own)
    lay = defaultdict(lambda: [0, 0.0, 0.0])
    for (n, v) in fetch:
        if kernel_class(n) != "gemm":
            continue
        k = gemm_layout_of(n) or "splitk_reduce"
        lay[k][0] += 1
        lay[k][1] += v * 1024 * fs
    for (n, v) in write:
        if kernel_class(n) != "gemm":
            continue
        lay[gemm_layout_of(n) or "splitk_reduce"][2] += v * 1024 * ws
    alg_lay = defaultdict(float)
    calls_lay = defaultdict(int)
    for (m, n, k, e), t in zip(gemm_products(), gemm_layouts()):
        alg_lay[t] += 4.0 * (m * k + k * n + (1 + e) * m * n)
        calls_lay[t] += 1
    per_layout = {}
    for t in ("NN", "NT", "TN"):
        meas = (lay[t][1] + lay[t][2]) / steps
        per_layout[t] = {"calls_per_step": calls_lay[t], "dispatches_per_step": lay[t][0] / steps,
                         "measured_bytes_per_step": round(meas), "algorithmic_bytes_per_step": round(alg_lay[t]),
                         "measured_over_algorithmic": round(meas / alg_lay[t], 3) if alg_lay[t] else None}
    rsum = (lay["splitk_reduce"][1] + lay["splitk_reduce"][2]) / steps
    per_layout["splitk_reduce"] = {"dispatches_per_step": lay["splitk_reduce"][0] / steps,
                                   "measured_bytes_per_step": round(rsum)}
    alg = gemm_bytes_per_step()
    rec = {
        "kernel": "gemm_f32_mfma (every bt_gemm call of the step, with its split-K reductions; not the batched "
                  "causal dQ product inside the attention backward)",
        "workload": "GPT-2 124M FP32 train step, B=16, T=1024 (147 products per step)",
        "commands": a.command or [],
        "copy_calibration": {"bytes_read": 1 << 30, "bytes_written": 1 << 30, "FETCH_SIZE_KiB": fkib,
                             "WRITE_SIZE_KiB": wkib, "fetch_scale": round(fs, 4),
                             "write_scale": round(ws, 4)},
        "steps_profiled": steps,
        "gemm_launches": launches,
        "gemm_kernel_dispatches_counted": g[0],
        "fetch_bytes_per_step": round(g[1] / steps),
        "write_bytes_per_step": round(g[2] / steps),
        "traffic_bytes_per_launch": round((g[1] + g[2]) / launches),
        "algorithmic_bytes_per_step": round(alg),
        "algorithmic_bytes_per_launch": round(alg / 147),
        "per_layout": per_layout,
        "gemm_source_sha256": code_sha256(os.path.join(HERE, "csrc", "gemm.hip")),
        "sha_note": "sha256 of gemm.hip with // comments and blank lines removed (bench.py code_sha256)",
    }
    with open(a.json, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    dur = {}
    if a.stats:
        for r in read_stats(a.stats):
            dur[short_name(r["name"])] = r["avg_ns"]
    alg_per = {"ln_fwd_kernel": LN_FWD_BYTES, "ln_bwd_kernel": LN_BWD_BYTES, "xent_stream_kernel": XENT_BYTES,
               "adamw_kernel": ADAMW_BYTES, "sumsq_kernel": SUMSQ_BYTES, "emb_fwd_kernel": EMB_FWD_BYTES,
               "emb_index_kernel": EMB_INDEX_BYTES}
    out = ["HBM-side bytes per dispatch from rocprofv3 `FETCH_SIZE` and `WRITE_SIZE` (separate passes), "
           f"scaled by a plain 1 GiB copy (counter bytes x {fs:.4f} for FETCH_SIZE, x {ws:.4f} for WRITE_SIZE).", ""]
    if a.command:
        out += ["Commands (run from the repository root):", "", "```"] + a.command + ["```", ""]
    out += ["| kernel | dispatches/step | read MB | written MB | measured MB | algorithmic MB | measured / alg. "
            "| avg us (stats run) | algorithmic GB/s | % of 8 TB/s |", "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for k, (nd, fb, wb) in sorted(per_kernel.items(), key=lambda x: -(x[1][1] + x[1][2])):
        base = next((b for p, b in alg_per.items() if k.startswith(p)), None)
        if base is None:
            continue
        base_note = base
        d = dur.get(k)
        gbs = base_note / (d * 1e-9) / 1e9 if d else float("nan")
        out.append(f"| `{k}` | {nd / steps:g} | {fb / nd / 1e6:.1f} | {wb / nd / 1e6:.1f} | {(fb + wb) / nd / 1e6:.1f} | "
                   f"{base_note / 1e6:.1f} | {(fb + wb) / nd / base_note:.3f} | {d / 1e3 if d else float('nan'):.1f} | "
                   f"{gbs:.0f} | {100 * gbs / HBM_PEAK_GBS:.1f} |")
    if getattr(a, "distinct", 0):
        # the two embedding-backward kernels share one algorithmic byte count
        parts = [k for k in per_kernel if k.startswith("emb_bwd_kernel") or k.startswith("emb_finish_kernel")]
        if parts:
            nd = per_kernel[parts[0]][0]
            fb = sum(per_kernel[k][1] for k in parts)
            wb = sum(per_kernel[k][2] for k in parts)
            base = emb_bwd_bytes(a.distinct)
            d = sum(dur.get(k, float("nan")) for k in parts)
            gbs = base / (d * 1e-9) / 1e9
            out.append(f"| `{' + '.join(sorted(parts))}` | {nd / steps:g} | {fb / nd / 1e6:.1f} | {wb / nd / 1e6:.1f} | "
                       f"{(fb + wb) / nd / 1e6:.1f} | {base / 1e6:.1f} | {(fb + wb) / nd / base:.3f} | {d / 1e3:.1f} | "
                       f"{gbs:.0f} | {100 * gbs / HBM_PEAK_GBS:.1f} |")
            out += ["", f"Embedding backward bytes count the dwte rows of the {a.distinct} distinct tokens of the "
                        "batch (read and written) plus the index pairs, dx0 and dwpe; the index kernel runs on a side "
                        "stream, overlapped with the first layer's forward."]
    out += ["", f"GEMM class: {g[0] / steps:g} dispatches per step (147 bt_gemm calls); "
            f"{(g[1] + g[2]) / launches / 1e6:.1f} MB per call measured against {alg / 147 / 1e6:.1f} MB algorithmic "
            f"({(g[1] + g[2]) / steps / alg:.2f}x)."]
    with open(a.md, "w") as f:
        f.write("\n".join(out) + "\n")
    print(json.dumps({k: rec[k] for k in ("traffic_bytes_per_launch", "algorithmic_bytes_per_launch",
                                          "gemm_kernel_dispatches_counted")}))


def ratio_markdown(path, num, den, full, steps, command=None):
    """Per kernel: sum of counter `num` over sum of counter `den` over its
    dispatches (one --pmc pass holding both), and that ratio over `full`."""
    acc = defaultdict(lambda: [0, 0.0, 0.0])
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            k = short_name(r["Kernel_Name"])
            if r["Counter_Name"] == num:
                acc[k][1] += float(r["Counter_Value"])
                acc[k][0] += 1
            elif r["Counter_Name"] == den:
                acc[k][2] += float(r["Counter_Value"])
    out = []
    if command:
        out += ["Command (run from the repository root):", "", "```", command, "```", ""]
    out += [f"| kernel | dispatches/step | {num} / {den} | of {full:g} |", "|---|---:|---:|---:|"]
    for k, (n, a, b) in sorted(acc.items(), key=lambda x: -x[1][2]):
        if b <= 0 or n == 0 or a <= 0:
            continue  # kernels that never use the counted unit
        out.append(f"| `{k}` | {n / steps:g} | {a / b:.1f} | {100 * a / b / full:.1f}% |")
    return "\n".join(out) + "\n"


def mode_markdown(bench_json, stats_csv, commands=None):
    """A bench.py protocol measurement (last JSON line of its output) and the
    rocprofv3 kernel statistics of the same command, as markdown."""
    lines = [ln for ln in open(bench_json).read().splitlines() if ln.strip().startswith("{")]
    rec = json.loads(lines[-1])
    out = [f"Workload: {rec['config']['workload']}.", ""]
    if commands:
        out += ["Commands (run from the repository root):", "", "```", *commands, "```", ""]
    pr = rec.get("protocol", {})
    out += [f"Protocol: {pr.get('warmup')} warm-up runs, {pr.get('timed')} timed runs, {pr.get('statistic')}; "
            f"{pr.get('flush')}; {pr.get('timer')}.", ""]
    rows = rec.get("rows")
    if rows:
        keys = [k for k in rows[0].keys() if k not in ("split_k_ws_bytes",)]
        for r in rows[1:]:
            keys += [k for k in r if k not in keys and k != "split_k_ws_bytes"]
        out += ["| " + " | ".join(keys) + " |", "|" + "---|" * len(keys)]
        for r in rows:
            out.append("| " + " | ".join(str(r.get(k, "")) for k in keys) + " |")
        out.append("")
    if rec.get("value") is not None:
        out += [f"Headline: {rec['metric']}: {rec['value']} {rec['unit']}"
                + (f"; roofline {rec['roofline']['achieved']} of {rec['roofline']['peak']} {rec['roofline']['unit']} "
                   f"= {100 * rec['roofline']['frac']:.1f}%" if rec.get("roofline") else "") + ".", ""]
    st = read_stats(stats_csv)
    total = sum(r["total_ns"] for r in st)
    out += ["rocprofv3 kernel statistics of the same command (every dispatch, warm-up runs and the cache-flush "
            "fills included):", "", "| kernel | calls | avg us | % of GPU time |", "|---|---:|---:|---:|"]
    for r in sorted(st, key=lambda r: -r["total_ns"]):
        out.append(f"| `{short_name(r['name'])}` | {r['calls']} | {r['avg_ns'] / 1e3:.1f} | "
                   f"{100 * r['total_ns'] / total:.1f} |")
    return "\n".join(out) + "\n"


def _plain_kernel_name(name):
    name = name.strip()
    return name[5:] if name.startswith("void ") else name


def library_kernels(lib_path):
    """The __global__ functions of a library built here: HIP gives each one a
    host-side handle, a data symbol named like the kernel (demangled, a
    function signature)."""
    import subprocess
    out = subprocess.run(["nm", "-C", lib_path], capture_output=True, text=True, check=True).stdout
    names = set()
    for ln in out.splitlines():
        parts = ln.split(" ", 2)
        if len(parts) == 3 and parts[1] in ("d", "D") and parts[2].rstrip().endswith(")"):
            names.add(_plain_kernel_name(parts[2]))
    return names


def coverage_markdown(lib_path, stats_csv, commands=None):
    """Kernel instantiations of the library launched / never launched by the
    traced run, per kernel family."""
    built = library_kernels(lib_path)
    launched = {_plain_kernel_name(r["name"]) for r in read_stats(stats_csv)}
    family = lambda n: re.split(r"[<(]", n.replace("(anonymous namespace)::", ""))[0].split("::")[-1]
    fams = defaultdict(lambda: [0, 0])
    for n in built:
        fams[family(n)][0] += 1
        fams[family(n)][1] += n in launched
    missing = sorted(n for n in built if n not in launched)
    out = []
    if commands:
        out += ["Commands (run from the repository root):", "", "```", *commands, "```", ""]
    out += [f"{len(built)} kernel instantiations in the library; {len(built) - len(missing)} launched by the traced "
            f"run, {len(missing)} not.", "", "| kernel | instantiations | launched |", "|---|---:|---:|"]
    for f, (nb, nl) in sorted(fams.items()):
        out.append(f"| `{f}` | {nb} | {nl} |")
    if missing:
        out += ["", "Not launched:", ""] + [f"- `{n}`" for n in missing]
    return "\n".join(out) + "\n"


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("steps", type=int)
    s.add_argument("--command")
    s.add_argument("--tokens", type=int, default=M, help="B*T (default 16384)")
    s.add_argument("--d-model", type=int, default=C)
    s.add_argument("--layers", type=int, default=L)
    s.add_argument("--vocab-padded", type=int, default=VP)
    t = sub.add_parser("traffic")
    for n in ("copy_fetch", "copy_write", "step_fetch", "step_write"):
        t.add_argument(n)
    t.add_argument("steps", type=int)
    t.add_argument("--stats")
    t.add_argument("--json", required=True)
    t.add_argument("--md", required=True)
    t.add_argument("--command", action="append")
    t.add_argument("--distinct", type=int, default=0,
                   help="distinct token ids of the profiled batch (embedding-backward bytes)")
    mo = sub.add_parser("mode")
    mo.add_argument("bench_json")
    mo.add_argument("stats")
    mo.add_argument("--command", action="append")
    r = sub.add_parser("ratio")
    r.add_argument("csv")
    r.add_argument("num")
    r.add_argument("den")
    r.add_argument("full", type=float)
    r.add_argument("steps", type=int)
    r.add_argument("--command")
    cv = sub.add_parser("coverage")
    cv.add_argument("lib")
    cv.add_argument("stats")
    cv.add_argument("--command", action="append")
    a = ap.parse_args()
    if a.cmd == "coverage":
        print(coverage_markdown(a.lib, a.stats, a.command), end="")
    elif a.cmd == "mode":
        print(mode_markdown(a.bench_json, a.stats, a.command), end="")
    elif a.cmd == "ratio":
        print(ratio_markdown(a.csv, a.num, a.den, a.full, a.steps, a.command), end="")
    elif a.cmd == "stats":
        print(stats_markdown(a.csv, a.steps, a.command, M=a.tokens, C=a.d_model, L=a.layers, VP=a.vocab_padded),
              end="")
    else:
        traffic(a)


if __name__ == "__main__":
    main()
