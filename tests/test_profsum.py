"""The rocprofv3 summariser (CPU): step totals of the GEMM class and the
parsing of the statistics and counter CSVs it reads."""
import csv
import json

from paper_2606_24780_amd import profsum


def test_gemm_totals_match_the_step():
    # 12 layers x 12 products + 3 LM-head products; FLOPs 2MNK summed
    prods = profsum.gemm_products()
    assert len(prods) == 147
    assert profsum.gemm_flops_per_step() == 12147241254912
    assert profsum.gemm_bytes_per_step() == 46554808320


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(header)
        w.writerows(rows)


PMC = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size", "Kernel_Id",
       "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count",
       "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _pmc_row(i, name, counter, kib):
    return [i, i, "Agent 1", 1, 1, 1, 256, 1, name, 256, 0, 0, 4, 0, 16, counter, kib, 0, 1]


def test_stats_and_traffic_parsing(tmp_path):
    gemm = "void bt::(anonymous namespace)::gemm_f32_mfma<true, true, 0, false, false, 16, 4, 2, 2, 2, 2, true, 0>(x)"
    dq = "void bt::(anonymous namespace)::gemm_f32_mfma<true, false, 0, false, false, 16, 1, 2, 2, 2, 1, true, 1>(x)"
    ln = "void bt::(anonymous namespace)::ln_fwd_kernel<3, 2>(float const*)"
    stats = tmp_path / "s.csv"
    _write(stats, ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"],
           [[gemm, 2, 2e6, 1e6, 90.0, 1, 1, 0], [dq, 2, 1e5, 5e4, 5.0, 1, 1, 0], [ln, 50, 1e5, 2e3, 5.0, 1, 1, 0]])
    md = profsum.stats_markdown(str(stats), 2)
    assert "`gemm_f32_mfma<true, true, 0, false, false, 16, 4, 2, 2, 2, 2, true, 0>` | 1 | 1.000 |" in md
    assert profsum.kernel_class(dq) == "attn_bwd" and profsum.kernel_class(gemm) == "gemm"
    # copy calibration: 1 GiB read as 524288 KiB of FETCH_SIZE (x2), written as 1048576 KiB
    cf, cw = tmp_path / "cf.csv", tmp_path / "cw.csv"
    _write(cf, PMC, [_pmc_row(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288.0)])
    _write(cw, PMC, [_pmc_row(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576.0)])
    sf, sw = tmp_path / "sf.csv", tmp_path / "sw.csv"
    _write(sf, PMC, [_pmc_row(i, ln, "FETCH_SIZE", 100.0) for i in range(50)])
    _write(sw, PMC, [_pmc_row(i, ln, "WRITE_SIZE", 200.0) for i in range(50)])

    import types
    A = types.SimpleNamespace(copy_fetch=str(cf), copy_write=str(cw), step_fetch=str(sf), step_write=str(sw), steps=2,
                              stats=str(stats), json=str(tmp_path / "t.json"), md=str(tmp_path / "t.md"),
                              command=["cmd"])
    profsum.traffic(A)
    rec = json.load(open(A.json))
    assert rec["copy_calibration"]["fetch_scale"] == 2.0 and rec["copy_calibration"]["write_scale"] == 1.0
    assert rec["gemm_launches"] == 294
    text = open(A.md).read()
    # 100 KiB x 2048 B read and 200 KiB x 1024 B written per dispatch
    assert "| `ln_fwd_kernel<3, 2>` | 25 | 0.2 | 0.2 | 0.4 |" in text
    assert set(rec["per_layout"]) == {"NN", "NT", "TN", "splitk_reduce"}


def test_gemm_layouts():
    lay = profsum.gemm_layouts()
    prods = profsum.gemm_products()
    assert len(lay) == len(prods) == 147
    assert lay.count("NN") == 49 and lay.count("NT") == 49 and lay.count("TN") == 49
    # the weight-gradient products reduce over the M = 16384 tokens, the others keep M rows
    for (m, n, k, e), t in zip(prods, lay):
        assert (k == profsum.M) == (t == "TN")
    g = "void bt::(anonymous namespace)::gemm_f32_mfma<{}, {}, 0, false, false, 16, 4, 2, 2, 2, 2, true, 0>(x)"
    assert profsum.gemm_layout_of(g.format("true", "false")) == "NN"
    assert profsum.gemm_layout_of(g.format("true", "true")) == "NT"
    assert profsum.gemm_layout_of(g.format("false", "false")) == "TN"
    assert profsum.gemm_layout_of("void bt::(anonymous namespace)::splitk_reduce<0>(x)") is None


def test_embedding_bytes():
    # ids + index pairs + dx0 + dwpe + 2 x dwte rows of the distinct tokens, float32
    M, C, T = 16384, 768, 1024
    assert profsum.emb_bwd_bytes(4132) == 4.0 * (2 * M + M * C + T * C + 2 * 4132 * C)
    assert profsum.EMB_FWD_BYTES == 4.0 * (M + 2 * M * C + T * C)


def test_mode_markdown(tmp_path):
    bench = tmp_path / "b.json"
    bench.write_text('{"progress": 1}\n' + json.dumps({
        "metric": "m", "value": 2.0, "unit": "u", "config": {"workload": "w"},
        "roofline": {"achieved": 1.0, "peak": 2.0, "unit": "TFLOP/s", "frac": 0.5},
        "protocol": {"warmup": 25, "timed": 100, "statistic": "median", "flush": "f", "timer": "t"},
        "rows": [{"kernel": "a", "median_ms": 0.5}, {"kernel": "b", "median_ms": 1.0, "gbs": 3.0}]}) + "\n")
    stats = tmp_path / "s.csv"
    stats.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
                     '"k1",2,4000,2000,80,1,1,0\n"k2",1,1000,1000,20,1,1,0\n')
    md = profsum.mode_markdown(str(bench), str(stats), ["cmd"])
    assert "| kernel | median_ms | gbs |" in md and "| b | 1.0 | 3.0 |" in md
    assert "50.0%" in md and "| `k1` | 2 | 2.0 | 80.0 |" in md


def test_coverage_markdown(tmp_path):
    """Kernel instantiations of the built library (its host-side kernel
    handles) against the kernels a traced run launched."""
    import os
    import pytest
    lib = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2606_24780_amd",
                       "libbt.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    import shutil
    if shutil.which("nm") is None:
        pytest.skip("nm (binutils) not installed")
    built = profsum.library_kernels(lib)
    assert "bt::fill_zero_kernel(float*, unsigned long)" in built
    assert sum("gemm_f32_mfma<" in n for n in built) > 40
    assert not any(n.startswith("void ") for n in built)
    picked = sorted(built)[:3]
    stats = tmp_path / "s.csv"
    _write(stats, ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"],
           [["void " + picked[0], 1, 1e3, 1e3, 50.0, 1, 1, 0], [picked[1], 2, 1e3, 5e2, 40.0, 1, 1, 0],
            [picked[2], 1, 1e2, 1e2, 5.0, 1, 1, 0], ["__amd_rocclr_copyBuffer", 4, 1e2, 25, 5.0, 1, 1, 0]])
    md = profsum.coverage_markdown(lib, str(stats), ["cmd"])
    assert f"{len(built)} kernel instantiations in the library; 3 launched by the traced run, " \
           f"{len(built) - 3} not." in md
    assert f"- `{picked[0]}`" not in md and f"- `{sorted(built)[3]}`" in md
    assert "| `fill_zero_kernel` | 1 |" in md
