"""Host logic of bench.py (no GPU): algorithmic work, the source hash that gates the traffic figure,
the rocprofv3 summaries, and the one-GPU guard."""
import csv
import json
import os
import shutil
import subprocess
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, REPO)
import bench  # noqa: E402


def test_algorithmic_bytes_per_tensor():
    M, N, K, sb = 256, 128, 64, 8
    x_bf16, w_bf16, y_ref, dy = 2 * M * K, 2 * N * K, 2 * M * N, 2 * M * N
    x_packed, w_packed = M * (K // 2 + K // 32), N * (K // 2 + K // 32)  # codes + one E8M0 byte per 32
    s_fp, coeff = 4 * N * K // 32, 4 * N * K // sb                          # fp32 parameters
    grad_s, grad_c = s_fp, coeff
    assert bench.algorithmic_bytes("fwd_mfma_kernel", M, N, K, sb) == x_bf16 + w_bf16 + y_ref + dy
    assert bench.algorithmic_bytes("fwd_mfma_kernel_mx", M, N, K, sb) == x_packed + w_packed + y_ref + dy
    # the backward reads dY, X_hat and W with its scales and coefficients, and writes both gradients
    assert bench.algorithmic_bytes("bwd_mfma_kernel", M, N, K, sb) == dy + x_bf16 + w_bf16 + s_fp + coeff + grad_s + grad_c
    assert bench.algorithmic_bytes("bwd_mfma_mx_kernel", M, N, K, sb) == dy + x_packed + w_bf16 + s_fp + coeff + grad_s + grad_c
    # fake quantisation of one [N][K] bf16 tensor as the default steps run it
    assert bench.algorithmic_bytes("fq_act_mx_kernel", M, N, K, sb) == w_bf16 + w_packed
    assert bench.algorithmic_bytes("fq_weight_kernel", M, N, K, sb) == w_bf16 + s_fp + coeff + w_packed
    nv_s = 4 * N * K // 16
    assert bench.algorithmic_bytes("fq_weight_kernel", M, N, K, sb, fmt=1) == w_bf16 + nv_s + coeff + w_bf16
    assert bench.algorithmic_bytes("fq_act_nv_kernel", M, N, K, sb, fmt=1) == 2 * w_bf16
    assert bench.algorithmic_bytes("absmax_partial_kernel", M, N, K, sb, fmt=1) == w_bf16


def test_step_launch_map():
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block8192_mxfp4"]
    skip, shapes = bench.step_launches("fq_act_mx_kernel", w)
    assert skip == 0 and [s[1:] for s in shapes] == [(w.M, K) for K in w.inputs.values()]
    skip, shapes = bench.step_launches("fq_weight_kernel", w)
    assert skip == 0 and [s[1:] for s in shapes] == [(l.N, l.K) for l in w.linears]
    # the default step's grouped weight launch covers every linear: its bytes are their sum
    skip, shapes = bench.step_launches("fq_weight_group_kernel", w)
    assert skip == 0 and len(shapes) == 1 and shapes[0][1] == [(l.N, l.K) for l in w.linears]
    per_layer = sum(bench.algorithmic_bytes("fq_weight_kernel", w.M, l.N, l.K, w.sub_block, w.fmt) for l in w.linears)
    assert bench.launch_algorithmic_bytes("fq_weight_group_kernel", w, shapes[0]) == per_layer
    assert "fq_weight_group_kernel" in bench.PROFILED
    # NVFP4: the weights' tensor-absmax passes (one per linear) run before the step
    skip, shapes = bench.step_launches("absmax_partial_kernel", synth.WORKLOADS["block2560_nvfp4"])
    assert skip == 7 and len(shapes) == 4


def test_source_hash_ignores_comments_not_code(tmp_path):
    src = os.path.join(REPO, "paper_2608_01847_amd", "csrc")
    d = tmp_path / "csrc"
    shutil.copytree(src, d)
    h0 = bench.kernel_source_hash(str(d))
    assert h0 == bench.kernel_source_hash()
    f = d / "optim.hip"
    text = f.read_text()
    f.write_text("// a new comment line\n/* and a block\n comment */\n" + text.replace("\n", "\n\n", 3))
    assert bench.kernel_source_hash(str(d)) == h0
    f.write_text(text + "\nstatic int focus_unused_symbol = 1;\n")
    assert bench.kernel_source_hash(str(d)) != h0


def test_traffic_reported_only_for_the_recorded_hash(tmp_path):
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps({"bwd_mfma_mx_kernel": {"bytes_per_launch": 123.0, "source_hash": "abc", "launches": 7}}))
    assert bench.traffic_from_profile("bwd_mfma_mx_kernel", "abc", str(p)) == 123.0
    assert bench.traffic_from_profile("bwd_mfma_mx_kernel", "abd", str(p)) is None
    assert bench.traffic_from_profile("fwd_mfma_kernel", "abc", str(p)) is None
    assert bench.traffic_from_profile("bwd_mfma_mx_kernel", "abc", str(tmp_path / "missing.json")) is None


COLS = ["Correlation_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
        "End_Timestamp"]


def write_counter_csv(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=COLS)
        w.writeheader()
        for i, (disp, name, counter, value, ns) in enumerate(rows):
            w.writerow({"Correlation_Id": i, "Dispatch_Id": disp, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": value, "Start_Timestamp": 1000, "End_Timestamp": 1000 + ns})


BWD_MX = "void focus::bwd_mfma_mx_kernel<1>(unsigned short const*)"
COPY = "__amd_rocclr_copyBuffer"


def test_counter_summary_scales_by_the_copy(tmp_path):
    # the 1 GiB copy reads 524288 KiB on FETCH_SIZE (scale 2) and 1048576 KiB on WRITE_SIZE (scale 1)
    fetch = [(1, COPY, "FETCH_SIZE", 524288.0, 10)] + [(10 + i, BWD_MX, "FETCH_SIZE", 1000.0 * (i + 1), 10)
                                                       for i in range(7)]
    write = [(1, COPY, "WRITE_SIZE", 1048576.0, 10)] + [(10 + i, BWD_MX, "WRITE_SIZE", 10.0, 10) for i in range(7)]
    write_counter_csv(tmp_path / "f", fetch)
    write_counter_csv(tmp_path / "w", write)
    out = tmp_path / "out"
    out.mkdir()
    bench.summarize_counters(str(tmp_path / "f"), str(tmp_path / "w"), "block2560_mxfp4", out_dir=str(out))
    data = json.loads((out / "traffic_block2560_mxfp4.json").read_text())
    assert data["_calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert data["_calibration"]["write_scale"] == pytest.approx(1.0)
    want = sum(1000.0 * (i + 1) * 1024 * 2 + 10.0 * 1024 for i in range(7)) / 7
    assert data["bwd_mfma_mx_kernel"]["bytes_per_launch"] == pytest.approx(want)
    assert data["bwd_mfma_mx_kernel"]["source_hash"] == bench.kernel_source_hash()
    assert "fwd_mfma_kernel" not in data  # no rows, no entry
    assert (out / "hbm_traffic_block2560_mxfp4.md").exists()


FQ_ACT = "void focus::fq_act_mx_kernel<1, 1>(void const*, unsigned int)"


def test_counter_summary_maps_fakequant_launches(tmp_path):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    # one launch per block input in the step (4), then later launches that must be ignored
    fetch = [(1, COPY, "FETCH_SIZE", 524288.0, 10)] + [(10 + i, FQ_ACT, "FETCH_SIZE", 100.0, 10) for i in range(6)]
    write = [(1, COPY, "WRITE_SIZE", 1048576.0, 10)] + [(10 + i, FQ_ACT, "WRITE_SIZE", 50.0, 10) for i in range(6)]
    write_counter_csv(tmp_path / "f", fetch)
    write_counter_csv(tmp_path / "w", write)
    bench.summarize_counters(str(tmp_path / "f"), str(tmp_path / "w"), "block2560_mxfp4", out_dir=str(tmp_path))
    data = json.loads((tmp_path / "traffic_block2560_mxfp4.json").read_text())
    assert data["fq_act_mx_kernel"]["launches"] == 4
    assert data["fq_act_mx_kernel"]["bytes_per_launch"] == pytest.approx((100.0 * 2 + 50.0) * 1024)
    algs = [bench.algorithmic_bytes("fq_act_mx_kernel", w.M, w.M, K, 8) for K in w.inputs.values()]
    assert data["fq_act_mx_kernel"]["algorithmic_bytes_per_launch"] == pytest.approx(sum(algs) / 4)
    text = (tmp_path / "hbm_traffic_block2560_mxfp4.md").read_text()
    assert sum(l.startswith("| `fq_act_mx_kernel`") for l in text.splitlines()) == 4


ADAMW = "focus::adamw_kernel(float*, float const*)"
KLTOP = "void focus::(anonymous namespace)::kl_top_kernel<1>(void const*)"


def test_extras_summary_pools_each_launch_position(tmp_path):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    n = 2 * len(w.linears)  # AdamW launches per call: S_fp, then c, of every linear
    # three calls of AdamW: position j reads 10 j + 5 KiB in the middle call, +/- 1 in the others;
    # KL-Top twice, 2000 and 4000 KiB fetched (median 3000)
    fetch = [(1, COPY, "FETCH_SIZE", 524288.0, 10)]
    for call, d in enumerate((-1.0, 0.0, 1.0)):
        fetch += [(100 + call * n + j, ADAMW, "FETCH_SIZE", 10.0 * j + 5 + d, 10) for j in range(n)]
    fetch += [(500, KLTOP, "FETCH_SIZE", 2000.0, 10), (501, KLTOP, "FETCH_SIZE", 4000.0, 10)]
    write = [(1, COPY, "WRITE_SIZE", 1048576.0, 10)]
    for call in range(3):
        write += [(100 + call * n + j, ADAMW, "WRITE_SIZE", 7.0, 10) for j in range(n)]
    write += [(500, KLTOP, "WRITE_SIZE", 100.0, 10), (501, KLTOP, "WRITE_SIZE", 100.0, 10)]
    write_counter_csv(tmp_path / "f", fetch)
    write_counter_csv(tmp_path / "w", write)
    bench.summarize_extras(str(tmp_path / "f"), str(tmp_path / "w"), "block2560_mxfp4", out_dir=str(tmp_path))
    rows = [l for l in (tmp_path / "hbm_traffic_extras_block2560_mxfp4.md").read_text().splitlines()
            if l.startswith("| `")]
    adam = [l for l in rows if l.startswith("| `adamw_kernel`")]
    assert len(adam) == n
    # position 3 (k_proj's c): fetched (10 * 3 + 5) KiB x 2, written 7 KiB x 1
    lin = w.linears[1]
    cells = [c.strip() for c in adam[3].split("|")]
    assert cells[2] == f"{lin.name} c {lin.N}x{lin.K // w.sub_block}"
    assert float(cells[3]) == pytest.approx(35 * 1024 * 2 / 1e6, abs=0.05)
    assert float(cells[4]) == pytest.approx(7 * 1024 / 1e6, abs=0.05)
    assert float(cells[5]) == pytest.approx(28 * lin.N * (lin.K // w.sub_block) / 1e6, abs=0.05)
    kl = [l for l in rows if l.startswith("| `kl_top_kernel`")]
    assert len(kl) == 1 and float(kl[0].split("|")[3]) == pytest.approx(3000 * 1024 * 2 / 1e6, abs=0.05)
    assert not any(l.startswith("| `transpose_kernel`") for l in rows)  # no launches, no rows


def test_no_child_program_under_the_profiler(monkeypatch):
    def refuse(*a, **k):
        raise AssertionError("a child program was started under the profiler")
    monkeypatch.setattr(subprocess, "run", refuse)
    monkeypatch.setenv("ROCPROFILER_LIBRARY_CTOR", "1")
    assert bench.under_profiler()
    assert bench.gpu_clocks() == {"skipped": "under rocprofv3"}
    monkeypatch.delenv("ROCPROFILER_LIBRARY_CTOR")
    monkeypatch.setenv("LD_PRELOAD", "/opt/rocm/lib/rocprofiler-sdk/librocprofiler-sdk-tool.so")
    assert bench.under_profiler()


def test_mfma_summary_row(tmp_path):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    lin = w.linears[0]
    alg = 2.0 * w.M * lin.N * lin.K
    ns = 1.0e6
    busy = alg / 32768 * 32          # 32 busy cycles per 32x32x16 bf16 MFMA, summed over SIMDs
    util = 55.0                      # percent of GPU-busy cycles x 1024 SIMDs
    rows = [(20, BWD_MX, "MfmaUtil", util, ns), (20, BWD_MX, "SQ_VALU_MFMA_BUSY_CYCLES", busy, ns),
            (20, BWD_MX, "SQ_INSTS_VALU_MFMA_MOPS_BF16", alg / 512, ns),
            (20, BWD_MX, "SQ_LDS_BANK_CONFLICT", 10.0, ns), (20, BWD_MX, "SQ_LDS_IDX_ACTIVE", 1000.0, ns)]
    write_counter_csv(tmp_path / "m", rows)
    bench.summarize_mfma(str(tmp_path / "m"), "block2560_mxfp4", out_dir=str(tmp_path))
    text = (tmp_path / "mfma_util_block2560_mxfp4.md").read_text()
    row = next(l for l in text.splitlines() if l.startswith("| `bwd_mfma_mx_kernel`"))
    cells = [c.strip() for c in row.strip("|").split("|")]
    ghz = busy * 100 / (util * 1024) / ns
    frac = alg / ns / 1e3 / bench.PEAK_BF16_TFLOPS
    assert cells[1] == f"{lin.N}x{lin.K}"
    assert cells[3] == "55.0%"
    assert float(cells[4]) == pytest.approx(ghz, abs=0.006)
    assert cells[5] == "1.000"
    assert float(cells[7]) == pytest.approx(frac, abs=0.0006)
    assert float(cells[8]) == pytest.approx(frac * 2.4 / ghz, abs=0.0006)
    assert cells[9] == "1.0%"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=REPO)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_stall_summary_row(tmp_path):
    rows = [(30, BWD_MX, "SQ_WAVE_CYCLES", 1000.0, 5.0e5), (30, BWD_MX, "SQ_WAIT_ANY", 170.0, 5.0e5),
            (30, BWD_MX, "SQ_WAIT_INST_ANY", 343.0, 5.0e5), (30, BWD_MX, "SQ_ACTIVE_INST_LDS", 125.0, 5.0e5)]
    write_counter_csv(tmp_path / "s", rows)
    bench.summarize_stalls(str(tmp_path / "s"), "block2560_mxfp4", out_dir=str(tmp_path))
    text = (tmp_path / "gemm_stalls_block2560_mxfp4.md").read_text()
    row = next(l for l in text.splitlines() if l.startswith("| `bwd_mfma_mx_kernel`"))
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[2] == "500"
    assert cells[3:7] == ["17.0%", "34.3%", "0.0%", "12.5%"]


def test_memory_summary_row(tmp_path):
    from paper_2608_01847_amd import synth
    w = synth.WORKLOADS["block2560_mxfp4"]
    lin = w.linears[0]
    gui = 1.0e6
    op_kb = bench.algorithmic_bytes("bwd_mfma_mx_kernel", w.M, lin.N, lin.K, w.sub_block, w.fmt) / 1024
    rows = [(40, BWD_MX, "TCC_HIT_sum", 900.0, 5.0e5), (40, BWD_MX, "TCC_MISS_sum", 100.0, 5.0e5),
            (40, BWD_MX, "TA_BUSY_avr", 0.6 * gui, 5.0e5), (40, BWD_MX, "GRBM_GUI_ACTIVE", gui, 5.0e5),
            (40, BWD_MX, "TA_ADDR_STALLED_BY_TC_CYCLES_sum", 0.1 * 256 * gui, 5.0e5),
            (40, BWD_MX, "TCP_PENDING_STALL_CYCLES_sum", 0.2 * 256 * gui, 5.0e5),
            (40, BWD_MX, "TCP_TCC_READ_REQ_sum", 2.0 * op_kb, 5.0e5),
            (40, BWD_MX, "TCP_TCC_READ_REQ_LATENCY_sum", 2.0 * op_kb * 700, 5.0e5)]
    write_counter_csv(tmp_path / "mem", rows)
    bench.summarize_memory(str(tmp_path / "mem"), "block2560_mxfp4", out_dir=str(tmp_path))
    text = (tmp_path / "gemm_memory_block2560_mxfp4.md").read_text()
    row = next(l for l in text.splitlines() if l.startswith("| `bwd_mfma_mx_kernel`"))
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1] == f"{lin.N}x{lin.K}" and cells[2] == "500"
    assert cells[3:9] == ["0.900", "0.600", "0.100", "0.200", "700", "2.00"]
