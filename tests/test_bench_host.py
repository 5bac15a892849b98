"""Host logic of bench.py that needs no GPU: the refusal of several GPUs, the reduction of a
rocprofv3 kernel trace and counter collection to the fenced timed regions (the summaries under
profiles/ are made this way), and the input check of the vendor comparison."""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def run_bench(*args):
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True,
                          cwd=ROOT, timeout=300)


def write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def table_rows(text, title):
    """{kernel: cells} of the markdown table that follows the heading containing `title`."""
    out, on = {}, False
    for line in text.splitlines():
        if line.startswith("###"):
            on = title in line
        elif on and line.startswith("| `"):
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            out[cells[0].strip("`")] = cells[1:]
    return out


def test_bench_refuses_several_gpus():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_trace_summary_keeps_only_fenced_launches(tmp_path):
    # a warm-up launch, then two fenced regions (spin-kernel pairs); timestamps in ns
    fence = "void pcm::spin_kernel(long)"
    gemm, comb = "void pcm::gemm_il_kernel<3>(pcm::GemmArgs)", "combine_kernel(float const*)"
    rows = [[gemm, 0, 50_000],                       # warm-up: outside every region
            [fence, 60_000, 61_000],
            [gemm, 62_000, 72_000], [comb, 72_500, 77_500], [gemm, 78_000, 98_000],
            [fence, 99_000, 100_000],
            [fence, 200_000, 201_000],
            [gemm, 202_000, 232_000],
            [fence, 233_000, 234_000]]
    write_csv(str(tmp_path / "run" / "t_kernel_trace.csv"),
              ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    r = run_bench("--trace-summary", str(tmp_path))
    assert r.returncode == 0, r.stderr
    reg0 = table_rows(r.stdout, "timed region 0")
    reg1 = table_rows(r.stdout, "timed region 1")
    g = "gemm_il_kernel<3>"
    # launches, avg, min, max, total (us)
    assert reg0[g] == ["2", "15.0", "10.0", "20.0", "30.0"]
    assert reg0["combine_kernel"] == ["1", "5.0", "5.0", "5.0", "5.0"]
    assert reg1 == {g: ["1", "30.0", "30.0", "30.0", "30.0"]}
    assert "spin_kernel" not in r.stdout


def test_trace_summary_counters_mfma_busy_and_clock(tmp_path):
    # one fenced dispatch of 100 us: 8 XCDs count 170000 GUI cycles each (1.7 GHz) and 1024
    # SIMDs 119000 MFMA-busy cycles each (70% busy)
    fence = "void pcm::spin_kernel(long)"
    k = "void pcm::gemm_il_kernel<0>(pcm::GemmArgs)"
    hdr = ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Counter_Name",
           "Counter_Value"]
    rows = []
    for did, name, t0, t1 in ((1, fence, 0, 1_000), (2, k, 2_000, 102_000), (3, fence, 103_000, 104_000)):
        busy, gui = (1024 * 119_000, 8 * 170_000) if name == k else (0, 8 * 1_000)
        rows.append([did, name, t0, t1, "SQ_VALU_MFMA_BUSY_CYCLES", busy])
        rows.append([did, name, t0, t1, "GRBM_GUI_ACTIVE", gui])
    write_csv(str(tmp_path / "c" / "c_counter_collection.csv"), hdr, rows)
    r = run_bench("--trace-summary", str(tmp_path))
    assert r.returncode == 0, r.stderr
    cells = table_rows(r.stdout, "counters, timed region 0")["gemm_il_kernel<0>"]
    # dispatches, avg us, GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES, MFMA busy, clock GHz
    assert cells[0] == "1" and cells[1] == "100.0"
    assert cells[-2:] == ["70.0%", "1.70"]


def test_vendor_compare_needs_uniform_rows():
    # 60 experts do not divide the fine-grained workload's 16384 tokens
    r = run_bench("--vendor-compare", "--config", "finegrained_shared")
    assert r.returncode != 0
    assert "multiples of n" in r.stderr
