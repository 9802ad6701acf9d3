"""Host-side logic of bench.py (no GPU): kernel-instance naming and the
counter-record summary."""
import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("O,I,name", [
    (4096, 4096, "gemv_b1_kernel<4, 4, false, false>"),      # 8192 blocks: one-shot, 1024 tiles -> T = 4
    (1024, 4096, "gemv_b1_kernel<4, 1, false, false>"),
    (14336, 4096, "gemv_b1s_kernel<4, 4, false, false, false>"),  # 28672 blocks: streaming, 8 gblocks: depth 4
    (4096, 14336, "gemv_b1s_kernel<4, 2, true, false, false>"),   # 28 gblocks per row, 4 tiles per workgroup
    (8192, 28672, "gemv_b1s_kernel<4, 3, true, false, false>"),   # 56 gblocks per row, 8 tiles per workgroup
    (8192, 8192, "gemv_b1s_kernel<4, 2, false, false, false>"),
    (1024, 8192, "gemv_b1_kernel<4, 1, false, false>"),
    (8192, 1024, "gemv_b1_kernel<4, 2, false, false>"),      # 2 gblocks: T = 2 keeps >= 2048 wavefronts
    (2048, 4096, "gemv_b1_kernel<4, 2, false, false>"),
])
def test_kernel_instance_names(O, I, name):
    assert bench.b1_kernel_instance(O, I, 4) == name
    assert bench.b1_kernel_instance(O, I, 4, a8=True) == name.replace("false, false>", "true, false>")
    # the coefficient-cache format keeps the depth-2 ring of 512 workgroups
    ix_name = name.replace("false, false>", "false, true>").replace("gemv_b1s_kernel<4, 4,", "gemv_b1s_kernel<4, 2,")
    assert bench.b1_kernel_instance(O, I, 4, ix=True) == ix_name


def _write_counter_csv(path, counter, rows):
    """rows: (kernel, value) or (kernel, value, grid threads)."""
    cols = ["Correlation_Id", "Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=cols)
        w.writeheader()
        for i, row in enumerate(rows):
            kernel, value = row[0], row[1]
            grid = row[2] if len(row) > 2 else 131072
            w.writerow({"Correlation_Id": i, "Dispatch_Id": i, "Grid_Size": grid, "Kernel_Name": kernel,
                        "Counter_Name": counter, "Counter_Value": value})


def test_traffic_summary_scales_by_copy(tmp_path):
    copy = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(at::TensorIteratorBase&)::{lambda()#1}>"
    kern = "void sbvr::gemv_b1s_kernel<4, 2, false, false, false>(sbvr::GemvArgs)"
    calib_kib = bench.CALIB_BYTES / 1024
    # counters that see half of what moves: the scale must double them back
    _write_counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                       [(kern, 16000.0), (kern, 16200.0), (kern, 16100.0), (copy, calib_kib / 2)])
    _write_counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                       [(kern, 7.0), (kern, 7.0), (kern, 7.0), (copy, calib_kib / 2)])
    text = bench.traffic_summary(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    import json
    import re
    rec = json.loads(re.search(r"^traffic-record: (\{.*\})$", text, re.M).group(1))
    k = rec["kernels"]["gemv_b1s_kernel<4, 2, false, false, false>"]
    assert k["dispatches"] == 3
    assert k["bytes_per_launch"] == round(16100.0 * 1024 * 2 + 7.0 * 1024 * 2)
    assert rec["source_sha256"] == bench.kernel_source_digest()


def test_traffic_summary_separates_grids_and_sizes(tmp_path):
    """One instance at two grids is keyed per grid; one launch configuration
    serving two shapes (same grid, 4x the bytes) is split by size."""
    copy = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(at::TensorIteratorBase&)::{lambda()#1}>"
    kern = "void sbvr::gemm_sbs_kernel<4, 8, 2, false>(sbvr::GemvArgs)"
    calib_kib = bench.CALIB_BYTES / 1024
    rows = [(kern, 1200.0), (kern, 4800.0), (kern, 1210.0), (kern, 4790.0), (kern, 9000.0, 65536),
            (copy, calib_kib)]
    _write_counter_csv(tmp_path / "f.csv", "FETCH_SIZE", rows)
    _write_counter_csv(tmp_path / "w.csv", "WRITE_SIZE", [(r[0], 0.0) + tuple(r[2:]) for r in rows[:-1]]
                       + [(copy, calib_kib)])
    text = bench.traffic_summary(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    import json
    import re
    rec = json.loads(re.search(r"^traffic-record: (\{.*\})$", text, re.M).group(1))["kernels"]
    base = "gemm_sbs_kernel<4, 8, 2, false> grid 131072"
    assert rec[base + " size 1 of 2"]["dispatches"] == 2
    assert rec[base + " size 1 of 2"]["bytes_per_launch"] == round(1205.0 * 1024)
    assert rec[base + " size 2 of 2"]["bytes_per_launch"] == round(4795.0 * 1024)
    assert rec["gemm_sbs_kernel<4, 8, 2, false> grid 65536"]["bytes_per_launch"] == 9000 * 1024


def test_more_than_one_gpu_is_refused():
    """bench.py measures one GPU: --gpus N > 1 exits with a message (before
    touching torch or the GPU)."""
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_kernel_summary_groups_dispatches(tmp_path):
    """--kernel-summary: per (instance, workgroup, grid) mean and median of
    end - start, over all dispatches and over the back-to-back ones (started
    when the dispatch before them, of any kernel, ended), the traced run's
    own per-launch times, and the machine-readable record the bench reads
    back."""
    cols = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Workgroup_Size_X", "Grid_Size_X"]
    gate = "void sbvr::gemv_b1s_kernel<4, 4, false, false, false>(HIP_vector_type<unsigned int, 4u> const*)"
    kv = "void sbvr::gemv_b1_kernel<4, 1, false, false>(HIP_vector_type<unsigned int, 4u> const*)"
    # gate 2 starts when the other kernel ends, gate 3 when gate 2 ends: back to
    # back; gate 1 and the k/v launch start after a gap
    rows = [(gate, 1000, 8000, 512, 131072), ("other_kernel(int)", 8500, 9000, 64, 64),
            (gate, 9000, 16200, 512, 131072), (gate, 16200, 23600, 512, 131072),
            (kv, 30000, 32600, 512, 131072)]
    path = tmp_path / "trace.csv"
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(cols)
        for name, a, b, wg, grid in rows:
            w.writerow(["KERNEL_DISPATCH", name, a, b, wg, grid])
    shapes = {"q": [4096, 4096], "k": [1024, 4096], "v": [1024, 4096], "o": [4096, 4096], "gate": [14336, 4096],
              "up": [14336, 4096], "down": [4096, 14336]}
    line = {"config": {"workload": "llama3-8b decode-layer projections; SBVR k=4, group 128", "shapes": shapes},
            "step_launch_us": {"q": 3.8, "k": 2.6, "v": 2.6, "o": 3.8, "gate": 7.5, "up": 7.3, "down": 7.7}}
    js = tmp_path / "bench.json"
    js.write_text("some log line\n" + json.dumps(line) + "\n")
    text = bench.kernel_summary(str(path), str(js))
    assert ("| `gemv_b1s_kernel<4, 4, false, false, false>` | 512 | 131072 | 3 | 7200 | 7200 | 7000 | 7400 | "
            "2 | 7300 | 7300 |") in text
    assert "| `gemv_b1_kernel<4, 1, false, false>` | 512 | 131072 | 1 | 2600 | 2600 | 2600 | 2600 | 0 | - | - |" in text
    assert "other_kernel" not in text
    rec = [ln for ln in text.splitlines() if ln.startswith("rocprof-record:")]
    r = json.loads(rec[0].split(":", 1)[1])
    assert r["kernels"]["gemv_b1s_kernel<4, 4, false, false, false>"] == {
        "workgroup": 512, "grid": 131072, "calls": 3, "mean_ns": 7200.0, "median_ns": 7200.0,
        "b2b_calls": 2, "b2b_mean_ns": 7300.0, "b2b_median_ns": 7300.0, "traced_live_us": 7.4}
    assert r["kernels"]["gemv_b1_kernel<4, 1, false, false>"]["traced_live_us"] == 2.6
    assert r["source_sha256"] == bench.kernel_source_digest()


def test_prefill_summary_segments_by_marker(tmp_path):
    """--prefill-summary: phases are cut at the marker fills, the second pass
    of each case is used, library time is per call (all its kernels summed)."""
    fill = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>(int)"
    dec = "void sbvr::decompress_kernel<4, false, 4>(sbvr::Dims)"
    lib = "Cijk_Alik_Bljk_HHS_BH_MT16x16x256"
    fus = "void sbvr::prefill_kernel<4, 1>(sbvr::PrefillArgs)"
    n = bench.PREFILL_PROBE_CALLS
    rows, t = [(fill, 0, 1)], 10

    def add(name, dur, count):
        nonlocal t
        for _ in range(count):
            rows.append((name, t, t + dur))
            t += dur + 5

    for ci, _ in enumerate(bench.prefill_probe_cases()):
        for rep in range(2):
            scale = 1 if rep else 3  # first pass slower: must be ignored
            add(fill, 1, 1)
            add(dec, 1000 * scale + ci, n)
            add(fill, 1, 1)
            add(lib, 500 * scale, 2 * n)  # two library kernels per call
            add("__amd_rocclr_fillBufferAligned", 7, 1)
            add(fill, 1, 1)
            add(fus, 2000 * scale, n)
    path = tmp_path / "trace.csv"
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writerows(rows)
    text = bench.prefill_summary(str(path))
    import json
    rec = json.loads([ln for ln in text.splitlines() if ln.startswith("prefill-record:")][0].split(":", 1)[1])
    cases = bench.prefill_probe_cases()
    assert len(rec) == len(cases)
    label, O, I, T = cases[2]
    r = rec[f"{label} T={T}"]
    # library: 2 kernels of 0.5 us plus the 7 ns fill, per call
    assert r == {"decompress_us": round((1000 + 2) / 1e3, 2), "library_us": round((2 * 500 * n + 7) / n / 1e3, 2),
                 "fused_us": 2.0}
