"""Host-only checks of bench.py's profile summaries (no GPU): the per-call HBM traffic
attribution from rocprofv3 FETCH_SIZE / WRITE_SIZE counter files, on synthetic files
in rocprofv3's CSV layout."""
import csv
import json
import os

import bench

FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def write_run(path, counter, dispatches):
    """dispatches: [(kernel name, value in KiB)], one counter instance each (the value is
    split over two instances to check that instances are summed)."""
    os.makedirs(path)
    with open(os.path.join(path, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for i, (name, v) in enumerate(dispatches):
            for half in (0.25 * v, 0.75 * v):
                row = {k: 0 for k in FIELDS}
                row.update({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                            "Counter_Value": half})
                w.writerow(row)


def test_traffic_attribution(tmp_path):
    wl = bench.case_name(1, 0, 1)  # the 1k x 1k INT2 GEMV
    head_fused = "void lutgemm::lut_fused_gemv_kernel<2, 2, 2, 1, 16, true>(lutgemm::LutParams, int)"
    split = "void lutgemm::lut_gemv_split_kernel<2, 4, false, false, 4>(lutgemm::LutParams, int)"
    fin = "void lutgemm::lut_finalize_kernel<false, 16, 256>(lutgemm::LutParams, int, int, long)"
    fused = "void lutgemm::lut_fused_split_kernel<2, 4, 4>(lutgemm::LutParams, int)"
    copy = bench.COPY_KERNEL
    # FETCH_SIZE reads half the bytes (scale 2), WRITE_SIZE all of them (scale 1)
    fetch = [(head_fused, 100.0), (head_fused, 100.0), (copy, 131072.0),
             ("lutgemm::precompute_kernel", 5.0), (split, 50.0), (fin, 10.0), (split, 50.0), (fin, 10.0),
             (fused, 60.0), (fin, 10.0)]
    write = [(head_fused, 1.0), (head_fused, 1.0), (copy, 262144.0),
             ("lutgemm::precompute_kernel", 5.0), (split, 8.0), (fin, 2.0), (split, 8.0), (fin, 2.0),
             (fused, 8.0), (fin, 2.0)]
    write_run(str(tmp_path / f"fetch_{wl}"), "FETCH_SIZE", fetch)
    write_run(str(tmp_path / f"write_{wl}"), "WRITE_SIZE", write)
    text = bench.summarize_traffic([str(tmp_path / f"fetch_{wl}"), str(tmp_path / f"write_{wl}")], "cmd")
    recs = {(r["workload"], r["timed_kernel"]): r for r in
            (json.loads(line) for line in text.splitlines() if line.startswith("{"))}
    head = bench.case_name(2, 0, 1)
    assert recs[(head, "fused")]["read_bytes"] == 200 * 1024 and recs[(head, "fused")]["write_bytes"] == 1024
    mp = recs[(wl, "mpgemm")]
    assert mp["calls"] == 2
    assert mp["read_bytes"] == 2 * (50 + 10) * 1024 and mp["write_bytes"] == (8 + 2) * 1024
    assert sorted(mp["kernels"]) == sorted([split, fin])
    fu = recs[(wl, "fused")]
    assert fu["calls"] == 1 and fu["read_bytes"] == 2 * 70 * 1024 and fu["write_bytes"] == 10 * 1024
    assert mp["bytes_per_launch"] == mp["read_bytes"] + mp["write_bytes"]
    assert mp["kernel_source_sha256_16"] == bench.kernel_source_hash("mpgemm")
