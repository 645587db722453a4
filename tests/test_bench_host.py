"""Host logic of bench.py: the traffic summariser and the flow kernel names
(no GPU; synthetic rocprofv3 counter files)."""
from __future__ import annotations

import csv
import os

import pytest

import bench
from paper_2609_35115_amd import synth

FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _counters(d, counter, rows):
    """rows: (dispatch id, kernel, grid size, values per XCD)."""
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for i, name, grid, vals in rows:
            for v in vals:
                w.writerow({k: 0 for k in FIELDS} | {"Dispatch_Id": i, "Kernel_Name": f"void {name}(P)",
                                                     "Grid_Size": grid, "Counter_Name": counter,
                                                     "Counter_Value": v})


def _summary(path):
    return {k.strip(): v.strip() for k, v in (l.split(":", 1) for l in open(path) if ":" in l and l[0] != "#")}


@pytest.mark.parametrize("workload,want_fetch", [("flow_real_bf16_b128", 30.0), ("real_bf16_b128_n25", 20.0)])
def test_traffic_summary(tmp_path, workload, want_fetch):
    """Values of one dispatch are summed over its rows (XCDs); a flow workload
    averages only the dispatches of the last one's grid size (the timed
    calls), a vocoder workload every dispatch of the kernel."""
    k, other = "dcf::attn_kernel<true, 4, 8>", "dcf::euler_kernel<true>"
    rows = [(1, k, 100, [5.0, 5.0]), (2, k, 100, [10.0]), (3, other, 4000, [999.0]),
            (4, k, 4000, [10.0, 20.0]), (5, k, 4000, [30.0])]
    _counters(tmp_path / "f", "FETCH_SIZE", rows)
    _counters(tmp_path / "w", "WRITE_SIZE", [(i, n, g, [1.0]) for i, n, g, _ in rows])
    out = tmp_path / "traffic.txt"
    bench.summarize_traffic(str(tmp_path / "f"), str(tmp_path / "w"), workload, k, str(out), "cmd")
    s = _summary(out)
    assert float(s["fetch_kib_per_dispatch"]) == pytest.approx(want_fetch)
    assert float(s["write_kib_per_dispatch"]) == pytest.approx(1.0)
    want = (want_fetch * bench.FETCH_SCALE + 1.0 * bench.WRITE_SCALE) * 1024.0
    assert float(s["hbm_bytes_per_launch"]) == pytest.approx(want)
    assert s["dispatches"].startswith("2 / 2" if workload.startswith("flow_") else "4 / 4")
    # the run's other kernels are recorded too, and found by traffic_from_profiles
    want_other = (999.0 * bench.FETCH_SCALE + 1.0 * bench.WRITE_SCALE) * 1024.0
    line = [x for x in out.read_text().splitlines() if x.startswith(f"hbm_bytes_per_launch[{other}]:")]
    assert len(line) == 1 and float(line[0].rsplit(":", 1)[1]) == pytest.approx(want_other)


def test_flow_kernel_names_follow_the_launch_rules():
    a = synth.REAL_FLOW_ARCH
    name = bench.flow_kernel_name
    # batch 1: 112 rows, skinny; LayerNorm operands 8 waves x 2 column blocks, K >= 1024 plain 8 waves
    assert name("gemm:qkv", "bf16", 112, arch=a) == "dcf::skinny_kernel<true, 1, true, 8, 2, 1>"
    assert name("gemm:fc2", "bf16", 112, arch=a) == "dcf::skinny_kernel<true, 2, false, 8, 1, 1>"
    assert name("gemm:o", "f32", 112, arch=a) == "dcf::skinny_kernel<false, 2, false, 4, 1, 1>"
    # one head: K = 64 keeps the 4-wave LayerNorm shape
    one = dict(synth.TINY_FLOW_ARCH, dim=64, heads=1)
    assert name("gemm:fc1", "bf16", 44, arch=one) == "dcf::skinny_kernel<true, 3, true, 4, 2, 1>"
    # batch 16 (1,792 rows): tiers by the number of 64 x 64 tiles
    assert name("gemm:fc1", "bf16", 1792, arch=a) == "dcf::gemm_kernel<true, 3, 4, 2>"   # 896 tiles
    assert name("gemm:o", "bf16", 1792, arch=a) == "dcf::gemm_kernel<true, 2, 1, 1>"     # 224 tiles
    assert name("gemm:fc1", "bf16", 14336, arch=a) == "dcf::gemm_kernel<true, 3, 4, 4>"  # 7,168 tiles
    # attention: the wide shape from 64 blocks of 64 queries
    assert name("attn", "bf16", 112, attn_blocks=16) == "dcf::attn_kernel<true, 1, 4>"
    assert name("attn", "bf16", 1792, attn_blocks=256) == "dcf::attn_kernel<true, 4, 8>"
