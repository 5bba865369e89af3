"""Host-side pieces of bench.py that turn profiler output into the committed
summaries and the bench line's per-tier bytes: CSV summaries per kernel and
launch shape, the per-tier and traffic profiles, the tier lookup by kernel
source and modulus.  Synthetic rocprofv3-style CSVs stand in for a run."""
import csv
import hashlib
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

COUNTER_FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id",
                  "Thread_Id", "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size",
                  "LDS_Block_Size", "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count",
                  "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp",
                  "End_Timestamp"]


def write_counters(path, rows):
    """rows: (dispatch id, kernel name, grid, {counter: value})"""
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=COUNTER_FIELDS)
        wr.writeheader()
        for d, name, grid, counters in rows:
            for c, v in counters.items():
                wr.writerow({"Dispatch_Id": d, "Kernel_Name": name, "Grid_Size": grid,
                             "Counter_Name": c, "Counter_Value": v})


def test_summarize_pmc_means_per_kernel_and_grid(tmp_path):
    name = "void (anonymous namespace)::gemv_kernel<1, 1, 8, 1>((anonymous namespace)::P)"
    write_counters(str(tmp_path), [
        (1, name, 1024, {"A": 10.0, "B": 1.0}),
        (2, name, 1024, {"A": 30.0, "B": 3.0}),
        (3, name, 2048, {"A": 5.0}),
        (4, "__amd_rocclr_copyBuffer", 512, {"A": 7.0})])
    s = bench.summarize_pmc(str(tmp_path))
    assert s["gemv_kernel<1, 1, 8, 1> grid=1024"] == {"dispatches": 2,
                                                      "per_dispatch": {"A": 20.0, "B": 2.0}}
    assert s["gemv_kernel<1, 1, 8, 1> grid=2048"]["per_dispatch"] == {"A": 5.0}
    assert s["__amd_rocclr_copyBuffer grid=512"]["dispatches"] == 1


def test_summarize_trace_tables(tmp_path):
    fields = ["Kernel_Name", "Grid_Size_X", "Start_Timestamp", "End_Timestamp"]
    with open(tmp_path / "run_kernel_trace.csv", "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=fields)
        wr.writeheader()
        for i, (name, grid, us) in enumerate([("void (anonymous namespace)::attn_merge(P)", 64, 4),
                                              ("void (anonymous namespace)::attn_merge(P)", 64, 6),
                                              ("at::native::fill(int)", 8, 100)]):
            wr.writerow({"Kernel_Name": name, "Grid_Size_X": grid,
                         "Start_Timestamp": 1000 * i * 1000,
                         "End_Timestamp": 1000 * i * 1000 + us * 1000})
    md = bench.summarize_trace(str(tmp_path))
    lines = md.splitlines()
    assert "| `attn_merge` | 2 | 5.00 | 4.00 | 6.00 | 0.01 |" in lines
    # torch's own kernels stay out of the per-shape table
    shape_rows = lines[lines.index("| kernel | grid (threads) | dispatches | median us | "
                                   "mean us | total ms |"):]
    assert any(r.startswith("| `attn_merge` | 64 | 2 | 5.00 |") for r in shape_rows)
    assert not any("fill" in r for r in shape_rows)


def test_tier_profile_and_lookup(tmp_path, monkeypatch):
    d = tmp_path / "tiers"
    gemv = "void (anonymous namespace)::gemv_kernel<1, 1, 8, 1>(P)"
    write_counters(str(d / "chain"), [
        (1, gemv, 100, {"TCC_EA0_RDREQ_DRAM_32B": 1000.0, "TCC_EA0_RDREQ_IO_32B": 10.0}),
        (2, gemv, 200, {"TCC_EA0_RDREQ_DRAM_32B": 3000.0, "TCC_EA0_RDREQ_IO_32B": 0.0}),
        (3, "stream_read(char const*)", 300, {"TCC_EA0_RDREQ_DRAM_32B": 9e9})])
    (d / "chain.json").write_text(json.dumps({"part": "chain", "modulus": 126,
                                              "weight_hbm_bytes": 120000,
                                              "weight_host_bytes": 320}))
    out = tmp_path / "out"
    out.mkdir()
    bench.write_tier_profile(str(d), str(out))
    prof = json.loads((out / "tier_counters.json").read_text())["chain"]
    assert prof["hbm_bytes"] == 4000 * 32 and prof["host_bytes"] == 320
    assert prof["modulus"] == 126 and prof["host_over_placement"] == 1.0
    src = open(os.path.join(ROOT, "paper_2609_13592_amd", "csrc", "gemv.hip"), "rb").read()
    assert prof["source_sha256"] == hashlib.sha256(src).hexdigest()
    # the bench line's lookup: counters at the same modulus, the counters'
    # ratio to the placement at another, placement bytes without counters
    monkeypatch.setattr(bench, "tier_counter_entry", lambda part: prof)
    same = bench.per_tier("chain", 1.0, 120000, 320, 126)
    assert (same["hbm_bytes"], same["host_bytes"]) == (128000, 320)
    other = bench.per_tier("chain", 1.0, 60000, 640, 127)
    assert other["hbm_bytes"] == int(60000 * prof["hbm_over_placement"])
    assert other["host_bytes"] == 640
    monkeypatch.setattr(bench, "tier_counter_entry", lambda part: None)
    bare = bench.per_tier("chain", 2.0, 1000, 10, 126)
    assert bare["bytes_from"] == "placement" and bare["hbm_gbps"] == round(1000 / 2e-3 / 1e9, 1)


def test_traffic_profile_scales_by_references(tmp_path):
    gemv = "void (anonymous namespace)::gemv_kernel<1, 1, 8, 1>(P)"
    fetch_rows = [(1, "(anonymous namespace)::stream_read(char const*)", 524288,
                   {"FETCH_SIZE": 2 * 1024 * 1024.0})]          # 4 GiB reads as 2 GiB
    write_rows = [(1, "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor"
                      "<unsigned char> >(int)", 999, {"WRITE_SIZE": 1024 * 1024.0})]
    did = 10
    for g, _ in bench.CHAIN_GRIDS.values():
        fetch_rows.append((did, gemv, g, {"FETCH_SIZE": 100.0}))
        write_rows.append((did, gemv, g, {"WRITE_SIZE": 2.0}))
        did += 1
    for g in (777, 778):                                            # the head, two legs
        fetch_rows.append((did, gemv, g, {"FETCH_SIZE": 1000.0}))
        write_rows.append((did, gemv, g, {"WRITE_SIZE": 4.0}))
        did += 1
    fetch_rows.append((did, "attn_partition<4>(P)", 5, {"FETCH_SIZE": 50.0}))
    write_rows.append((did, "attn_partition<4>(P)", 5, {"WRITE_SIZE": 6.0}))
    write_counters(str(tmp_path / "f"), fetch_rows)
    write_counters(str(tmp_path / "w"), write_rows)
    out = tmp_path / "out"
    out.mkdir()
    bench.write_traffic_profile(f"{tmp_path / 'f'},{tmp_path / 'w'}", str(out))
    prof = json.loads((out / "traffic_counters.json").read_text())
    assert prof["fetch_scale"] == 2.0 and prof["write_scale"] == 1.0
    launches = sum(n for _, n in bench.CHAIN_GRIDS.values()) + 1
    assert prof["gemv"]["launches_per_step"] == launches
    fetch = (launches - 1) * 100 * 1024 * 2 + 1000 * 1024 * 2
    write = (launches - 1) * 2 * 1024 + 4 * 1024
    assert prof["gemv"]["traffic_bytes_per_launch"] == int((fetch + write) / launches)
    assert prof["attn_partition"]["traffic_bytes_per_launch"] == 50 * 1024 * 2 + 6 * 1024


def test_host_topology_keys():
    topo = bench.host_topology()
    assert topo["logical_cpus"] >= 1
    assert "sockets" in topo or "model" in topo or len(topo) >= 1


def test_more_gpus_refused():
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def _cap_out(points_by_layout, modes):
    out = {"hbm_stream_modes": {k: {"us": v} for k, v in modes.items()}}
    for tag, (ref_us, spread, pts) in points_by_layout.items():
        out[tag] = {"hbm_only_us": ref_us, "hbm_only_spread": spread,
                    "points": [{"host_share": f, "host_workgroups": h, "us": us,
                                "speedup_vs_hbm_only": round(ref_us / us, 4)}
                               for f, h, us in pts]}
    return out


def test_cap_optimum_against_fastest_stream():
    """A layout that beats its own slow all-HBM reference but not the fastest
    all-HBM stream of another layout yields "no host page"; a point that beats
    the fastest stream by more than its layout's spread is the optimum."""
    modes = {"static": 316.0, "one_per_cu": 292.0}
    out = _cap_out({"concurrent_queue": (348.0, 0.002, [(1 / 130, 16, 343.0)]),
                    "concurrent_one_per_cu": (292.5, 0.003, [(1 / 1024, 8, 294.0)])}, modes)
    opt = bench.cap_measured_optimum(out)
    assert out["fastest_hbm_only_us"] == 292.0
    assert opt["host_share"] == 0.0 and opt["modulus"] is None and opt["speedup_vs_hbm_only"] == 1.0
    assert opt["best_host_point"]["layout"] == "concurrent_one_per_cu"
    q = out["concurrent_queue"]["points"][0]
    assert q["speedup_vs_hbm_only"] > 1.0 > q["speedup_vs_fastest_hbm_only"]
    # a real gain over the fastest stream, above the 0.3 % spread
    out = _cap_out({"concurrent_one_per_cu": (292.5, 0.003, [(1 / 130, 8, 289.0),
                                                             (1 / 256, 8, 291.5)])}, modes)
    opt = bench.cap_measured_optimum(out)
    assert opt["host_share"] == 1 / 130 and opt["modulus"] == 130 and opt["host_workgroups"] == 8
    assert opt["speedup_vs_hbm_only"] == round(292.0 / 289.0, 4)
    # within the spread: no gain
    out = _cap_out({"concurrent_one_per_cu": (292.5, 0.003, [(1 / 130, 8, 291.5)])}, modes)
    assert bench.cap_measured_optimum(out)["host_share"] == 0.0
