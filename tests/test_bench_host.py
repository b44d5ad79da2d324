"""Host-side logic of bench.py, on the CPU: the one-GPU refusal, the dispatch keys that
join a plan with rocprofv3's kernel names (the measured-traffic lookup depends on
them), and the scaling of HBM counters by a plain copy."""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench
import paper_2509_18344_amd as ss

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr, (r.returncode, r.stderr)


def _kernel_name(plan, bits, group):
    """The demangled name rocprofv3 reports for the kernel a plan launches."""
    if plan["path"] == ss.SUBSPEC_PATH_GEMV:
        t = (bits, group, plan["rows"], plan["tiles_per_wave"], plan["chunk_blocks"], plan["waves"], 2)
        return "void subspec::k_qgemv<%s>(subspec::QArgs)" % ", ".join(map(str, t))
    if plan["mfma_rows"] == 32:
        t = (bits, group, plan["rows"] // 32, plan["tiles_per_wave"] // 2, plan["ring_chunks"], plan["waves"],
             plan["teams"])
        return "void subspec::qmma::k_qmma<%s>(subspec::QArgs)" % ", ".join(map(str, t))
    t = (bits, group, plan["rows"] // 16, plan["tiles_per_wave"], plan["chunk_blocks"], plan["waves"], 2)
    return "void subspec::k_qgemm_mfma<%s>(subspec::QArgs)" % ", ".join(map(str, t))


@pytest.mark.parametrize("M,N,K,bits,group", [(1, 7168, 5120, 3, 128), (16, 55296, 5120, 3, 128),
                                              (64, 7168, 5120, 3, 128), (128, 5120, 5120, 3, 128),
                                              (64, 55296, 5120, 3, 128), (128, 5120, 27648, 3, 128),
                                              (48, 3584, 18944, 4, 128), (128, 55296, 5120, 2, 64)])
def test_plan_key_matches_the_traced_kernel(M, N, K, bits, group):
    """A launch's key from its plan equals the key built from the kernel name and the
    whole grid (both dimensions, in work-items) that a trace or counter file gives."""
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    wg = plan["waves"] * 64
    grid_items = plan["grid"] * plan["row_blocks"] * wg
    assert bench.plan_key(plan, bits, group) == bench.library_key(_kernel_name(plan, bits, group), grid_items, wg)


def test_library_key_ignores_other_kernels():
    assert bench.library_key("void at::native::vectorized_elementwise_kernel<4>(int)", 1024, 256) is None


def _counter_csv(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Grid_Size", "Workgroup_Size",
                                          "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_counters_are_scaled_by_the_copy(tmp_path, monkeypatch):
    """FETCH_SIZE and WRITE_SIZE (KiB per dispatch, summed over the counter's
    instances) become bytes with the factors a copy of known size gives."""
    out = tmp_path / "traffic.json"
    fam = dict(bench.FAMILIES["qlinear"], json=str(out))
    monkeypatch.setitem(bench.FAMILIES, "qlinear", fam)
    name = "void subspec::qmma::k_qmma<3, 128, 4, 1, 4, 8, 1>(subspec::QArgs)"
    grid, wg = 110592, 512
    # two dispatches of one kernel, each counter reported by two instances
    fetch = [dict(Dispatch_Id=d, Kernel_Name=name, Grid_Size=grid, Workgroup_Size=wg, Counter_Name="FETCH_SIZE",
                  Counter_Value=v) for d, v in ((1, 30000.0), (1, 40000.0), (2, 35000.0), (2, 35000.0))]
    write = [dict(Dispatch_Id=d, Kernel_Name=name, Grid_Size=grid, Workgroup_Size=wg, Counter_Name="WRITE_SIZE",
                  Counter_Value=v) for d, v in ((1, 100.0), (1, 200.0), (2, 300.0), (2, 0.0))]
    copy = "void at::native::copy_kernel(int)"
    cfetch = [dict(Dispatch_Id=1, Kernel_Name=copy, Grid_Size=4096, Workgroup_Size=256, Counter_Name="FETCH_SIZE",
                   Counter_Value=512.0)]
    cwrite = [dict(Dispatch_Id=1, Kernel_Name=copy, Grid_Size=4096, Workgroup_Size=256, Counter_Name="WRITE_SIZE",
                   Counter_Value=1024.0)]
    for d, rows in (("f", fetch), ("w", write), ("cf", cfetch), ("cw", cwrite)):
        _counter_csv(tmp_path / d, rows)
    bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw"),
                        calib_bytes=1 << 20)
    res = json.loads(out.read_text())
    assert res["calibration"]["fetch_scale"] == 2.0 and res["calibration"]["write_scale"] == 1.0
    key = bench.library_key(name, grid, wg)
    e = res["kernels"][key]
    assert e["dispatches"] == 2 and e["fetch_kib_raw"] == 70000.0 and e["write_kib_raw"] == 300.0
    assert e["hbm_bytes_per_launch"] == int(round(70000.0 * 1024 * 2 + 300.0 * 1024))
    assert res["kernel_source_sha256_16"] == bench.kernel_source_hash("qlinear")
