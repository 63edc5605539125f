"""Host logic of bench.py's HBM-traffic figure: counter files in, bytes per call out.

The counters are rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE (KiB per dispatch);
each is scaled so that the calibration copy reads and writes exactly its size.
"""
import csv
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def write_counters(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_traffic_summary_scales_by_the_last_calibration_copy(tmp_path):
    bench = load_bench()
    calib_kib = 256 * 1024
    main = "void fathom::fused_main_kernel<true, 3, 16>(fathom::FusedArgs)"
    fetch = [("__amd_rocclr_copyBuffer", 2 * calib_kib),      # an earlier, unrelated large copy
             ("void fathom::fused_sample_kernel<true, 3>(fathom::FusedArgs)", 100.0),
             (main, 1000.0), (main, 3000.0),
             ("fathom::fused_rank_kernel(fathom::FusedArgs, int*, float*)", 50.0),
             ("__amd_rocclr_copyBuffer", 1.0),                # a small readback, not the calibration
             ("__amd_rocclr_copyBuffer", calib_kib / 2),      # the calibration copy: half counted
             ("__amd_rocclr_copyBuffer", 3.0)]
    write = [("__amd_rocclr_copyBuffer", 4 * calib_kib),
             ("void fathom::fused_sample_kernel<true, 3>(fathom::FusedArgs)", 1.0),
             (main, 10.0), (main, 30.0),
             ("fathom::fused_rank_kernel(fathom::FusedArgs, int*, float*)", 5.0),
             ("__amd_rocclr_copyBuffer", calib_kib)]
    fp, wp = tmp_path / "f.csv", tmp_path / "w.csv"
    write_counters(fp, "FETCH_SIZE", fetch)
    write_counters(wp, "WRITE_SIZE", write)
    t = bench.traffic_summary(str(fp), str(wp), 256)
    f, w = t["counters"]["FETCH_SIZE"], t["counters"]["WRITE_SIZE"]
    assert f["factor"] == pytest.approx(2.0) and w["factor"] == pytest.approx(1.0)
    # per kernel: the mean over its dispatches, in bytes, times the factor
    assert f["per_kernel_bytes"]["fused_main_kernel<true, 3, 16>"] == pytest.approx(2000.0 * 1024 * 2.0)
    assert f["per_kernel_bytes"]["fused_sample_kernel<true, 3>"] == pytest.approx(100.0 * 1024 * 2.0)
    assert w["per_kernel_bytes"]["fused_main_kernel<true, 3, 16>"] == pytest.approx(20.0 * 1024)
    expect = (100 + 2000 + 50) * 1024 * 2.0 + (1 + 20 + 5) * 1024 * 1.0
    assert t["bytes_per_call"] == pytest.approx(expect)
    assert t["source_sha256"] == bench.kernel_source_hash()


def test_measured_traffic_is_null_once_the_kernel_sources_change(tmp_path, monkeypatch):
    bench = load_bench()
    p = tmp_path / "t.json"
    monkeypatch.setattr(bench, "TRAFFIC_JSON", str(p))
    assert bench.measured_traffic() is None  # no file
    p.write_text(json.dumps({"bytes_per_call": 123.0, "source_sha256": bench.kernel_source_hash()}))
    assert bench.measured_traffic() == 123.0
    p.write_text(json.dumps({"bytes_per_call": 123.0, "source_sha256": "0" * 64}))
    assert bench.measured_traffic() is None


def test_sq_summary_means_per_kernel_and_valu_per_call(tmp_path):
    """SQ counters from several passes: per kernel of the fused call, the mean
    over its dispatches; VALU instructions per call = the sum over the call's
    kernels; other kernels ignored; the issue-side fraction uses 64 lanes per
    instruction against 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz."""
    bench = load_bench()
    main = "void fathom::fused_main_kernel<true, 3, 16>(fathom::FusedArgs)"
    rank = "fathom::fused_rank_kernel(fathom::FusedArgs, int*, float*)"
    a, b = tmp_path / "a.csv", tmp_path / "b.csv"
    write_counters(a, "SQ_INSTS_VALU", [(main, 1000.0), (main, 3000.0), (rank, 10.0), ("pack_kernel", 7.0)])
    with open(a, "a", newline="") as fh:
        w = csv.writer(fh)
        w.writerow([9, main, "SQ_WAVE_CYCLES", 400.0])
        w.writerow([10, main, "SQ_WAIT_ANY", 100.0])
    write_counters(b, "SQ_LDS_BANK_CONFLICT", [(main, 30.0)])
    with open(b, "a", newline="") as fh:
        csv.writer(fh).writerow([2, main, "SQ_LDS_IDX_ACTIVE", 120.0])
    t = bench.sq_summary([str(a), str(b)])
    assert t["per_kernel"]["fused_main_kernel<true, 3, 16>"]["SQ_INSTS_VALU"] == pytest.approx(2000.0)
    assert t["valu_insts_per_call"] == pytest.approx(2010.0)
    d = t["derived"]["fused_main_kernel<true, 3, 16>"]
    assert d["SQ_WAIT_ANY/SQ_WAVE_CYCLES"] == pytest.approx(0.25)
    assert d["SQ_LDS_BANK_CONFLICT/SQ_LDS_IDX_ACTIVE"] == pytest.approx(0.25)
    p = tmp_path / "sq.json"
    p.write_text(json.dumps(t))
    bench.SQ_JSON = str(p)
    iss = bench.issue_side(0.1)
    assert iss["frac"] == pytest.approx(2010.0 * 64 / 1e-4 / (256 * 4 * 16 * 2.4e9))
    p.write_text(json.dumps(dict(t, source_sha256="0" * 64)))
    assert bench.issue_side(0.1) is None
