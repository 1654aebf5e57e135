"""The benchmark's host-side logic on the CPU: spreading projections over
streams by work, the HBM-traffic summary built from rocprofv3 counter tables
(copy calibration, kernel-class attribution, the paired weight-gradient launch
counted as one class), and the refusal of more than one GPU."""
import csv
import json
import os
import subprocess
import sys
import types

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def proj(T, d_in, d_out, r):
    return types.SimpleNamespace(T=T, d_in=d_in, d_out=d_out, r=r)


def test_proj_work_cola_and_dense():
    p = proj(8, 3, 5, 2)
    assert bench.proj_work(p) == 8 * 2 * (3 + 5)
    assert bench.proj_work(p, dense=True) == 8 * 3 * 5
    g = object.__new__(bench.Group)
    g.m = [p, proj(8, 3, 7, 4)]
    assert bench.proj_work(g) == 8 * 2 * 8 + 8 * 4 * 10


def test_assign_streams_largest_first_least_loaded():
    # 10 -> s0, 7 -> s1, 6 -> s1 (7 < 10), 5 -> s0 (10 < 13), 1 -> s1 (13 < 15)
    works = [5, 10, 1, 7, 6]
    where = bench.assign_streams(works, 2)
    assert where == [0, 0, 1, 1, 1]
    loads = [sum(w for w, k in zip(works, where) if k == s) for s in range(2)]
    assert sorted(loads) == [14, 15]


def test_assign_streams_single_stream_and_ties():
    assert bench.assign_streams([3, 1, 2], 1) == [0, 0, 0]
    # equal work: stable order, first item on the caller's stream
    assert bench.assign_streams([4, 4, 4, 4], 2) == [0, 1, 0, 1]
    assert bench.assign_streams([], 3) == []


def test_assign_streams_balances_llama_block():
    """The seven projections of a LLaMA-1B-shaped block (d 2048, FFN 5461,
    rank d/4) on two streams: the two loads differ by at most the smallest
    projection's work."""
    d, f, r, T = 2048, 5461, 512, 4096
    shapes = [(d, d, r)] * 4 + [(d, f, r), (d, f, r), (f, d, r)]
    works = [bench.proj_work(proj(T, a, b, rr)) for a, b, rr in shapes]
    where = bench.assign_streams(works, 2)
    loads = [sum(w for w, k in zip(works, where) if k == s) for s in range(2)]
    assert abs(loads[0] - loads[1]) <= min(works)


def write_pmc(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, kib) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": kib})


def test_traffic_summary_attribution_and_calibration(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    gib_kib = bench.COPY_BYTES / 1024.0
    pair = "void gemm_pp_pair_kernel<64, 1, 1, 1, 4>(GemmArgs, GemmArgs, long) [clone .kd]"
    fwd_y = "void gemm_pp_persist_kernel<64, 0, 1, 0, 1>(GemmArgs) [clone .kd]"
    copy = "void at::native::elementwise_kernel<128, 4>(int, copy_functor) [clone .kd]"
    f = tmp_path / "fetch.csv"
    w = tmp_path / "write.csv"
    cf = tmp_path / "copy_fetch.csv"
    cw = tmp_path / "copy_write.csv"
    write_pmc(f, "FETCH_SIZE", [(pair, 100.0), (pair, 300.0), (fwd_y, 40.0), (copy, 5.0)])
    write_pmc(w, "WRITE_SIZE", [(pair, 10.0), (pair, 30.0), (fwd_y, 8.0)])
    # the copy of 1 GiB reads as 0.8 GiB fetched and 1 GiB written: factors 1.25 and 1
    write_pmc(cf, "FETCH_SIZE", [("small_copy_kernel", 1.0), (copy, 0.8 * gib_kib)])
    write_pmc(cw, "WRITE_SIZE", [(copy, gib_kib)])
    bench.traffic_summary(str(f), str(w), str(cf), str(cw))
    out = json.load(open(tmp_path / "profiles" / "traffic.json"))
    assert set(k for k in out if not k.startswith("_")) == {"bwd_da_db", "fwd_y"}
    p = out["bwd_da_db"]
    assert p["launches"] == 2
    assert p["fetch_bytes_per_launch"] == pytest.approx(200.0 * 1024 * 1.25)
    assert p["write_bytes_per_launch"] == pytest.approx(20.0 * 1024)
    assert p["bytes_per_launch"] == pytest.approx(200.0 * 1024 * 1.25 + 20.0 * 1024)
    assert out["fwd_y"]["bytes_per_launch"] == pytest.approx(40.0 * 1024 * 1.25 + 8.0 * 1024)
    assert p["source_sha256_16"] == "0123456789abcdef"
    # read back only while the kernel sources are unchanged
    assert bench.load_traffic("bwd_da_db") == pytest.approx(p["bytes_per_launch"])
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "fedcba9876543210")
    assert bench.load_traffic("bwd_da_db") is None


def test_traffic_summary_needs_copy_dispatch(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    empty = tmp_path / "e.csv"
    write_pmc(empty, "FETCH_SIZE", [("small_copy_kernel", 4.0)])
    with pytest.raises(SystemExit):
        bench.traffic_summary(str(empty), str(empty), str(empty), str(empty))


def test_more_than_one_gpu_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


# --------------------------------------------------------------------------
# the benchmark's flop formulas are the oracle's counted work (2 flops per
# multiply-add of every GEMM the oracle runs, Sec. 3.4)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (5, 12, 7, 3), (33, 40, 72, 8), (64, 24, 24, 24)])
def test_bench_flops_equal_oracle_mac_count(shape):
    import numpy as np
    import oracle
    T, d_in, d_out, r = shape
    g = np.random.Generator(np.random.PCG64(5))
    X = g.standard_normal((T, d_in))
    A = g.standard_normal((r, d_in))
    B = g.standard_normal((d_out, r))
    W = g.standard_normal((d_out, d_in))
    dY = g.standard_normal((T, d_out))
    oracle.reset_macs()
    Z, _, _ = oracle.cola_fwd(X, A, B)
    fwd = 2 * oracle.macs()
    oracle.cola_bwd(X, Z, A, B, dY)
    assert bench.algo_flops_cola(T, d_in, d_out, r) == 2 * oracle.macs()
    assert bench.algo_flops_cola_fwd(T, d_in, d_out, r) == fwd
    oracle.reset_macs()
    oracle.dense_fwd(X, W)
    oracle.dense_bwd(X, W, dY)
    assert bench.algo_flops_dense(T, d_in, d_out) == 2 * oracle.macs()


def test_traffic_summary_keeps_workload_sections(tmp_path, monkeypatch):
    """Counter readings of another workload go to their own section of
    traffic.json; a later headline summary replaces only the top level."""
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    gib_kib = bench.COPY_BYTES / 1024.0
    pair = "void gemm_pp_pair_kernel<64, 1, 1, 1, 4>(GemmArgs, GemmArgs, long) [clone .kd]"
    copy = "void at::native::elementwise_kernel<128, 4>(int, copy_functor) [clone .kd]"
    cf, cw = tmp_path / "cf.csv", tmp_path / "cw.csv"
    write_pmc(cf, "FETCH_SIZE", [(copy, 0.8 * gib_kib)])
    write_pmc(cw, "WRITE_SIZE", [(copy, gib_kib)])
    for wl, kib in ((2, 10.0), (4, 100.0), (3, 30.0)):
        f, w = tmp_path / f"f{wl}.csv", tmp_path / f"w{wl}.csv"
        write_pmc(f, "FETCH_SIZE", [(pair, kib)])
        write_pmc(w, "WRITE_SIZE", [(pair, 1.0)])
        bench.traffic_summary(str(f), str(w), str(cf), str(cw), workload=wl)
    out = json.load(open(tmp_path / "profiles" / "traffic.json"))
    assert out["bwd_da_db"]["fetch_bytes_per_launch"] == pytest.approx(100.0 * 1024 * 1.25)
    assert out["workload_2"]["bwd_da_db"]["fetch_bytes_per_launch"] == pytest.approx(10.0 * 1024 * 1.25)
    assert out["workload_3"]["bwd_da_db"]["fetch_bytes_per_launch"] == pytest.approx(30.0 * 1024 * 1.25)
    assert bench.load_traffic("bwd_da_db", 2) == pytest.approx(10.0 * 1024 * 1.25 + 1024)
    assert bench.load_traffic("bwd_da_db") == pytest.approx(100.0 * 1024 * 1.25 + 1024)
    assert bench.load_traffic("bwd_da_db", 5) is None
    # a new headline reading keeps the other workloads' sections
    f, w = tmp_path / "f4b.csv", tmp_path / "w4b.csv"
    write_pmc(f, "FETCH_SIZE", [(pair, 50.0)])
    write_pmc(w, "WRITE_SIZE", [(pair, 1.0)])
    bench.traffic_summary(str(f), str(w), str(cf), str(cw))
    out = json.load(open(tmp_path / "profiles" / "traffic.json"))
    assert out["bwd_da_db"]["fetch_bytes_per_launch"] == pytest.approx(50.0 * 1024 * 1.25)
    assert set(k for k in out if k.startswith("workload_")) == {"workload_2", "workload_3"}


def test_box_relative_only_for_hbm_bound_records():
    recs = {"2": {"roofline": {"bound": "hbm", "achieved": 4000.0, "avg_us": 50.0, "traffic": 250e6}},
            "5": {"roofline": {"bound": "mfma", "achieved": 1200.0, "avg_us": 300.0}},
            "1": {}}
    bench.box_relative(recs, {"read_gbs": 6000.0, "copy_gbs": 5000.0})
    v = recs["2"]["roofline"]["vs_box"]
    assert v["algorithmic"] == {"gbs": 4000.0, "of_read_only": pytest.approx(0.667, abs=1e-3),
                                "of_copy": 0.8}
    assert v["measured_traffic"]["gbs"] == pytest.approx(5000.0)
    assert v["measured_traffic"]["of_copy"] == 1.0
    assert "vs_box" not in recs["5"]["roofline"]
    bench.box_relative(recs, None)      # no ceilings measured: nothing added, no error


def test_roofline_at_sampled_clock():
    r = {"bound": "mfma", "achieved": 1000.0, "peak": 2516.6}
    bench.at_clock(r, 1800)
    assert r["peak_at_sclk"] == pytest.approx(2516.6 * 0.75, abs=0.1)
    assert r["frac_at_sclk"] == pytest.approx(1000.0 / (2516.6 * 0.75), abs=1e-4)
    h = {"bound": "hbm", "achieved": 4000.0, "peak": 8000.0}
    bench.at_clock(h, 1800)
    assert "frac_at_sclk" not in h
    m = {"bound": "mfma", "achieved": 1000.0, "peak": 2516.6}
    bench.at_clock(m, None)
    assert "frac_at_sclk" not in m


def test_power_sampler_reads_sensor_files(tmp_path):
    """Board power from hwmon power1_input (microwatts), summed over cards;
    median, maximum and the cap from power1_cap."""
    d = tmp_path / "hwmon0"
    d.mkdir()
    (d / "power1_input").write_text("1200000000\n")
    (d / "power1_cap").write_text("1400000000\n")
    s = bench.SclkSampler()
    s.files, s.pfiles = [], [str(d / "power1_input")]
    assert s.read_power() == pytest.approx(1200.0)
    assert s.power() is None
    s.pvals = [1100.0, 1300.0, 1200.0]
    assert s.power() == {"median": 1200.0, "max": 1300.0, "cap": 1400.0, "samples": 3}
    s.pfiles = [str(tmp_path / "missing")]
    assert s.read_power() is None
