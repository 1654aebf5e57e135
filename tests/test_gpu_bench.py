"""bench.py on the GPU: the one JSON line of a short run on the
fp32 single layer and on the 60M-shaped block (CoLA only), in process (no
second GPU process): the contract's fields, the headline value equal to the
step's algorithmic flops over its time (recomputed here from the workload's
shapes, 6 T r (d_in + d_out) per projection), a dominant kernel whose
roofline figures agree with each other, and the oracle baseline's fields."""
import json
import sys

import pytest

import bench
from paper_2502_10940_amd import inputs as I

CONTRACT = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
            "vs_baseline", "dtype", "data", "config")


@pytest.mark.gpu
@pytest.mark.parametrize("workload,extra", [(1, []), (2, ["--only", "cola"])], ids=["single_f32", "60m_bf16"])
def test_bench_line(workload, extra, capsys, monkeypatch):
    argv = ["bench.py", "--workload", str(workload), "--steps", "3", "--warmup", "1", "--no-block", "--no-workloads",
            "--cpu-tokens", "64"] + extra
    monkeypatch.setattr(sys, "argv", argv)
    print(f"bench line: workload {workload} {' '.join(extra)}", flush=True)
    bench.main()
    lines = [l for l in capsys.readouterr().out.splitlines() if l.startswith("{")]
    assert lines, "no JSON line"
    d = json.loads(lines[-1])
    for k in CONTRACT:
        assert k in d, k
    w = I.WORKLOADS[workload]
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "TFLOP/s" and d["higher_is_better"] is True and d["data"] == "synthetic"
    assert d["dtype"] == w["dtype"] and d["config"]["workload"] == w["name"]
    assert d["vs_baseline"] is None
    # the value: algorithmic flops of one step over its measured time
    flops = sum(6.0 * w["T"] * w["r"] * (din + dout) for _, _, din, dout in I.projections(workload))
    assert d["ms_per_step"] > 0
    # (value is rounded to 0.01 TFLOP/s and ms_per_step to 1e-4 ms)
    assert d["value"] == pytest.approx(flops / (d["ms_per_step"] * 1e9), rel=2e-3, abs=0.006)
    # the dominant kernel against its roofline
    rl = d["roofline"]
    assert rl["bound"] in ("mfma", "hbm") and rl["kernel"] in d["kernels"]
    # (achieved is rounded to 0.01 TFLOP/s or 0.1 GB/s, frac to 1e-4)
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-3, abs=1e-4)
    kd = d["kernels"][rl["kernel"]]
    if rl["bound"] == "mfma":
        assert rl["achieved"] == pytest.approx(kd["flops_per_launch"] / (kd["avg_us"] * 1e6), rel=1e-2, abs=0.006)
    else:
        assert rl["achieved"] == pytest.approx(kd["bytes_per_launch"] / (kd["avg_us"] * 1e3), rel=1e-2, abs=0.06)
    # every kernel class's flops per launch add up to the step's flops
    per_step = sum(k["flops_per_launch"] * k["launches"] for k in d["kernels"].values()) / 3
    assert per_step == pytest.approx(flops, rel=1e-9)
    # the oracle baseline, timed on the host
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0
