"""bench.py on the GPU, run in this process with few steps: the JSON line
carries the fields its contract names (metric, value, roofline with the
clocks under load, the eager Torch comparison, the error report), and the
W8A8 and bf16 paths' errors against X W^T + b in binary64 on the FFN-up case
stay within what the recipe and the bf16 output rounding allow."""
from __future__ import annotations

import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu


def test_bench_json_line(capsys, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench

    print("bench.py --steps 3 --warmup 1 --pool 1 --no-cpu-baseline", flush=True)
    monkeypatch.setattr(sys, "argv", ["bench.py", "--steps", "3", "--warmup", "1", "--pool", "1",
                                      "--no-cpu-baseline"])
    capsys.readouterr()
    bench.main()
    line = capsys.readouterr().out.strip().splitlines()[-1]
    d = json.loads(line)
    assert d["metric"] == bench.METRIC and d["unit"] == "TOPS" and d["n_gpus"] == 1
    assert d["steps"] == 3 and d["warmup"] == 1 and d["higher_is_better"] is True
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["dtype"] == "int8"
    assert d["config"]["workload"].startswith("DiT FFN up-projection 4608x4096->16384")
    r = d["roofline"]
    assert r["bound"] == "mfma" and r["unit"] == "TOP/s" and r["peak"] == 5000.0
    assert r["ops_per_launch"] == 2 * 4608 * 4096 * 16384
    assert r["achieved"] == pytest.approx(r["ops_per_launch"] / r["avg_launch_us"] / 1e6, rel=1e-3)
    assert 0 < r["frac"] < 1
    p10, p50, p90 = r["launch_us_p10_p50_p90"]
    assert 0 < p10 <= p50 <= p90
    clk = r["clock"]
    if clk is not None:  # amdsmi present
        assert len(clk["mhz_per_xcd"]) == 8 and 100 < clk["mhz_mean"] <= 2400
        assert r["frac"] < clk["frac_at_measured_clock"] < 1
        pw = clk["power"]
        if pw.get("ppt_throttle_share") is not None:  # the metrics table's accumulators
            assert 0 <= pw["ppt_throttle_share"] <= 1 and pw["launches"] > 0
        if pw.get("avg_power_w") is not None:
            assert 50 < pw["avg_power_w"] < 2000 and pw["joules_per_launch"] > 0
            assert pw["tops_per_watt"] == pytest.approx(
                r["ops_per_launch"] / pw["joules_per_launch"] / 1e12, rel=2e-3)
            # joules per launch = average power x time per launch, near the
            # timed launches' own duration
            assert pw["joules_per_launch"] / pw["avg_power_w"] == pytest.approx(
                r["avg_launch_us"] * 1e-6, rel=0.25)
    e = d["eager_torch"]
    assert e["shape"] == [4608, 4096, 16384] and e["us"] > 0 and e["fused_us"] > 0
    assert e["mean_abs_diff_rel"] < 1e-3
    a = d["accuracy"]
    assert a["shape"] == [4608, 4096, 16384]
    # bf16 output rounding alone: at most half an ulp, 2^-8 relative; its rms
    # over many outputs is near 2^-8 / sqrt(3)
    assert a["bf16"]["rel_frobenius"] < 2.0 ** -8
    # per-token and per-channel 8-bit grids with outlier channels smoothed
    assert a["bf16"]["rel_frobenius"] < a["w8a8"]["rel_frobenius"] < 0.05
    assert d["cpu_baseline"] is None


def test_branch_streams_write_the_same_outputs():
    """The DiT block's two branches issued on two streams (bench.py
    --branch-streams) give every layer the same output bits as the one-stream
    step, with the adaLN-fused inputs included."""
    sys.path.insert(0, ROOT)
    import torch

    import bench
    from paper_2606_12280_amd import layer as L

    dev = torch.device("cuda:0")
    print("dit_block, one stream against two", flush=True)
    layers = bench.build_workload("dit_block", dev, 1)
    bench.modulate(layers, dev, 11)
    assert sum(lin.mod is not None for lin in layers) == 4
    bench.run_step(layers, 0, L.Workspace(dev))
    torch.cuda.synchronize()
    one = [lin.Y.clone() for lin in layers]
    for lin in layers:
        lin.Y.zero_()
    two = bench.BranchStreams(layers, dev)
    two.step(0)
    torch.cuda.synchronize()
    for lin, y in zip(layers, one):
        assert torch.equal(lin.Y.view(torch.int16), y.view(torch.int16)), lin.name


def test_power_table_entries():
    """bench.py --power-table: one entry per kernel of the FFN-up layer (the
    GEMM, the quant step, the adaLN step), each with its time, rate and, where
    the metrics table has them, the socket power figures (short windows)."""
    sys.path.insert(0, ROOT)
    import torch

    import bench

    dev = torch.device("cuda:0")
    print("power table, ffn_up, 1 s windows", flush=True)
    layers = bench.build_workload("ffn_up", dev, 1)
    table = bench.power_table(layers, dev, seconds=1.0, settle=0.2)
    if table is None:  # amdsmi absent
        pytest.skip("amdsmi not available")
    kinds = [e["kernel"].split()[0] for e in table]
    assert kinds == ["w8a8_linear", "w8a8_quant_act", "w8a8_adaln_quant_act"]
    for e in table:
        assert e["us_per_launch"] > 0 and e["launches"] > 0
        assert ("TOPS" in e) == (e["kernel"].startswith("w8a8_linear"))
        if e.get("avg_power_w") is not None:
            assert 50 < e["avg_power_w"] < 2000 and e["joules_per_launch"] > 0
        if e.get("ppt_throttle_share") is not None:
            assert 0 <= e["ppt_throttle_share"] <= 1
