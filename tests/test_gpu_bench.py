"""bench.py's one JSON line, from a short run on the GPU: every field the line
promises is there, typed and consistent with the others."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.gpu
def test_bench_prints_one_complete_json_line(monkeypatch, capsys):
    print("bench: resnet50, 3 steps, headline only (in this process)", flush=True)
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import bench

    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "resnet50", "--steps", "3", "--warmup", "1",
                                      "--no-per-config",
                                      "--no-ablation", "--no-broadcast", "--cpu-seconds", "0.5"])
    capsys.readouterr()
    bench.main()
    lines = [line for line in capsys.readouterr().out.splitlines() if line.strip()]
    assert len(lines) == 1
    out = json.loads(lines[0])
    assert out["metric"] and out["unit"] == "GB/s" and out["n_gpus"] == 1
    assert out["steps"] == 3 and out["warmup"] == 1 and out["higher_is_better"] is True
    assert out["scaling"] == "weak" and out["vs_baseline"] is None and out["data"] == "synthetic"
    assert out["dtype"] == "f32" and out["config"]["workload"] == "resnet50"
    assert out["config"]["fusion_buffer_mode"] == "ring_on_tensors" and out["fusion_buffer_modes"] == {}
    # value is one rank's binary32 gradient bytes over the step time
    rank_bytes = 4 * 25_557_032
    assert out["value"] == pytest.approx(rank_bytes / (out["ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    roof = out["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert 0 < roof["achieved"] < roof["peak"]
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], abs=1e-3)
    assert roof["traffic"] is None or roof["traffic"] > 0
    per_launch = roof["algorithmic_bytes_per_step"] / roof["launches_per_step"]
    assert roof["achieved"] == pytest.approx(per_launch / (roof["avg_launch_us"] * 1e-6) / 1e9, rel=2e-3)
    ring = out["ring_roofline"]
    assert ring["bound"] == "hbm" and ring["peak"] == 8000.0 and 0 < ring["achieved"] < ring["peak"]
    assert set(ring["kernels"]) == {"rs_step_f32", "rs_ag_step_f32", "ag_step_f32"}
    assert ring["achieved"] == pytest.approx(
        ring["algorithmic_bytes_per_step"] / (ring["kernel_ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "GB/s" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert cpu["sample"]
