"""bench.py's output contract: one JSON line with the fields a driver reads,
`--gpus N` with N > 1 refused before any GPU work, and the roofline and
CPU-baseline blocks consistent with themselves."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, timeout):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args, cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused():
    p = _run(["--gpus", "2"], timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


@pytest.mark.gpu
def test_bench_json_line_fields():
    p = _run(["--layer", "cfg1_tiny_c3_32_3x3", "--steps", "3", "--warmup", "2", "--no-extras"], timeout=300)
    assert p.returncode == 0, p.stderr[-2000:]
    lines = [l for l in p.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, "exactly one JSON line"
    r = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in r, key
    assert r["n_gpus"] == 1 and r["steps"] == 3 and r["warmup"] == 2
    assert r["value"] > 0 and r["ms_per_step"] > 0 and r["higher_is_better"] is True
    assert r["unit"] == "TFLOP/s" and r["data"] == "synthetic"
    assert "cfg1_tiny_c3_32_3x3" in r["config"]["workload"]
    rl = r["roofline"]
    assert rl["bound"] in ("hbm", "mfma", "alu") and rl["unit"] in ("GB/s", "TFLOP/s")
    assert rl["peak"] == 157.3 and rl["achieved"] > 0
    assert abs(rl["frac"] - rl["achieved"] / rl["peak"]) < 1e-3
    assert rl["traffic"] is None   # counters are recorded for the benchmark workload only
    r16 = r["roofline_f16"]
    assert r16["bound"] == "mfma" and r16["peak"] == 2516.6 and r16["achieved"] > 0
    assert abs(r16["frac"] - r16["achieved"] / r16["peak"]) < 1e-3
    assert 0 < r16["frac_attainable"] and r16["attainable"] <= 2516.6
    # value: conv-only FLOPs of both precisions over their summed conv time
    co = r["conv_only"]
    t = co["f32"]["conv_ms_per_step"] + co["f16"]["conv_ms_per_step"]
    assert abs(r["value"] - (co["f32"]["GFLOP_per_step"] + co["f16"]["GFLOP_per_step"]) / t) < 2e-2 * r["value"]
    (lay,) = r["layers"]
    assert lay["f32"]["kernel"].startswith("conv_fp32_") and lay["f16"]["kernel"].startswith("conv_fp16_")
    ws = r["workspace"]["cfg1_tiny_c3_32_3x3"]
    for dt in ("f32", "f16"):
        assert ws[dt]["peak_bytes_im2win"] > 0 and ws[dt]["peak_bytes_im2col"] > 0
    cb = r["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    assert cb["single_thread"]["value"] > 0
