"""bench.py's output contract: the one-GPU refusal (CPU) and the fields of its
JSON line on a short run (GPU)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      (["--gpus", "1"], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    """Several GPUs (by flag or by a launcher's WORLD_SIZE) exit with status 2
    and a message, before anything touches a GPU or prints a JSON line."""
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, BENCH, *argv], cwd=ROOT, env=e, capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2, (r.returncode, r.stdout, r.stderr)
    assert r.stdout == ""
    assert "one GPU" in r.stderr


@pytest.mark.gpu
@pytest.mark.timeout(600)
def test_bench_json_line():
    """A short bench run (the timed loop, the per-phase launches, the copy
    reference and a small oracle sample) prints exactly one JSON line whose
    figures agree with each other."""
    cmd = [sys.executable, "-u", BENCH, "--steps", "20", "--warmup", "3", "--no-cold",
           "--no-dynamic", "--no-prefill", "--no-other-configs", "--cpu-seconds", "0.5"]
    print("bench contract run:", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=540)
    assert r.returncode == 0, r.stderr[-4000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout[-4000:]
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 20 and out["warmup"] == 3
    assert out["unit"] == "tok/s" and out["higher_is_better"] is True
    assert out["dtype"] == "f16" and out["data"] == "synthetic" and out["vs_baseline"] is None
    cfg = out["config"]
    assert cfg["workload"] and cfg["B"] == 32 and cfg["H"] == 32 and cfg["d"] == 128
    assert out["ms_per_step"] > 0
    assert out["value"] == pytest.approx(cfg["B"] / (out["ms_per_step"] * 1e-3), rel=1e-9)
    rf = out["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000
    assert rf["achieved"] == pytest.approx(rf["bytes_per_launch"] / (rf["us_per_launch"] * 1e-6) / 1e9,
                                           rel=1e-9)
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-9)
    assert 0.05 < rf["frac"] <= 1.0, rf
    # traffic comes from committed counter passes: a number only while the
    # kernel sources match the ones they were taken on
    if rf["traffic_source"]["status"] == "current":
        assert rf["traffic"] > 0
    else:
        assert rf["traffic"] is None
    cb = out["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "tok/s" and cb["value"] > 0
    assert 1 <= cb["cores"] <= 16 and cb["sample"]
