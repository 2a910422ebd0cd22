"""bench.py's output contract: one JSON line with the fields the measurement
record needs (metric, value, roofline of the dominant kernel, the oracle's
CPU baseline), and a clear refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, timeout):
    return subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"], timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert not r.stdout.strip()


@pytest.mark.gpu
def test_bench_line_fields():
    r = _run(["--steps", "3", "--warmup", "1", "--cpu-seconds", "1", "--no-schedule", "--no-opt", "--no-half",
              "--no-fp32-path", "--no-references", "--no-stabilised"], timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    assert d["unit"] == "layer-updates/s" and d["metric"] and d["value"] > 0
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["ms_per_step"] > 0 and abs(d["value"] - d["config"]["n_layers"] / (d["ms_per_step"] / 1e3)) < 1e-6 * d["value"]
    assert d["higher_is_better"] is True and d["scaling"] in ("weak", "strong")
    assert d["vs_baseline"] is None or d["vs_baseline"] > 0
    assert d["dtype"] == "f32" and d["data"].startswith("synthetic")
    assert "workload" in d["config"]
    roof = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in roof, k
    assert roof["bound"] in ("hbm", "mfma", "alu")
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"])
    assert 0 < roof["frac"] < 1
    pw = roof.get("power")
    if pw is not None:   # amd-smi present: the clock the dominant GEMM ran at
        assert 0 < pw["gfx_mhz"] <= pw["nominal_mhz"] * 1.05 and pw["board_w"] > 0 and pw["samples"] > 0
        assert pw["frac_at_clock"] == pytest.approx(roof["achieved"] / pw["peak_at_clock"])
        assert pw["frac_at_clock"] >= roof["frac"] * 0.999
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["unit"] and cb["sample"]
    assert len(d["timing"]["windows_ms_per_step"]) == d["timing"]["repeats"]
