"""bench.py's output contract, on a short run of the tiny workload: exactly
one JSON line on stdout, with the required keys, a value consistent with its
own step time, and a roofline whose fraction is achieved / peak."""
import json
import os
import subprocess
import sys

import pytest

from paper_2411_17866_amd import arena as A

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REQUIRED = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
            "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline")


@pytest.mark.parametrize("extra", [[], ["--sign", "rand", "--path", "split",
                                          "--replica-layout", "contiguous"],
                                   ["--replica-layout", "state-blocked", "--placement", "probe"]])
def test_bench_prints_one_consistent_json_line(extra):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny",
                        "--steps", "3", "--warmup", "1", "--extra-steps", "2", *extra],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    for key in REQUIRED:
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 3 and out["warmup"] == 1
    assert out["higher_is_better"] is True and out["data"] == "synthetic"
    cfg = out["config"]
    assert "workload" in cfg and cfg["updates_per_step"] == (cfg["n_workers"] * cfg["local_steps"] + 1) * cfg["d"]
    assert abs(out["value"] - cfg["updates_per_step"] / (out["ms_per_step"] / 1e3)) <= 1e-9 * out["value"]
    roof = out["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert roof["traffic"] is None or roof["traffic"] > 0
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0 and cpu["sample"]
    assert cpu["fp32"]["value"] > 0 and cpu["fp64"]["value"] > 0
    # The untimed round after the timed ones matched the oracle.
    par = out["parity"]
    assert par["elements"] > 0 and par["values_compared"] >= par["elements"]
    assert par["non_bit_identical"] == 0 and par["flips_outside_margin"] == 0
    for name, entry in out["breakdown"].items():
        assert entry is not None and entry["launches"] >= 2, name
    # The placement probe, when asked for, reports what it chose.
    pl = cfg.get("placement")
    if "probe" in extra:
        assert pl["candidates"] == A.PROBE_SPAN_BYTES // A.PROBE_STEP_BYTES + 1
        assert 0 <= pl["offset_GB"] <= A.PROBE_SPAN_BYTES / 1e9 + 0.01
        assert pl["probe_ms_best"] <= pl["probe_ms_worst"]
    else:
        assert pl is None
