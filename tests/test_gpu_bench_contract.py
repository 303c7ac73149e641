"""The benchmark's JSON line on the device: a short run (1 timed prefill
step, 4 decode steps, a small oracle sample) prints one line with every field
the contract asks for, the roofline and CPU-baseline objects included."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_has_the_contract_fields():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "1",
                          "--warmup", "1", "--decode-steps", "4", "--cpu-pairs", "300",
                          "--speedup-lengths", "16384"],
                         capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert res.returncode == 0, res.stderr[-2000:]
    line = res.stdout.strip().splitlines()[-1]
    d = json.loads(line)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 1 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert "workload" in d["config"]
    rl = d["roofline"]
    assert rl["bound"] == "mfma" and rl["unit"] == "TFLOP/s" and rl["peak"] == 2500.0
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-3)
    assert rl["traffic"] is None or rl["traffic"] > 0
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
    dec = d["decode"]
    assert dec["tok_per_s"] > 0
    drl = dec["roofline"]
    assert drl["bound"] == "hbm" and drl["unit"] == "GB/s" and drl["peak"] == 8000.0
    assert drl["frac"] == pytest.approx(drl["achieved"] / drl["peak"], rel=1e-3)
    assert dec["cpu_baseline"]["kind"] == "oracle" and dec["cpu_baseline"]["unit"] == "tok/s"
    assert cb["cpu_model"] and dec["cpu_baseline"]["cpu_model"]
    hs = dec["hbm_step"]
    assert hs["unit"] == "GB/s" and hs["frac"] == pytest.approx(hs["achieved"] / hs["peak"], rel=1e-3)
    assert sum(hs["share"].values()) == pytest.approx(1.0, abs=1e-3)
    # the other workloads and the sparse/dense ratios come in the same line
    pcts = sorted(r["density_pct"] for r in d["configs"] if r["workload"] == "stress")
    assert pcts == [10, 20, 40, 100]
    assert any(r["workload"] == "varlen" for r in d["configs"])
    assert d["speedup"]["prefill_one_layer"][0]["speedup_vs_dense_this_kernel"] > 1.0
    assert d["speedup"]["decode_one_layer"][0]["speedup_vs_dense_this_kernel"] > 1.0
