"""The benchmark's output contract, on the tiny workload: one JSON line with
the metric, the timing fields, the configuration, the roofline of the fused
kernel (against the HBM peak, with the probe beside it) and the step's phase
breakdown and percentiles."""
import json
import os
import subprocess
import sys

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bench_prints_one_contract_line(dtype):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny",
                        "--steps", "6", "--warmup", "2", "--no-cpu", "--dtype", dtype],
                       capture_output=True, text=True, timeout=280, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 6 and d["warmup"] == 2
    assert d["higher_is_better"] is True and d["unit"] == "positives/s"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert d["config"]["workload"] == "tiny" and d["config"]["tables"] == dtype
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["achieved"] > 0 and rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"])
    assert rf["probe"]["achieved"] > 0 and rf["timed_launches"] >= 1
    assert rf["traffic"] is None  # counters are committed for the SBM-100M workload only
    st = d["step"]
    assert st["unique_src_rows"] > 0 and st["unique_ctx_rows"] > 0
    assert 0 < st["ms_percentiles"]["p10"] <= st["ms_percentiles"]["p50"] \
        <= st["ms_percentiles"]["p90"]
    assert d["cpu_baseline"] is None  # --no-cpu

