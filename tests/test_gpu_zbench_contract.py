"""bench.py's output line on a small workload: one JSON object with the
fields the measurement contract names (metric, value, unit, n_gpus, steps,
warmup, ms_per_step, higher_is_better, scaling, vs_baseline, dtype, data,
config with the workload, roofline with bound / achieved / peak / unit /
frac / traffic, cpu_baseline with value / unit / cores / kind / sample), and
a value consistent with the step time."""
import json
import os
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_on_the_tiny_workload(monkeypatch, capsys):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # bench.main() in this process, with a command line of its own.
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "tiny", "--steps", "5",
                                      "--warmup", "1", "--detail-iters", "0"])
    bench.main()
    out = capsys.readouterr().out
    lines = [l for l in out.splitlines() if l.strip()]
    assert len(lines) == 1, out
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["data"] == "synthetic"
    assert d["config"]["workload"] == "tiny"
    n_t, b = d["config"]["n_triples"], d["config"]["batch"]
    assert abs(d["value"] - n_t * b / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    roof = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in roof, k
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    cpu = d["cpu_baseline"]
    for k in ("value", "unit", "cores", "kind", "sample"):
        assert k in cpu, k
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0
    assert d["cpu_baseline"]["sample"].startswith("the whole workload")
    par = d["parity"]["max_tol_ratio"]
    assert set(par) == {"Y", "dX", "dR"} and max(par.values()) <= 1.0, par
    assert d["kb_sha256"] and d["seeds"]["root"] == 20020615 and d["kb_stats"]
    assert roof["kernel"] in d["kernels"].values()
    assert roof["step"]["array_once_frac"] > 0


def test_bench_line_on_the_chain3_workload(monkeypatch, capsys):
    """The three-hop chain mode: one line, its value consistent with the step
    time (three follows per step), and parity with the chain oracle."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "chain3", "--steps", "5",
                                      "--warmup", "1"])
    bench.main()
    lines = [l for l in capsys.readouterr().out.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    assert d["config"]["workload"] == "chain3" and d["config"]["hops"] == 3
    n_t, b = d["config"]["n_triples"], d["config"]["batch"]
    assert abs(d["value"] - 3 * n_t * b / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    assert d["cpu_baseline"]["kind"] == "oracle" and d["cpu_baseline"]["value"] > 0
    assert max(d["parity"]["max_tol_ratio"].values()) <= 1.0
    assert d["parity"]["loss_abs_diff"] <= 1e-7 + 1e-5 * 10
