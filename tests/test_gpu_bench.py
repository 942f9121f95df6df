"""bench.py end to end on the GPU: a short tiny run prints one JSON line that
keeps the benchmark contract (value = the reconcile's replica-params/s, the
roofline objects, both shape-ceiling orders and both copy streams).  Runs
bench.main() in this process."""
import json
import sys

import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(monkeypatch, capsys, *args):
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py", *args])
    assert bench.main() == 0
    lines = [x for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    assert len(lines) == 1, lines
    return json.loads(lines[0])


def test_bench_line_keeps_the_contract(monkeypatch, capsys):
    d = _run(monkeypatch, capsys, "--workload", "tiny", "--steps", "3", "--warmup", "1",
             "--no-cpu-baseline")
    assert d["metric"].startswith("reconcile replica-params/s")
    assert d["unit"] == "replica-params/s" and d["n_gpus"] == 1 and d["higher_is_better"]
    assert d["steps"] == 3 and d["warmup"] == 1 and d["data"] == "synthetic"
    W, P = d["config"]["W"], d["config"]["P"]
    rec = d["reconcile"]
    assert rec["launches"] == 3
    # value is the reconcile's own rate, not the period's (ms is printed to 5
    # decimals, a few parts in 1e4 of tiny's 9 us)
    assert d["value"] == pytest.approx(W * P / (rec["ms"] * 1e-3), rel=2e-3)
    assert d["period_replica_params_per_s"] == pytest.approx(
        W * P * d["config"]["K"] / (d["ms_per_step"] * 1e-3), rel=1e-3)
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], abs=1e-4)
    assert roof["bytes_per_launch"] == (5 * W + 4) * 4 * P
    assert set(d["copy_ceiling_streams_GBps"]) == {"synth_copy_f32", "shape_1r1w"}
    assert d["copy_ceiling_GBps"] == max(d["copy_ceiling_streams_GBps"].values())
    shape = d["shape_ceiling"]
    assert set(shape["orders_GB_per_s"]) == {"batched_in_place", "library_order"}
    assert shape["GB_per_s"] == max(shape["orders_GB_per_s"].values())
    assert roof["frac_of_shape_ceiling"] == pytest.approx(roof["achieved"] / shape["GB_per_s"],
                                                          abs=1e-4)
    assert "cpu_baseline" not in d


def test_bench_line_of_a_baseline_strategy(monkeypatch, capsys):
    d = _run(monkeypatch, capsys, "--workload", "tiny", "--method", "localsgd", "--optimizer",
             "adamw", "--steps", "2", "--warmup", "1", "--no-cpu-baseline")
    assert d["sync_kernel"] == "localsgd_sync" and d["roofline"]["kernel"] == "localsgd_sync"
    assert set(d["shape_ceiling"]["orders_GB_per_s"]) == {"batched_in_place", "library_order"}
