"""bench.py on the CPU: the oracle baseline leg for every strategy and
optimizer, the refusal of more than one GPU, and the lookup of the committed
HBM-traffic summaries (which must name the sources they were taken on)."""
import json
import os

import pytest

import bench
from synth import WORKLOADS


@pytest.mark.parametrize("method", ["cpdp", "localsgd", "ddp"])
@pytest.mark.parametrize("optimizer", ["sgd", "sgd_wd", "adamw"])
def test_cpu_baseline_runs_every_strategy_and_optimizer(method, optimizer):
    w = WORKLOADS["tiny"]
    r = bench.cpu_baseline(w, budget_s=0.02, n_coords=256, parallel_budget_s=0.02,
                           method=method, optimizer=optimizer)
    assert r["kind"] == "oracle" and r["unit"] == "replica-params/s"
    assert r["cores"] == bench.cpu_threads()["threads"] and r["value"] > 0
    assert r["host_cpu_count"] == os.cpu_count()
    assert r["affinity_cpus"] == len(os.sched_getaffinity(0))
    assert f"({method}, {optimizer})" in r["sample"]
    one = r["single_thread"]
    assert one["cores"] == 1 and one["value"] > 0 and one["period_replica_params_per_s"] > 0
    assert f"({method}, {optimizer})" in one["sample"]
    assert one["extrapolated"] is True  # 256 of 262,144 coordinates
    assert one["s_per_reconcile_full_P"] > 0


def test_cpu_threads_follow_affinity_and_job_share(monkeypatch):
    """Every CPU of the affinity set, capped by the job's CPU share."""
    aff = len(os.sched_getaffinity(0))
    monkeypatch.delenv("OMP_NUM_THREADS", raising=False)
    assert bench.cpu_threads()["threads"] == aff
    monkeypatch.setenv("OMP_NUM_THREADS", "1")
    c = bench.cpu_threads()
    assert c["threads"] == 1 and c["omp_num_threads"] == 1 and c["affinity_cpus"] == aff
    monkeypatch.setenv("OMP_NUM_THREADS", str(aff + 100))
    assert bench.cpu_threads()["threads"] == aff


def test_oracle_slice_counts_whole_periods():
    """Every timed period is K steps: K-1 local steps and one synchronisation
    (DDP: K synchronisations)."""
    w = WORKLOADS["r50_100"]
    for method, local_per_period in (("cpdp", w.K - 1), ("ddp", 0)):
        r = bench._oracle_slice(w, 5, 64, 0.01, method, "sgd")
        assert r["periods"] >= 1
        assert r["loc_n"] == local_per_period * r["periods"]
        assert r["rec_n"] == (w.K - local_per_period) * r["periods"]


def test_more_than_one_gpu_is_refused(capsys, monkeypatch):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    assert bench.main() == 2
    assert "exactly one GPU" in capsys.readouterr().err


def test_traffic_summaries_name_their_sources():
    """Each committed FETCH_SIZE / WRITE_SIZE summary records the kernel-source
    hash it was taken on, the kernel, the workload and bytes close to the
    algorithmic ones; bench.py reports its figure only while that hash is the
    current one."""
    d = os.path.join(bench.ROOT, "profiles")
    found = 0
    for name in sorted(os.listdir(d)):
        if not name.endswith("_pmc.txt"):
            continue
        text = open(os.path.join(d, name)).read()
        line = [x for x in text.splitlines() if x.startswith("TRAFFIC_JSON: ")]
        assert len(line) == 1, name
        rec = json.loads(line[0][len("TRAFFIC_JSON: "):])
        assert name.startswith(f"{rec['kernel']}_{rec['workload']}"), name
        assert len(rec["source_hash"]) == 16
        assert 0.99 < rec["bytes_per_launch"] / rec["algorithmic_bytes"] < 1.01, name
        variant = name[len(f"{rec['kernel']}_{rec['workload']}"):-len("_pmc.txt")]
        got = bench.recorded_traffic(rec["kernel"], rec["workload"], variant)
        if rec["source_hash"] == bench.kernel_source_hash():
            assert got == rec["bytes_per_launch"], name
        else:
            assert got is None, name
        found += 1
    assert found >= 9
    assert bench.recorded_traffic("reconcile", "no_such_workload") is None


def test_source_hash_ignores_comments_and_layout_only():
    code = "int a = 1; // the count\n/* block\n comment */ float b;\n"
    assert bench._code_only(code) == "int a = 1; float b;"
    assert bench._code_only("int  a =\n 1;   float b;") == bench._code_only(code)
    assert bench._code_only(code.replace("1", "2")) != bench._code_only(code)
    h = bench.kernel_source_hash()
    assert len(h) == 16 and h == bench.kernel_source_hash()
