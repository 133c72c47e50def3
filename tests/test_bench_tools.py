"""CPU checks of bench.py's measurement tooling: the HBM bytes it takes
from the committed rocprofv3 summaries, the profiling commands it prints,
and the CPU baseline's sampling on a small workload."""
import dataclasses
import re

import pytest

import bench
import kgsynth
import oracle


def test_traffic_sums_the_kernels_timed_as_one_unit():
    one = bench.traffic_for("freebase", "k_heavy<3p> r0")
    units = bench.traffic_for("freebase", "k_units<3p> r0")
    if one is None:
        pytest.skip("profiles were taken on other sources")
    both = bench.traffic_for("freebase", "k_heavy<3p> r0 + k_units<3p> r0")
    assert both == one + units
    assert bench.traffic_for("freebase", "k_heavy<3p> r0 + k_nothing r0") is None
    assert bench.traffic_for("no_such_workload", "k_heavy<3p> r0") is None


def test_traffic_is_null_for_other_sources(monkeypatch):
    monkeypatch.setattr(bench, "sample_hip_sha", lambda: "0000000000000000")
    assert bench.traffic_for("freebase", "k_candidates<3p> r0") is None


@pytest.mark.parametrize("config", ["freebase", "wikikg2"])
def test_profile_commands(config):
    cmds = bench.profile_commands(config, 20, "out")
    assert cmds[0] == f"mkdir -p out/prof_{config}/trace"
    for c in cmds[1:]:
        assert c.startswith("rocprofv3 ")
        # the program itself follows "--": no shell, env or launcher in between
        prog = c.split(" -- ", 1)[1]
        assert prog.startswith("python3 -u bench.py")
        assert f" -d out/prof_{config}/" in c
        if "--copy-calibration" not in prog:     # the copy is the same for every workload
            assert (config == "freebase") == ("--config" not in prog)
        # counters never combined with a trace, and within one pass's limits
        if "--pmc" in c:
            assert "--kernel-trace" not in c and "--sys-trace" not in c
            ctrs = c.split("--pmc ", 1)[1].split(" -d ")[0].split()
            assert sum(x.startswith("TCC_") for x in ctrs) <= 4
            assert sum(x.startswith("SQ_") for x in ctrs) <= 8


def test_cpu_baseline_times_a_small_workload_over_a_measurable_span():
    # a batch of 16 queries: the oracle finishes it within the time slice
    # even on a loaded host, so the sample must go on past it
    cfg = dataclasses.replace(kgsynth.CONFIGS["tiny"], batch=16)
    tr = kgsynth.generate(cfg, threads=2)
    og = oracle.Graph(tr, cfg.n_entities, cfg.n_relations, cfg.add_inverse, threads=2)
    r = bench.cpu_baseline(cfg, og, ["1p", "2p"], 0.6, 2, 2)
    assert r["kind"] == "oracle" and r["cores"] == 2 and r["value"] > 0
    assert set(r["per_type_queries_per_s"]) == {"1p", "2p"}
    # later query ids extend the sample past the batch
    counts = [int(x) for x in re.findall(r": first (\d+)", r["sample"])]
    assert len(counts) == 2 and all(n > cfg.batch for n in counts)
