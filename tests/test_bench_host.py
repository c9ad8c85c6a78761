"""Host logic of the benchmark (CPU only): the run key that counter traffic is
stamped with, when the stored traffic is reported, and the algorithmic work the
roofline prices."""
import argparse
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _args(**kw):
    a = dict(config=5, cores=3, row_factors=None, dim_factors=None, reuse="prefix", sched="steal",
             unfused_sgd=False)
    a.update(kw)
    return argparse.Namespace(**a)


def test_run_key_names_what_changes_the_work():
    base = bench.run_key(_args())
    assert base["workload"].startswith("tt-embbag-train-8x1e7rows")
    assert base == {"workload": base["workload"], "reuse": "prefix", "sched": "steal", "fused_sgd": True}
    assert bench.run_key(_args(config=3))["workload"] != base["workload"]
    assert bench.run_key(_args(cores=4))["workload"] == base["workload"] + "_4cores"
    assert bench.run_key(_args(reuse="none")) != base
    assert bench.run_key(_args(sched="static")) != base
    assert bench.run_key(_args(unfused_sgd=True)) != base
    rf = bench.run_key(_args(row_factors="20,10,200,250", dim_factors="2,2,4,8"))
    assert rf["workload"].endswith("_4cores[20,10,200,250|2,2,4,8]")


def test_traffic_reported_only_for_the_run_and_source_it_was_taken_on(tmp_path):
    key = bench.run_key(_args())
    good = {"kernel": "bwd_fused", "symbol": "k_bwd_r32", "source": bench.source_digest("bwd_fused"), "run": key,
            "bytes_per_launch": 123}
    p = tmp_path / "traffic.json"

    def put(d):
        p.write_text(json.dumps(d))
        return str(p)

    assert bench.measured_traffic("bwd_fused", key, True, put(good)) == 123
    assert bench.measured_traffic("bwd_fused", key, False, put(good)) is None  # generic kernel ran
    assert bench.measured_traffic("fwd_fused", key, True, put(good)) is None
    assert bench.measured_traffic("bwd_fused", bench.run_key(_args(config=3)), True, put(good)) is None
    assert bench.measured_traffic("bwd_fused", key, True, put(dict(good, source="0" * 16))) is None
    assert bench.measured_traffic("bwd_fused", key, True, str(tmp_path / "missing.json")) is None


def test_algorithmic_work_of_the_fused_kernels():
    # one table, one prefix group of one row: the per-group and per-row terms
    case = {"T": 1, "B": 1, "R": 32, "n": (200, 200, 250), "d": (4, 4, 8), "idx": np.zeros(1, np.int64)}
    counts = {"U": 1, "P": 1, "nvalid": 1}
    fwd, unit, bound = bench.algorithmic_work("fwd_fused", case, counts)
    assert (unit, bound) == ("flop", "mfma") and fwd == 2 * 16 * 32 * 32 + 2 * 128 * 32
    bwd, _, _ = bench.algorithmic_work("bwd_fused", case, counts)
    assert bwd == 6 * 16 * 32 * 32 + 4 * 128 * 32
    # the dominant kernel of the training workload: 48.3 GFLOP at its grouping counts
    big = dict(case, T=8)
    w, _, _ = bench.algorithmic_work("bwd_fused", big, {"U": 1089937, "P": 309642, "nvalid": 5246700})
    assert abs(w / 1e9 - 48.3) < 0.1
