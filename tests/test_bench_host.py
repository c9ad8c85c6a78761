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
             unfused_sgd=False, mode=None, bags=None)
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
    # at R = 64 on the matrix cores dB leaves the fused kernel (formed by the dG2 reduction)
    r64 = dict(case, R=64)
    assert bench.algorithmic_work("bwd_fused", r64, counts)[0] == 6 * 16 * 64 * 64 + 4 * 128 * 64
    assert bench.algorithmic_work("bwd_fused", r64, counts, on_mfma=True)[0] == 4 * 16 * 64 * 64 + 4 * 128 * 64
    assert bench.algorithmic_work("bwd_fused", case, counts, on_mfma=True)[0] == bwd


def test_run_key_and_step_of_the_forward_only_workloads():
    # configs 1-4 time the forward (grouping, fused forward, pooling) unless told otherwise
    assert bench.step_mode(_args(config=4)) == "forward"
    assert bench.step_mode(_args(config=5)) == "train"
    assert bench.step_mode(_args(config=4, mode="train")) == "train"
    k4 = bench.run_key(_args(config=4))
    assert k4["mode"] == "forward" and "mode" not in bench.run_key(_args())
    assert bench.run_key(_args(config=4, mode="train")) != k4
    assert bench.run_key(_args(bags=4096))["workload"].endswith("_bags4096")
    # the forward's MFMA kernel at rank 64 is its own symbol
    assert bench.kernel_symbol("fwd_fused", 64) == "k_fwd_r64"
    assert bench.kernel_symbol("fwd_fused", 32) == "k_fwd_r32"
    assert bench.kernel_symbol("bwd_fused", 32) == "k_bwd_r32"
    assert bench.kernel_symbol("bwd_fused", 64) == "k_bwd_r64"


def _case8():
    n, d, R, T, B = (200, 200, 250), (4, 4, 8), 32, 8, 32768
    return {"T": T, "B": B, "R": R, "n": n, "d": d, "idx": np.zeros(5246700, np.int64),
            "G1": np.zeros((T, n[0], d[0], R), np.float32), "G2": np.zeros((T, n[1], R, d[1], R), np.float32),
            "G3": np.zeros((T, n[2], R, d[2]), np.float32)}


def test_step_work_of_the_training_workload():
    # the whole call's algorithmic flops and bytes at the training workload's grouping
    case = _case8()
    counts = {"U": 1089937, "P": 309642, "nvalid": 5246700}
    M, NB, D = 5246700, 8 * 32768, 128
    ncore = 8 * (200 * 4 * 32 + 200 * 32 * 4 * 32 + 250 * 32 * 8)
    Ff, Qf = bench.step_work(case, counts, "forward")
    assert Ff == 309642 * 2 * 16 * 32 * 32 + 1089937 * 2 * 128 * 32 + M * D
    assert Qf == 8 * M + 8 * (NB + 1) + 4 * NB * D + 4 * ncore
    Ft, Qt = bench.step_work(case, counts, "train")
    assert Ft - Ff == M * D + 1089937 * 4 * 128 * 32 + 309642 * 6 * 16 * 32 * 32 + 2 * ncore
    assert Qt - Qf == 4 * NB * D + 16 * ncore
    # about 19.8 + 49 GFLOP: compute-bound, about 0.44 ms of FP32 peak
    assert 68e9 < Ft < 70e9
    w = bench.whole_call(case, counts, "train", 2.0)
    assert w["bound"] == "fp32" and abs(w["roof_ms"] - Ft / 157.3e12 * 1e3) < 1e-4
    assert abs(w["frac"] - (Ft / 157.3e12) / 2.0e-3) < 1e-4
    # a latency-scale forward of 4,096 single lookups is bound by its bytes
    small = {"T": 1, "B": 4096, "R": 8, "n": (100, 100, 100), "d": (2, 2, 4), "idx": np.zeros(4096, np.int64),
             "G1": np.zeros((1, 100, 2, 8)), "G2": np.zeros((1, 100, 8, 2, 8)), "G3": np.zeros((1, 100, 8, 4))}
    ws = bench.whole_call(small, {"U": 4090, "P": 3356, "nvalid": 4096}, "forward", 0.1)
    assert ws["bound"] == "hbm"


def test_cpu_model_is_named():
    name, n = bench.cpu_model()
    assert isinstance(name, str) and name and n >= 1
