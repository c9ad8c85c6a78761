#!/usr/bin/env python3
"""TT-embedding benchmark on one MI355X.

Default: the training step of the 8-table workload.  One step is the whole
hot path over one batch: prefix-based index grouping, fused forward
(C = A.B per prefix group, E = C.D per unique row), sum pooling, backward
(dE segment sums, per-group dD/dC/dA/dB, core-gradient reduction) and the
in-place SGD update.  Workload: 8 TT tables of 1e7 rows (200 x 200 x 250),
D = 128 = 4 x 4 x 8, rank 32, 32,768 bags per table with Poisson(20) lengths
clipped to [1, 64], Zipf(1.1) row popularity over a seeded permutation,
upstream gradient N(0, 1), lr 0.01.

`--config 1..4` runs the forward-only workloads (one step = grouping, fused
forward and pooling); `--mode` overrides the step kind.  Inputs are synthetic
and already resident in HBM when the timed region starts.

Prints one JSON line (see the keys at the end of main()).
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3e12  # MI355X dense FP32 matrix FLOP/s
PEAK_HBM = 8.0e12          # MI355X HBM3E bytes/s
PEAK_FP32_VALU = 157.3e12  # MI355X FP32 vector FLOP/s
METRIC = "TT-embedding lookups/s + batch-32768 fwd/bwd latency (ms), % of roofline"


class HipEvents:
    """hipEvent_t handles through the HIP runtime (timed on the library's stream)."""

    def __init__(self):
        self.hip = C.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [C.c_void_p]
        self.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]

    def create(self):
        e = C.c_void_p()
        assert self.hip.hipEventCreate(C.byref(e)) == 0
        return e.value

    def record(self, e, stream):
        assert self.hip.hipEventRecord(e, stream) == 0

    def elapsed_ms(self, a, b):
        assert self.hip.hipEventSynchronize(b) == 0
        ms = C.c_float()
        assert self.hip.hipEventElapsedTime(C.byref(ms), a, b) == 0
        return float(ms.value)

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


# Source files that define each benchmarked kernel and its launch (the counters
# of a kernel stay valid while these files are unchanged).
KERNEL_SOURCES = {
    # the fused kernels' work units (slices, chunks) are cut by the grouping, sized in tt_emb.hip
    "bwd_fused": ["bwd_r32.hip", "bwd_r64.hip", "common.h", "group.hip", "tt_emb.hip"],
    "fwd_fused": ["fwd.hip", "common.h", "group.hip", "tt_emb.hip"],
    "pool": ["fwd.hip", "common.h"],
    "seg_sum": ["bwd.hip", "common.h"],
    "ingest": ["group.hip", "common.h"],
    "merge": ["cores.hip", "common.h"],
    "split": ["cores.hip", "common.h"],
}


def source_digest(kernel: str) -> str:
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2609_03459_amd", "csrc")
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(d, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


# Factorisations of the 10^7-row, D = 128 tables over L cores (--cores); for
# L >= 4 the first L-2 cores merge into a first core of (4, ...) columns, so the
# fused kernels see the same (4, 4, 8), R = 32 shape as with three cores.
CORE_SPLITS = {
    2: ((4000, 2500), (16, 8)),
    3: ((200, 200, 250), (4, 4, 8)),
    4: ((20, 10, 200, 250), (2, 2, 4, 8)),
    5: ((10, 20, 10, 20, 250), (2, 2, 1, 4, 8)),
}


def view_dims(n, d):
    """Three-factor view (rows, columns) that the grouping and fused kernels use."""
    L = len(n)
    if L == 2:
        return (n[0], 1, n[1]), (d[0], 1, d[1])
    p = lambda xs: int(__import__("numpy").prod(xs))
    return (p(n[:L - 2]), n[L - 2], n[L - 1]), (p(d[:L - 2]), d[L - 2], d[L - 1])


def chain_flops(n, d, R):
    """Flops of one merged-core row (L >= 4): the products S_0 . S_1 ... S_{L-3}."""
    m, f = d[0], 0.0
    for k in range(1, len(n) - 2):
        f += 2.0 * m * R * d[k] * R
        m *= d[k]
    return f


def algorithmic_work(kernel, case, counts, on_mfma=False):
    """(amount, unit, bound) per launch of `kernel` from the workload and its grouping.

    The fused backward's per-group work is C recomputed, dA and dB (6 d1 d2 R^2), except
    on the R = 64 matrix-core path, where dB is formed by the dG2 reduction from the
    per-slice dC partials and the fused kernel does C and dA (4 d1 d2 R^2)."""
    T, B, R = case["T"], case["B"], case["R"]
    _, (d1, d2, d3) = view_dims(case["n"], case["d"])
    D = d1 * d2 * d3
    U, P, nv = counts["U"], counts["P"], counts["nvalid"]
    M = int(case["idx"].size)
    NB = T * B
    if kernel == "fwd_fused":
        return P * 2.0 * d1 * d2 * R * R + U * 2.0 * D * R, "flop", "mfma"
    if kernel == "bwd_fused":
        g = 4.0 if (R == 64 and on_mfma) else 6.0
        return P * g * d1 * d2 * R * R + U * 4.0 * D * R, "flop", "mfma"
    if kernel == "pool":
        return 4.0 * M + 8.0 * (NB + 1) + 4.0 * NB * D + 4.0 * U * D, "byte", "hbm"
    if kernel == "seg_sum":  # dV rows read once, dE rows written, row id and bag per sorted occurrence
        return 4.0 * NB * D + 4.0 * U * D + 8.0 * nv + 4.0 * (U + 1), "byte", "hbm"
    if kernel == "ingest":
        return 8.0 * M + 8.0 * (NB + 1) + 12.0 * M, "byte", "hbm"
    (n1, _, _), _ = view_dims(case["n"], case["d"])
    if kernel == "merge":
        return T * n1 * chain_flops(case["n"], case["d"], R), "flop", "alu"
    if kernel == "split":  # two products per chain step, on every merged row
        return T * n1 * 2.0 * chain_flops(case["n"], case["d"], R), "flop", "alu"
    raise ValueError(kernel)


KERNEL_SYMBOL = {"fwd_fused": "k_fwd_r32", "bwd_fused": "k_bwd_r32", "pool": "k_pool", "seg_sum": "k_seg_dE",
                 "ingest": "k_ingest"}


def kernel_symbol(kernel, R=32):
    """Symbol of the MFMA kernel that serves `kernel` at rank R (the forward and the
    backward have one for R = 32 and one for R = 64)."""
    if kernel == "fwd_fused" and R == 64:
        return "k_fwd_r64"
    if kernel == "bwd_fused" and R == 64:
        return "k_bwd_r64"
    return KERNEL_SYMBOL[kernel]


def step_work(case, counts, mode):
    """Algorithmic flops F and HBM bytes Q of one whole step (all tables), from the
    workload and its grouping (U unique rows, P prefix groups over all tables).
      forward: F = P 2 d1 d2 R^2 + U 2 D R + M D (stage 1, stage 2, pooling adds)
               Q = 8 M (indices) + 8 (T B + 1) (offsets) + 4 T B D (output) + 4 |cores| (read once)
      train  : adds F += M D (dE aggregation) + U 4 D R (dD, dC) + P 6 d1 d2 R^2 (C again, dA, dB)
                        + 2 |cores| (the update)
                    Q += 4 T B D (upstream gradient) + 4 |cores| (gradients) + 12 |cores| (update:
                        read core and gradient, write core)"""
    T, B, R = case["T"], case["B"], case["R"]
    (n1, n2, n3), (d1, d2, d3) = view_dims(case["n"], case["d"])
    D = d1 * d2 * d3
    U, P = counts["U"], counts["P"]
    M = int(case["idx"].size)
    if "cores" in case:
        ncore = sum(int(G.size) for G in case["cores"])
    else:
        ncore = int(case["G1"].size + case["G2"].size + case["G3"].size)
    F = P * 2.0 * d1 * d2 * R * R + U * 2.0 * D * R + M * D
    Q = 8.0 * M + 8.0 * (T * B + 1) + 4.0 * T * B * D + 4.0 * ncore
    if mode == "train":
        F += M * D + U * 4.0 * D * R + P * 6.0 * d1 * d2 * R * R + 2.0 * ncore
        Q += 4.0 * T * B * D + 4.0 * ncore + 12.0 * ncore
    return F, Q


def whole_call(case, counts, mode, ms):
    """The step's roofline time max(F / peak FP32, Q / peak HBM) and its fraction of the
    measured step time."""
    F, Q = step_work(case, counts, mode)
    tf, tq = F / PEAK_FP32_MFMA, Q / PEAK_HBM
    t = max(tf, tq)
    return {"flop": F, "bytes": Q, "bound": "fp32" if tf >= tq else "hbm", "roof_ms": round(t * 1e3, 5),
            "frac": round(t / (ms * 1e-3), 4)}


def cpu_model():
    """Model name of the host CPU (first entry of /proc/cpuinfo) and its logical CPU count."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return name, os.cpu_count() or 0


def run_key(args):
    """What a counter measurement holds for: the workload and the flags that change the kernels' work."""
    import ttgen

    name = ttgen.CONFIGS[args.config]["workload"]
    if getattr(args, "bags", None):
        name += f"_bags{args.bags}"
    if args.row_factors or args.cores != 3:
        L = len(args.row_factors.split(",")) if args.row_factors else args.cores
        name += f"_{L}cores"
        if args.row_factors:
            name += f"[{args.row_factors}|{args.dim_factors}]"
    key = {"workload": name, "reuse": args.reuse, "sched": args.sched, "fused_sgd": not args.unfused_sgd}
    mode = step_mode(args)
    if mode != "train":
        key["mode"] = mode
    return key


def step_mode(args):
    """The step the run times: the training step for the training workloads (configs 5 and 6),
    the forward for the forward-only workloads, unless --mode says otherwise."""
    import ttgen

    m = getattr(args, "mode", None)
    return m if m else ("train" if ttgen.CONFIGS[args.config]["train"] else "forward")


def write_traffic(pmc_dir, key, copy_mib=1024, kernel="bwd_fused", R=32):
    """HBM bytes per launch of `kernel` from rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch).

    Each counter is scaled by the factor that makes it read the true size on the
    calibration copy (one elementwise kernel that reads and writes copy_mib MiB).
    """
    import csv
    import glob

    import numpy as np

    sym = kernel_symbol(kernel, R)
    vals = {"FETCH_SIZE": {"k": [], "copy": []}, "WRITE_SIZE": {"k": [], "copy": []}}
    for f in sorted(glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)):
        for r in csv.DictReader(open(f)):
            c = r["Counter_Name"]
            if c not in vals:
                continue
            name = r["Kernel_Name"]
            if f"::{sym}(" in name or f"::{sym}<" in name:
                vals[c]["k"].append(float(r["Counter_Value"]))
            elif "elementwise" in name:
                vals[c]["copy"].append(float(r["Counter_Value"]))
    true_kib = copy_mib * 1024.0
    out = {"kernel": kernel, "symbol": sym, "source": source_digest(kernel), "run": key, "copy_mib": copy_mib}
    total = 0.0
    for c, v in vals.items():
        if not v["k"] or not v["copy"]:
            raise SystemExit(f"{pmc_dir}: no {c} rows for {sym} and the calibration copy")
        raw = float(np.mean(v["k"]))
        scale = true_kib / max(v["copy"])
        out[c] = {"raw_kib_per_dispatch": round(raw, 1), "dispatches": len(v["k"]),
                  "copy_raw_kib": round(max(v["copy"]), 1), "scale": round(scale, 4),
                  "bytes_per_launch": round(raw * scale * 1024.0)}
        total += raw * scale * 1024.0
    out["bytes_per_launch"] = round(total)
    path = os.path.join(ROOT, "profiles", "traffic.json")
    entries = traffic_entries(path)
    entries = [e for e in entries if not (e.get("kernel") == kernel and e.get("run") == key)] + [out]
    with open(path, "w") as f:
        json.dump({"entries": entries}, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


def traffic_entries(path):
    """Stored counter measurements: one entry per (kernel, run)."""
    if not os.path.exists(path):
        return []
    tr = json.load(open(path))
    return tr.get("entries", [tr] if "kernel" in tr else [])


def measured_traffic(kernel, key, on_mfma, path=None, R=32):
    """HBM bytes per launch from profiles/traffic.json, or None unless counters were
    taken on this kernel as it is now (source digest), on this run (workload, reuse,
    schedule, update mode, step) and on the MFMA kernel the entry names."""
    path = path or os.path.join(ROOT, "profiles", "traffic.json")
    if not on_mfma:
        return None
    for tr in traffic_entries(path):
        if (tr.get("kernel") == kernel and tr.get("source") == source_digest(kernel) and tr.get("run") == key
                and tr.get("symbol") == kernel_symbol(kernel, R)):
            return tr.get("bytes_per_launch")
    return None


def cpu_baseline(case, target_s, mode="train"):
    """The oracle (plain fp64 C, one thread) on a bounded sample of the same workload:
    a seeded subset of bags of every table, forward then (training step) backward.
    Returns the one-thread figure and the same sample with the tables (independent)
    run on a thread pool, one single-table oracle call per table."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    T, B = case["T"], case["B"]
    off = case["offsets"]

    def sub(nb):
        rng = np.random.default_rng(99)
        bags = np.sort(rng.choice(B, size=nb, replace=False))
        idx_parts, lens, dv = [], [], []
        for t in range(T):
            for b in bags:
                gb = t * B + b
                lo, hi = (off[gb], off[gb + 1]) if off is not None else (gb, gb + 1)
                idx_parts.append(case["idx"][lo:hi])
                lens.append(hi - lo)
            if "dV" in case:
                dv.append(case["dV"][t, bags])
        o = np.zeros(T * nb + 1, np.int64)
        o[1:] = np.cumsum(lens)
        out = dict(case, B=nb, idx=np.concatenate(idx_parts), offsets=o)
        if dv:
            out["dV"] = np.stack(dv)
        return out

    def run(c):
        t0 = time.perf_counter()
        if "cores" in c:
            oracle.forward_n(c)
            if mode == "train":
                oracle.backward_n(c)
        else:
            oracle.forward(c)
            if mode == "train":
                oracle.backward(c)
        return time.perf_counter() - t0

    def table(c, t):  # table t of a sample as a one-table case
        nb = c["B"]
        o = c["offsets"]
        lo, hi = o[t * nb], o[(t + 1) * nb]
        one = dict(c, T=1, idx=c["idx"][lo:hi], offsets=o[t * nb:(t + 1) * nb + 1] - lo)
        if "dV" in c:
            one["dV"] = c["dV"][t:t + 1]
        if "cores" in c:
            one["cores"] = [G[t:t + 1] for G in c["cores"]]
        else:
            one.update(G1=c["G1"][t:t + 1], G2=c["G2"][t:t + 1], G3=c["G3"][t:t + 1])
        return one

    probe = sub(8)
    dt = run(probe)
    rate = probe["idx"].size / max(dt, 1e-6)
    nb = int(min(B, max(8, target_s * rate / max(probe["idx"].size / 8.0, 1.0))))
    s = sub(nb)
    dt = run(s)
    lookups = int(s["idx"].size)
    what = "forward + backward" if mode == "train" else "forward"
    model, ncpu = cpu_model()
    one = dict(value=lookups / dt, unit="lookups/s", cores=1, kind="oracle",
               sample=f"{nb} seeded bags per table x {T} tables ({lookups} lookups), {what}, "
                      f"fp64 C oracle, 1 thread, {dt:.1f} s", cpu_model=model, host_cpus=ncpu)
    from concurrent.futures import ThreadPoolExecutor
    nthr = max(1, min(T, os.cpu_count() or 1, 16))
    parts = [table(s, t) for t in range(T)]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(nthr) as ex:
        list(ex.map(run, parts))
    dtm = time.perf_counter() - t0
    many = dict(value=lookups / dtm, unit="lookups/s", cores=nthr, kind="oracle",
                sample=f"the same sample, {T} tables on {nthr} threads (one single-table oracle call each), "
                       f"{dtm:.1f} s", cpu_model=model, host_cpus=ncpu)
    return one, many


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=5,
                    help="workload recipe (5 = training step; 1-4 = the forward-only workloads; 6 = the "
                         "training step at the paper's D = 32, R = 32)")
    ap.add_argument("--mode", choices=["train", "forward"], default=None,
                    help="step to time: training step (default for config 5) or forward = grouping, fused "
                         "forward and pooling (default for configs 1-4)")
    ap.add_argument("--bags", type=int, default=None, help="bags per table (default: the workload's 32,768)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--reuse", choices=["prefix", "unique", "none"], default="prefix",
                    help="reuse level (ablation of Section 4.5): prefix groups (default), exact dedup only, none")
    ap.add_argument("--sched", choices=["steal", "static", "steal_ckpt", "group"], default="steal",
                    help="work distribution (ablation of Section 4.4): stealing (default), static shares, "
                         "stealing with checkpointed intermediates, static prefix mapping (whole groups)")
    ap.add_argument("--cores", type=int, choices=sorted(CORE_SPLITS), default=3,
                    help="number of TT cores: the same tables factorised over L cores (L > 3: future work in "
                         "the paper)")
    ap.add_argument("--row-factors", default=None, help="comma-separated row factors (overrides --cores)")
    ap.add_argument("--dim-factors", default=None, help="comma-separated column factors (with --row-factors)")
    ap.add_argument("--unfused-sgd", action="store_true",
                    help="backward into gradient arrays, then a separate SGD call (default with three cores: "
                         "the fused backward-and-SGD call)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run one plain elementwise copy of this many MiB (counter calibration runs)")
    ap.add_argument("--write-traffic", metavar="DIR", default=None,
                    help="CPU only: turn the FETCH_SIZE / WRITE_SIZE counter CSVs under DIR (one rocprofv3 --pmc "
                         "pass each, of a run with --copy-mib and the same workload flags) into "
                         "profiles/traffic.json, then exit")
    ap.add_argument("--traffic-kernel", default=None, choices=sorted(KERNEL_SYMBOL),
                    help="with --write-traffic: the kernel the counters are for (default: the step's fused kernel)")
    args = ap.parse_args()
    mode = step_mode(args)
    if args.write_traffic:
        import ttgen

        kern = args.traffic_kernel or ("bwd_fused" if mode == "train" else "fwd_fused")
        write_traffic(args.write_traffic, run_key(args), kernel=kern, R=ttgen.CONFIGS[args.config]["R"])
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_03459_amd as P
    import ttgen

    case = ttgen.make(args.config, bags=args.bags, with_grad=mode == "train")
    if args.row_factors or args.cores != 3:
        if args.row_factors:
            nL = tuple(int(x) for x in args.row_factors.split(","))
            dL = tuple(int(x) for x in args.dim_factors.split(","))
        else:
            nL, dL = CORE_SPLITS[args.cores]
        if int(np.prod(nL)) < case["N"] or int(np.prod(dL)) != int(np.prod(case["d"])):
            sys.exit(f"factors {nL} x {dL} do not hold {case['N']} rows of {int(np.prod(case['d']))} columns")
        rng = np.random.default_rng([int(case["seed"]), 4242])
        # random cores of the same spread as the three-core recipe's, per core
        sig = float(np.std(case["G2"]))
        case = dict(case, n=nL, d=dL, L=len(nL), workload=case["workload"] + f"_{len(nL)}cores",
                    cores=[(rng.standard_normal(sh) * sig).astype(np.float32)
                           for sh in ttgen.core_shapes_n(case["T"], nL, dL, case["R"])])
        for k in ("G1", "G2", "G3"):
            case.pop(k)
    T, n, d, R, B = case["T"], case["n"], case["d"], case["R"], case["B"]
    L = len(n)
    D = int(np.prod(d))
    M = int(case["idx"].size)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    emb = P.TTEmbedding(T, case["N"], n, d, R, max_indices=M, max_bags=B, reuse=args.reuse, sched=args.sched)
    if "cores" in case:
        G = [torch.from_numpy(x).to(dev) for x in case["cores"]]
    else:
        G = [torch.from_numpy(case[k]).to(dev) for k in ("G1", "G2", "G3")]
    idx = torch.from_numpy(case["idx"]).to(dev)
    off = None if case["offsets"] is None else torch.from_numpy(case["offsets"]).to(dev)
    dV = torch.from_numpy(case["dV"]).to(dev) if mode == "train" else None
    out = torch.empty((T, B, D), dtype=torch.float32, device=dev)
    grads = tuple(torch.empty(s, dtype=torch.float32, device=dev) for s in emb.core_shapes()) if (
        mode == "train" and ("cores" in case or args.unfused_sgd)) else None
    lr = case.get("lr", 0.01)
    stream = torch.cuda.current_stream().cuda_stream
    ev = HipEvents()

    if "cores" in case:
        def fwd(reuse):
            emb.forward_n(G, idx, off, num_bags=B, out=out, reuse_grouping=reuse)

        def bwd():
            emb.backward_n(G, idx, off, dV, num_bags=B, grads=grads, reuse_grouping=True)

        def sgd():
            emb.sgd_n(G, grads, lr)
    elif args.unfused_sgd:
        def fwd(reuse):
            emb.forward(*G, idx, off, num_bags=B, out=out, reuse_grouping=reuse)

        def bwd():
            emb.backward(*G, idx, off, dV, num_bags=B, grads=grads, reuse_grouping=True)

        def sgd():
            emb.sgd(*G, *grads, lr)
    else:
        # the library's training step: backward with the SGD update applied in its
        # final gradient reductions (no gradient arrays, no separate update pass)
        def fwd(reuse):
            emb.forward(*G, idx, off, num_bags=B, out=out, reuse_grouping=reuse)

        def bwd():
            emb.backward_sgd(*G, idx, off, dV, lr, num_bags=B, reuse_grouping=True)

        def sgd():
            pass

    def step():
        fwd(False)
        if mode == "train":
            bwd()
            sgd()

    if args.copy_mib:
        # reads and writes exactly copy_mib MiB each: the calibration of the byte counters
        x = torch.ones(args.copy_mib << 18, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        torch.mul(x, 2.0, out=y)
        torch.cuda.synchronize()
        del x, y

    # warmup; the first steps also time each candidate kernel once
    kernels = [k for k in P.N.KERNELS if (L >= 4 or k not in ("merge", "split")) and
               (mode == "train" or k not in ("seg_sum", "bwd_fused", "split"))]
    kernel_ms = {}
    e0, e1 = ev.create(), ev.create()
    for w in range(max(args.warmup, len(kernels))):
        k = kernels[w] if w < len(kernels) else None
        if k:
            P.N.tt_emb_profile(emb.handle, P.N.KERNELS[k], e0, e1)
        step()
        if k:
            torch.cuda.synchronize()
            kernel_ms[k] = ev.elapsed_ms(e0, e1)
            P.N.tt_emb_profile(emb.handle, 0, None, None)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    counts = emb.counts()
    dominant = max(kernel_ms, key=kernel_ms.get)

    # timed region: K steps; the dominant kernel is bracketed by events in every
    # step, and every step by events on the stream (for the per-step median)
    K = args.steps
    evs = [(ev.create(), ev.create()) for _ in range(K)]
    sev = [ev.create() for _ in range(K + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        ev.record(sev[i], stream)
        P.N.tt_emb_profile(emb.handle, P.N.KERNELS[dominant], evs[i][0], evs[i][1])
        step()
    ev.record(sev[K], stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    P.N.tt_emb_profile(emb.handle, 0, None, None)
    ms_per_step = (t1 - t0) * 1e3 / K
    dom_ms = float(np.mean([ev.elapsed_ms(a, b) for a, b in evs]))
    step_med = float(np.median([ev.elapsed_ms(sev[i], sev[i + 1]) for i in range(K)]))

    # measured copy bandwidth: one elementwise kernel reading and writing 1 GiB each
    x = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    cps = []
    ce0, ce1 = ev.create(), ev.create()
    for _ in range(4):
        ev.record(ce0, stream)
        torch.mul(x, 2.0, out=y)
        ev.record(ce1, stream)
        torch.cuda.synchronize()
        cps.append(ev.elapsed_ms(ce0, ce1))
    copy_gbps = 2.0 * x.numel() * 4 / (float(np.median(cps[1:])) * 1e-3) / 1e9
    del x, y

    # phase split (grouping / forward / backward / sgd), as in the paper's breakdown
    phases = {"group": [], "forward": [], "backward": [], "sgd": []}
    if mode != "train":
        phases = {"group": [], "forward": []}
    pe = [ev.create() for _ in range(5)]
    for _ in range(3):
        ev.record(pe[0], stream)
        emb.group(idx, off, num_bags=B)
        ev.record(pe[1], stream)
        fwd(True)
        ev.record(pe[2], stream)
        if mode == "train":
            bwd()
            ev.record(pe[3], stream)
            sgd()
            ev.record(pe[4], stream)
        torch.cuda.synchronize()
        for j, name in enumerate(phases):
            phases[name].append(ev.elapsed_ms(pe[j], pe[j + 1]))
    phases_ms = {k: round(float(np.median(v)), 4) for k, v in phases.items()}

    # the fused kernels run on the matrix cores only for the shapes the MFMA kernels serve
    on_mfma = dominant in ("fwd_fused", "bwd_fused") and P.N.tt_emb_kernel_uses_mfma(
        emb.handle, P.N.KERNELS[dominant], M)
    work, unit, bound = algorithmic_work(dominant, case, counts, on_mfma=bool(on_mfma))
    if bound == "mfma" and not on_mfma:
        bound = "alu"
    if unit == "flop" and bound == "alu":
        achieved = work / (dom_ms * 1e-3) / 1e12
        roof = dict(bound=bound, achieved=round(achieved, 3), peak=PEAK_FP32_VALU / 1e12, unit="TFLOP/s",
                    frac=round(achieved / (PEAK_FP32_VALU / 1e12), 4))
    elif unit == "flop":
        achieved = work / (dom_ms * 1e-3) / 1e12
        roof = dict(bound=bound, achieved=round(achieved, 3), peak=PEAK_FP32_MFMA / 1e12, unit="TFLOP/s",
                    frac=round(achieved / (PEAK_FP32_MFMA / 1e12), 4))
    else:
        achieved = work / (dom_ms * 1e-3) / 1e9
        roof = dict(bound=bound, achieved=round(achieved, 1), peak=PEAK_HBM / 1e9, unit="GB/s",
                    frac=round(achieved / (PEAK_HBM / 1e9), 4))
    roof["traffic"] = measured_traffic(dominant, run_key(args), on_mfma, R=R)
    roof["kernel"] = dominant
    roof["symbol"] = kernel_symbol(dominant, R) if on_mfma else None
    roof["kernel_ms"] = round(dom_ms, 4)

    lookups = M
    res = {
        "metric": METRIC,
        "value": lookups / (ms_per_step * 1e-3),
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": case["workload"], "tables": T, "rows_per_table": case["N"], "cores": L,
                   "row_factors": list(n),
                   "dim_factors": list(d), "rank": R, "batch_per_table": B, "lookups": lookups,
                   "step": ("group+forward+pool+backward+sgd" + (
                       " (sgd fused into the backward's reductions)" if L == 3 and not args.unfused_sgd else ""))
                   if mode == "train" else "group+forward+pool",
                   "parallelism": "single-gpu",
                   "reuse": args.reuse, "sched": args.sched},
        "roofline": roof,
        "whole_call": whole_call(case, counts, mode, ms_per_step),
        "step_ms_median": round(step_med, 4),
        "copy_gbps_measured": round(copy_gbps, 1),
        "phases_ms": phases_ms,
        "kernel_ms_warmup": {k: round(v, 4) for k, v in kernel_ms.items()},
        "grouping": {"unique_rows": counts["U"], "prefix_groups": counts["P"], "slices": counts["nslices"]},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"], res["cpu_baseline_threads"] = cpu_baseline(case, args.cpu_seconds, mode)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
