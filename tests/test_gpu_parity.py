"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer grouping outputs must match bit for bit; float outputs within the
scaled-error bound of tests/_util.py.  Small cases compare every element;
full-size workloads compare seeded samples the oracle computes one by one.
"""
import sys

import numpy as np
import pytest
import torch

import ttgen
from tests._util import TOL, abs_case, assert_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_03459_amd as P

    return P


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dev(case):
    G = [torch.from_numpy(np.ascontiguousarray(case[k])).cuda() for k in ("G1", "G2", "G3")]
    idx = torch.from_numpy(np.ascontiguousarray(case["idx"], dtype=np.int64)).cuda()
    off = None if case["offsets"] is None else torch.from_numpy(np.ascontiguousarray(case["offsets"])).cuda()
    return G, idx, off


def _make(lib, case):
    M = int(case["idx"].size)
    return lib.TTEmbedding(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=max(M, 1),
                           max_bags=max(int(case["B"]), 1))


def gpu_forward(lib, case):
    emb = _make(lib, case)
    G, idx, off = _dev(case)
    out = emb.forward(*G, idx, off, num_bags=case["B"])
    torch.cuda.synchronize()
    D = int(np.prod(case["d"]))
    return out.cpu().numpy().reshape(case["T"] * case["B"], D), emb, G, idx, off


def check_forward(lib, orc, case, bags=None, name=""):
    _say(f"[fwd] {name} T={case['T']} n={case['n']} d={case['d']} R={case['R']} B={case['B']} "
         f"M={case['idx'].size}")
    V, emb, *_ = gpu_forward(lib, case)
    assert emb.check_errors() == 0
    ref, inv = orc.forward(case, bags=bags)
    mag, _ = orc.forward(abs_case(case), bags=bags)
    got = V if bags is None else V[bags]
    return assert_close(f"forward {name}", got, ref, mag)


TINY = [
    dict(T=1, n=(3, 4, 5), d=(2, 3, 2), R=3, B=7, max_len=5),
    dict(T=2, n=(2, 3, 7), d=(1, 2, 4), R=5, B=40, max_len=6),
    dict(T=3, n=(1, 5, 2), d=(3, 1, 1), R=1, B=9, max_len=4),
    dict(T=2, n=(7, 1, 3), d=(2, 2, 2), R=4, B=33, max_len=5),
    dict(T=1, n=(50, 40, 30), d=(4, 4, 8), R=32, B=300, max_len=20, zipf=1.1),
    dict(T=2, n=(20, 30, 40), d=(4, 4, 8), R=64, B=100, max_len=32, zipf=1.2),
    dict(T=1, n=(100, 100, 100), d=(2, 2, 4), R=8, B=1000, single=True),
    dict(T=2, n=(9, 11, 13), d=(3, 5, 7), R=17, B=50, max_len=9),
    dict(T=4, n=(200, 200, 250), d=(4, 4, 4), R=16, B=512, single=True, zipf=1.05),
    # D = 32 at R = 32 (the paper's operating point): MFMA forward over groups of eight rows
    dict(T=2, n=(30, 20, 40), d=(4, 4, 2), R=32, B=300, max_len=20, zipf=1.1),
]


@pytest.mark.parametrize("k", range(len(TINY)))
def test_forward_small(lib, orc, k):
    c = dict(TINY[k])
    case = ttgen.tiny(1000 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    check_forward(lib, orc, case, name=f"tiny{k}")


@pytest.mark.parametrize("k", [0, 1, 4, 5, 7])
def test_grouping_bit_exact(lib, orc, k):
    c = dict(TINY[k])
    case = ttgen.tiny(2000 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    _say(f"[group] tiny{k}")
    emb = _make(lib, case)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    got = emb.debug_grouping(case["idx"].size)
    ref = orc.grouping(case)
    n = case["n"]
    npad = n[0] * n[1] * n[2]
    assert got["U"] == ref["U"] and got["P"] == ref["P"] and got["nvalid"] == ref["nvalid"]
    assert np.array_equal(got["uniq_keys"], ref["uniq_t"] * npad + ref["uniq_g"])
    assert np.array_equal(got["digits"], orc.digits(ref["uniq_g"], n).astype(np.int32))
    assert np.array_equal(got["inv"], ref["inv"])
    assert np.array_equal(got["occ_start"], ref["occ_start"])
    assert np.array_equal(got["occ_pos"], ref["occ_pos"])
    assert np.array_equal(got["pg_start"], ref["pg_start"])
    assert np.array_equal(got["pg_keys"], ref["pg_t"] * (n[0] * n[1]) + ref["pg_q"])


# key widths that select each radix digit width: 19 bits (two 10-bit passes),
# 22 bits (two 11-bit passes), 31 and 32 bits (three 11-bit passes)
WIDE_KEYS = [
    dict(T=1, n=(64, 64, 64)),
    dict(T=1, n=(128, 128, 128)),
    dict(T=3, n=(1000, 1000, 700)),
    dict(T=2, n=(1024, 1024, 1024)),
]


def _check_grouping(lib, orc, case):
    emb = _make(lib, case)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    got = emb.debug_grouping(case["idx"].size)
    ref = orc.grouping(case)
    n = case["n"]
    npad = n[0] * n[1] * n[2]
    assert got["U"] == ref["U"] and got["P"] == ref["P"] and got["nvalid"] == ref["nvalid"]
    assert np.array_equal(got["uniq_keys"], ref["uniq_t"] * npad + ref["uniq_g"])
    assert np.array_equal(got["inv"], ref["inv"])
    assert np.array_equal(got["occ_start"], ref["occ_start"])
    assert np.array_equal(got["occ_pos"], ref["occ_pos"])
    assert np.array_equal(got["pg_start"], ref["pg_start"])
    assert np.array_equal(got["pg_keys"], ref["pg_t"] * (n[0] * n[1]) + ref["pg_q"])


# 300 bags (about 1,000 keys) are sorted in one launch, 3,000 bags in radix passes over tiles
@pytest.mark.parametrize("bags", [300, 3000])
@pytest.mark.parametrize("k", range(len(WIDE_KEYS)))
def test_grouping_and_forward_wide_keys(lib, orc, k, bags):
    c = WIDE_KEYS[k]
    case = ttgen.tiny(2500 + k, c["T"], c["n"], (1, 2, 2), 2, B=bags, max_len=6, zipf=1.1)
    _say(f"[group wide] T={c['T']} n={c['n']} M={case['idx'].size}")
    _check_grouping(lib, orc, case)
    check_forward(lib, orc, case, name=f"wide{k} B={bags}")


# the chunk list of up to 4,095 (table, i2) runs is built by one workgroup, of more
# runs by three launches
@pytest.mark.parametrize("n", [(3, 2047, 4), (3, 2048, 4)])
def test_grouping_many_runs(lib, orc, n):
    case = ttgen.tiny(2700 + n[1], 2, n, (2, 2, 2), 4, B=400, max_len=8, zipf=1.05)
    _say(f"[group runs] T=2 n={n} M={case['idx'].size}")
    _check_grouping(lib, orc, case)
    check_forward(lib, orc, case, name=f"runs n2={n[1]}")
    check_backward(lib, orc, case, name=f"runs n2={n[1]}")


# a sort tile holds 4,096 keys: up to one tile is sorted in a single launch
@pytest.mark.parametrize("m", [4095, 4096, 4097, 8193])
def test_grouping_at_sort_tile_sizes(lib, orc, m):
    case = ttgen.tiny(2600 + m, 1, (30, 20, 40), (2, 2, 2), 4, B=m, single=True, zipf=1.1)
    _say(f"[group tile] M={m}")
    _check_grouping(lib, orc, case)
    check_forward(lib, orc, case, name=f"M={m}")


def test_many_short_bags(lib, orc):
    # 20,000 bags of at most one index: a tile of 4096 occurrences spans more
    # bags than the ingest window holds, so bag ids come from the global search
    case = ttgen.tiny(2600, 1, (10, 10, 10), (2, 2, 2), 2, B=20000, max_len=1)
    check_forward(lib, orc, case, name="short bags")
    emb = _make(lib, case)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    got = emb.debug_grouping(case["idx"].size)
    ref = orc.grouping(case)
    assert np.array_equal(got["inv"], ref["inv"]) and np.array_equal(got["occ_pos"], ref["occ_pos"])


@pytest.mark.parametrize("reuse", ["unique", "none"])
@pytest.mark.parametrize("k", [4, 5, 7, 9])
def test_reuse_levels_same_results(lib, orc, reuse, k):
    # Section 4.5 ablation levels compute the same function: forward and backward
    # against the oracle with exact dedup only, and with no dedup at all
    c = dict(TINY[k])
    case = ttgen.tiny(4000 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    _say(f"[reuse {reuse}] tiny{k}")
    M = int(case["idx"].size)
    emb = lib.TTEmbedding(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=max(M, 1),
                          max_bags=max(int(case["B"]), 1), reuse=reuse)
    G, idx, off = _dev(case)
    D = int(np.prod(case["d"]))
    out = emb.forward(*G, idx, off, num_bags=case["B"])
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    ref, _ = orc.forward(case)
    mag, _ = orc.forward(abs_case(case))
    assert_close(f"forward {reuse}", out.cpu().numpy().reshape(-1, D), ref, mag)
    dV = torch.from_numpy(case["dV"]).cuda()
    grads = emb.backward(*G, idx, off, dV, num_bags=case["B"])
    torch.cuda.synchronize()
    refg = orc.backward(case)
    magg = orc.backward(abs_case(case))
    for k2, name in enumerate(("dG1", "dG2", "dG3")):
        assert_close(f"{name} {reuse}", grads[k2].cpu().numpy().ravel(), refg[k2].ravel(), magg[k2].ravel())


def _rank2_cores(n, d, R):
    n1, n2, n3 = n
    d1, d2, d3 = d
    D = d1 * d2 * d3
    G1 = np.zeros((1, n1, d1, R), np.float32)
    G2 = np.zeros((1, n2, R, d2, R), np.float32)
    G3 = np.zeros((1, n3, R, d3), np.float32)
    G1[0, :, :, 0] = (np.arange(n1)[:, None] * n2 * n3 * D + np.arange(d1)[None, :] * d2 * d3)
    G1[0, :, :, 1] = 1
    G2[0, :, 0, :, 0] = 1
    G2[0, :, 1, :, 0] = np.arange(n2)[:, None] * n3 * D + np.arange(d2)[None, :] * d3
    G2[0, :, 1, :, 1] = 1
    G3[0, :, 0, :] = 1
    G3[0, :, 1, :] = np.arange(n3)[:, None] * D + np.arange(d3)[None, :]
    return G1, G2, G3


def test_rank2_closed_form_bit_exact_config1_shape(lib):
    # E[g][j] = g*D + j exactly in fp32 while N*D < 2^24 (1e6 rows, D = 16)
    case = ttgen.make(1)
    case["G1"], case["G2"], case["G3"] = _rank2_cores(case["n"], case["d"], case["R"])
    _say("[fwd] rank-2 closed form, 1e6 x 16, R=8")
    V, emb, *_ = gpu_forward(lib, case)
    D = 16
    ref = case["idx"][:, None].astype(np.float64) * D + np.arange(D)[None, :]
    assert np.array_equal(V.astype(np.float64), ref)


def test_full_config1(lib, orc):
    check_forward(lib, orc, ttgen.make(1), name="config1 full")


def test_full_config2(lib, orc):
    check_forward(lib, orc, ttgen.make(2), name="config2 full")


def test_config3_small_batch(lib, orc):
    check_forward(lib, orc, ttgen.make(3, bags=256), name="config3 B=256")


def test_config4_small_batch(lib, orc):
    check_forward(lib, orc, ttgen.make(4, bags=128), name="config4 B=128")


def test_config6_small_batch(lib, orc):
    check_forward(lib, orc, ttgen.make(6, bags=256), name="config6 B=256")


@pytest.mark.parametrize("cfg", [3, 4, 6])
def test_full_size_sampled_bags(lib, orc, cfg):
    case = ttgen.make(cfg)
    bags = ttgen.sample_bags(cfg, case["T"], case["B"], 96)
    check_forward(lib, orc, case, bags=bags, name=f"config{cfg} full, 96 sampled bags")


@pytest.mark.parametrize("k", [1, 7])
def test_generic_backward_deterministic(lib, k):
    # the generic backward reduces its partials by fixed-order segment sums: two runs
    # (fresh handles and workspaces, so the scheduling differs) give the same bits
    c = dict(TINY[k])
    case = ttgen.tiny(3500 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    _say(f"[bwd determinism] tiny{k}")
    runs = []
    for _ in range(2):
        emb, G, grads, dV = gpu_train(lib, case)
        assert not lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], case["idx"].size)
        runs.append([g.cpu().numpy() for g in grads])
    for a, b in zip(*runs):
        assert np.array_equal(a, b)


def test_r64_backward_deterministic(lib):
    # the R = 64 MFMA backward writes per-slice, per-chunk and per-row partials that the
    # same fixed-order segment sums reduce: two runs give the same bits
    c = dict(TINY[5])
    case = ttgen.tiny(3505, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    _say("[bwd determinism] tiny5 R=64")
    runs = []
    for _ in range(2):
        emb, G, grads, dV = gpu_train(lib, case)
        assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], case["idx"].size)
        runs.append([g.cpu().numpy() for g in grads])
    for a, b in zip(*runs):
        assert np.array_equal(a, b)


def test_forward_deterministic(lib):
    case = ttgen.make(3, bags=512)
    _say("[fwd] determinism config3 B=512")
    V1, *_ = gpu_forward(lib, case)
    V2, *_ = gpu_forward(lib, case)
    assert np.array_equal(V1, V2)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------
def _edge(kind, d=(2, 2, 2), R=4):
    case = ttgen.tiny(77, 2, (6, 5, 100), d, R, B=40, max_len=8, zipf=1.1)
    idx = case["idx"].copy()
    rng = np.random.default_rng(5)
    n3 = 100
    if kind == "all_equal":
        idx[:] = 1234
    elif kind == "one_prefix":
        idx = 7 * n3 + rng.integers(0, n3, idx.size)  # one (i1, i2) group, up to 100 rows: several slices
    elif kind == "distinct_prefixes":
        q = rng.permutation(30)[: min(30, idx.size)]
        idx = (np.resize(q, idx.size) * n3 + rng.integers(0, n3, idx.size)).astype(np.int64)
    case["idx"] = idx.astype(np.int64)
    return case


EDGE_SHAPES = [((2, 2, 2), 4), ((4, 4, 8), 32), ((4, 4, 8), 64), ((4, 4, 2), 32)]


@pytest.mark.parametrize("dR", EDGE_SHAPES, ids=["generic", "mfma_r32", "mfma_r64", "mfma_r32_d32"])
@pytest.mark.parametrize("kind", ["all_equal", "one_prefix", "distinct_prefixes"])
def test_edge_index_patterns(lib, orc, kind, dR):
    # each pattern through the forward, the backward and the fused backward-and-SGD,
    # on the generic kernels and on the MFMA shapes (R = 32 and R = 64: both fused
    # kernels on the matrix cores)
    case = _edge(kind, *dR)
    name = f"{kind} d={dR[0]} R={dR[1]}"
    check_forward(lib, orc, case, name=name)
    check_backward(lib, orc, case, name=name)
    _say(f"[bwd+sgd] {name}")
    emb = _make(lib, case)
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.backward_sgd(*G, idx, off, dV, 0.01, num_bags=case["B"], reuse_grouping=False)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    _check_sgd(orc, case, G, 0.01, name)


def _run_slices(g, n, slice_rows=32):
    """Work slices (at most slice_rows rows each: 32, or 16 on the R = 64 matrix-core shape)
    of every prefix group from a debug grouping, in the fused kernels' (table, i2, i1)
    order, with each group's first slice within its (table, i2) run: returns (rows,
    slices, first, run) per group."""
    n1, n2 = n[0], n[1]
    keys = np.asarray(g["pg_keys"], np.int64)
    rows = np.diff(np.asarray(g["pg_start"], np.int64))
    t, q = keys // (n1 * n2), keys % (n1 * n2)
    i1, i2 = q // n2, q % n2
    order = np.lexsort((i1, i2, t))
    sl = (rows + slice_rows - 1) // slice_rows
    run = (t * n2 + i2)[order]
    first = np.zeros(len(order), np.int64)
    acc, prev = 0, -1
    for j, p in enumerate(order):
        if run[j] != prev:
            acc, prev = 0, run[j]
        first[j] = acc
        acc += sl[p]
    return rows[order], sl[order], first, run


def _hot_prefix_case(seed, T, n, B, hot, per_bag=20, d=(4, 4, 8), R=32):
    """Bags whose indices fall in the listed hot prefixes (i1, i2) with uniform i3 most
    of the time, else anywhere: long prefix groups of many work slices."""
    case = ttgen.tiny(seed, T, n, d, R, B=B, max_len=per_bag, zipf=1.1, empty_bags=False)
    rng = np.random.default_rng(seed)
    idx = case["idx"].copy()
    pick = rng.random(idx.size) < 0.85
    h = np.asarray(hot)[rng.integers(0, len(hot), idx.size)]
    idx[pick] = ((h[pick, 0] * n[1] + h[pick, 1]) * n[2] + rng.integers(0, n[2], int(pick.sum())))
    case["idx"] = idx.astype(np.int64)
    return case


def test_forward_prefix_group_longer_than_a_chunk(lib, orc):
    # one (i1, i2) prefix with about 2,000 distinct suffixes: its group is cut into more
    # work slices than a chunk holds (32 x 32 rows), so the MFMA forward meets the same
    # group in consecutive chunks and quads
    n = (3, 2, 2000)
    case = _hot_prefix_case(7101, 1, n, B=300, hot=[(1, 1), (2, 0)], per_bag=24)
    emb = _make(lib, case)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["fwd_fused"], case["idx"].size)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    g = emb.debug_grouping(case["idx"].size)
    rows, sl, first, run = _run_slices(g, n)
    assert sl.max() > 32, sl.max()
    check_forward(lib, orc, case, name="group of > 32 slices")
    check_backward(lib, orc, case, name="group of > 32 slices (generic backward)")


def test_forward_d32_full_and_partial_row_groups(lib, orc):
    # D = 32 = (4, 4, 2): the MFMA forward takes eight rows of a slice per product.  Hot
    # prefixes give slices of 32 rows (four full groups) and the rest slices of one to a
    # few rows (one partial group), across chunk ends and quads
    n = (6, 4, 300)
    case = _hot_prefix_case(7303, 2, n, B=200, hot=[(1, 1), (4, 2), (5, 3)], per_bag=16, d=(4, 4, 2), R=32)
    emb = _make(lib, case)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["fwd_fused"], case["idx"].size)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    g = emb.debug_grouping(case["idx"].size)
    rows, sl, first, run = _run_slices(g, n)
    assert rows.max() > 64 and (rows % 8 != 0).any() and (rows < 8).any()
    check_forward(lib, orc, case, name="d=(4,4,2) hot prefixes")


def test_backward_d32_full_and_partial_row_groups(lib, orc):
    # D = 32 = (4, 4, 2) on the MFMA backward, which takes eight rows of a slice per
    # product: slices of 32 rows (four full groups) and of one to a few rows (a partial
    # group, whose missing rows add zeros elsewhere), across chunk ends and quads; the
    # gradients and the fused update against the oracle
    n = (6, 4, 250)
    case = _hot_prefix_case(7304, 2, n, B=200, hot=[(1, 1), (4, 2), (5, 3)], per_bag=16, d=(4, 4, 2), R=32)
    emb = _make(lib, case)
    M = case["idx"].size
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], M)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    g = emb.debug_grouping(M)
    rows, sl, first, run = _run_slices(g, n)
    assert rows.max() > 64 and (rows % 8 != 0).any() and (rows < 8).any()
    check_backward(lib, orc, case, name="d=(4,4,2) hot prefixes")
    _say("[bwd+sgd] d=(4,4,2) hot prefixes")
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.backward_sgd(*G, idx, off, dV, 0.01, num_bags=case["B"], reuse_grouping=False)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    _check_sgd(orc, case, G, 0.01, "d=(4,4,2) hot prefixes")


def test_backward_prefix_groups_across_chunk_ends(lib, orc):
    # twelve prefixes of one (table, i2) run, each with nearly all 250 suffixes: groups
    # of 7-8 work slices, so the run's slices fill several chunks and groups straddle
    # their ends, on both fused MFMA kernels (forward, backward, fused update)
    n = (12, 2, 250)
    hot = [(i1, 0) for i1 in range(12)]
    case = _hot_prefix_case(7102, 2, n, B=400, hot=hot, per_bag=20)
    emb = _make(lib, case)
    M = case["idx"].size
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["fwd_fused"], M)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], M)
    _, idx, off = _dev(case)
    emb.group(idx, off, num_bags=case["B"])
    g = emb.debug_grouping(M)
    rows, sl, first, run = _run_slices(g, n)
    straddle = (first // 32) != ((first + sl - 1) // 32)
    assert rows.max() > 200 and straddle.sum() >= 2, (rows.max(), straddle.sum())
    check_forward(lib, orc, case, name="groups across chunk ends")
    check_backward(lib, orc, case, name="groups across chunk ends")
    _say("[bwd+sgd] groups across chunk ends")
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.backward_sgd(*G, idx, off, dV, 0.01, num_bags=case["B"], reuse_grouping=False)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    _check_sgd(orc, case, G, 0.01, "groups across chunk ends")


@pytest.mark.parametrize("sched", ["steal", "group"])
def test_r64_backward_groups_across_quads_and_chunks(lib, orc, sched):
    # R = 64 cuts a (table, i2) run into chunks of four work slices (one quad) of at most
    # 16 rows; groups of 13-16 slices straddle quads and chunks.  Under the static prefix
    # mapping a chunk is a whole group of several quads.  Forward, backward (per-slice dC
    # sums, dG2 formed per run) and the fused update.
    n = (12, 2, 250)
    hot = [(i1, 0) for i1 in range(12)]
    case = _hot_prefix_case(7103, 2, n, B=300, hot=hot, per_bag=20, R=64)
    M = case["idx"].size
    name = f"R=64 groups across quads, {sched}"
    V, grads, emb = _run_mode(lib, case, sched=sched)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["fwd_fused"], M)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], M)
    g = emb.debug_grouping(M)
    rows, sl, first, run = _run_slices(g, n, slice_rows=16)
    assert sl.max() > 4 and ((first // 4) != ((first + sl - 1) // 4)).sum() >= 2
    ref_v, _ = orc.forward(case)
    mag_v, _ = orc.forward(abs_case(case))
    assert_close(f"forward {name}", V, ref_v, mag_v)
    ref = orc.backward(case)[:3]
    mag = orc.backward(abs_case(case))[:3]
    for k in range(3):
        assert_close(f"dG{k + 1} {name}", grads[k], ref[k], mag[k])
    _say(f"[bwd+sgd] {name}")
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.backward_sgd(*G, idx, off, dV, 0.01, num_bags=case["B"], reuse_grouping=False)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    _check_sgd(orc, case, G, 0.01, name)


def test_edge_empty_and_single_bag(lib, orc):
    case = ttgen.tiny(8, 2, (3, 4, 5), (2, 2, 2), 3, B=6, max_len=0)  # every bag empty, no indices
    assert case["idx"].size == 0
    _say("[fwd] all bags empty")
    V, *_ = gpu_forward(lib, case)
    assert np.array_equal(V, np.zeros_like(V))
    check_forward(lib, orc, ttgen.tiny(9, 3, (3, 4, 5), (2, 2, 2), 3, B=1, max_len=7, empty_bags=False),
                  name="B=1")


def test_invalid_indices_flagged_and_skipped(lib, orc):
    case = ttgen.tiny(10, 2, (4, 5, 6), (2, 2, 2), 3, B=30, max_len=6, N=100)
    idx = case["idx"].copy()
    idx[::5] = 100  # == N: first invalid row
    idx[1::7] = -2
    case["idx"] = idx
    _say("[fwd] invalid indices")
    V, emb, *_ = gpu_forward(lib, case)
    assert emb.check_errors() == 4  # TT_EMB_ERANGE
    assert emb.check_errors() == 0  # cleared
    ref, ninv = orc.forward(case)
    assert ninv > 0
    mag, _ = orc.forward(abs_case(case))
    assert_close("forward with invalid", V, ref, mag)


@pytest.mark.parametrize("kind", ["decreasing", "last_short", "first_nonzero"])
def test_malformed_offsets_flagged(lib, orc, kind):
    # offsets that are not a CSR partition of [0, M): every range is clamped into
    # [0, M] on the device, the error word reports it, and a later grouping with
    # good offsets clears it and gives the oracle's result
    case = ttgen.tiny(11, 2, (4, 5, 6), (2, 2, 2), 3, B=30, max_len=6, empty_bags=False)
    bad = dict(case)
    off = case["offsets"].copy()
    if kind == "decreasing":
        off[7] = off[9] + 2
    elif kind == "last_short":
        off[-1] -= 1
    else:
        off[0] = 1
    bad["offsets"] = off
    _say(f"[fwd] malformed offsets {kind}")
    emb = _make(lib, case)
    G, idx, good = _dev(case)
    _, _, wrong = _dev(bad)
    emb.forward(*G, idx, wrong, num_bags=case["B"])
    torch.cuda.synchronize()
    assert emb.check_errors() == 4  # TT_EMB_ERANGE
    out = emb.forward(*G, idx, good, num_bags=case["B"])  # same handle and workspace
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    V = out.cpu().numpy().reshape(case["T"] * case["B"], -1)
    ref, _ = orc.forward(case)
    mag, _ = orc.forward(abs_case(case))
    assert_close("forward after malformed offsets", V, ref, mag)


# ---------------------------------------------------------------------------
# backward and SGD
# ---------------------------------------------------------------------------
def gpu_train(lib, case):
    V, emb, G, idx, off = gpu_forward(lib, case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = emb.backward(*G, idx, off, dV, num_bags=case["B"], reuse_grouping=True)
    torch.cuda.synchronize()
    return emb, G, grads, dV


def check_backward(lib, orc, case, name="", want=None):
    _say(f"[bwd] {name} T={case['T']} n={case['n']} d={case['d']} R={case['R']} B={case['B']} "
         f"M={case['idx'].size}")
    emb, G, grads, dV = gpu_train(lib, case)
    ref = orc.backward(case, want=want)[:3]
    mag = orc.backward(abs_case(case), want=want)[:3]
    for k in range(3):
        got = grads[k].cpu().numpy()
        if want is None:
            assert_close(f"dG{k + 1} {name}", got, ref[k], mag[k])
        else:
            sel = np.flatnonzero(want[k])
            T = case["T"]
            g = got.reshape(T * got.shape[1], -1)[sel]
            r = ref[k].reshape(T * ref[k].shape[1], -1)[sel]
            m = mag[k].reshape(T * mag[k].shape[1], -1)[sel]
            assert_close(f"dG{k + 1} {name} (sampled slices)", g, r, m)
    return emb, G, grads, ref, mag


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4, 5, 7, 9])
def test_backward_small(lib, orc, k):
    c = dict(TINY[k])
    case = ttgen.tiny(3000 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    check_backward(lib, orc, case, name=f"tiny{k}")


@pytest.mark.parametrize("T,n,d,mfma", [
    (2, (6, 5, 252), (4, 4, 8), True),   # MFMA backward at its limit: the dG3 half plus scratch fill all 160 KB of LDS
    (2, (6, 5, 253), (4, 4, 8), False),  # one past it: the generic kernels
    (64, (2, 2, 9), (4, 4, 8), True),    # MFMA backward at its table limit (64 tables, 128 owners)
    (2, (6, 5, 252), (4, 4, 2), True),   # D = 32: the same n3 limit (i3 in 8-bit fields)
    (2, (6, 5, 253), (4, 4, 2), False),
    (64, (2, 2, 9), (4, 4, 2), True),
])
def test_backward_shape_limits(lib, orc, T, n, d, mfma):
    case = ttgen.tiny(3100 + n[2] + T + d[2], T, n, d, 32, B=24, max_len=10, zipf=1.1)
    emb = _make(lib, case)
    assert bool(lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], case["idx"].size)) == mfma
    check_backward(lib, orc, case, name=f"limits T={T} n3={n[2]} d={d}")
    check_forward(lib, orc, case, name=f"limits T={T} n3={n[2]} d={d}")


def _row_runs_case(seed, d, R):
    """Two tables whose sorted occurrences come in runs of chosen lengths, so that
    the ends of the 256-occurrence dE chunks fall before, inside and just past rows
    of 255, 256, 257, 511-513 and 1000 occurrences (the second table starts at
    another offset modulo 256)."""
    mult = [255, 256, 257, 1, 2, 511, 512, 513, 3, 1000, 256, 255, 1, 257, 7]
    T, n, B = 2, (6, 5, 40), 64
    case = ttgen.tiny(seed, T, n, d, R, B=B, max_len=1)
    rng = np.random.default_rng(seed)
    N = n[0] * n[1] * n[2]
    idx, lens = [], []
    for t in range(T):
        rows = np.sort(rng.choice(N, len(mult), replace=False))
        occ = np.repeat(rows, mult)
        rng.shuffle(occ)  # bag order: each row's occurrences spread over the bags
        cuts = np.sort(rng.integers(0, occ.size + 1, B - 1))
        lens.append(np.diff(np.concatenate([[0], cuts, [occ.size]])))
        idx.append(occ)
    case["idx"] = np.concatenate(idx).astype(np.int64)
    case["offsets"] = np.concatenate([[0], np.cumsum(np.concatenate(lens))]).astype(np.int64)
    return case


@pytest.mark.parametrize("d,R", [((4, 4, 8), 32), ((4, 4, 2), 32), ((2, 2, 2), 4)])
def test_backward_rows_across_dE_chunk_ends(lib, orc, d, R):
    check_backward(lib, orc, _row_runs_case(3300 + R, d, R), name=f"row runs d={d} R={R}")


@pytest.mark.parametrize("cfg", [5, 6])
def test_backward_small_batch(lib, orc, cfg):
    check_backward(lib, orc, ttgen.make(cfg, bags=64), name=f"config{cfg} B=64")


def _table_case(case, t):
    """Table t of a case as a one-table case of its own."""
    B = case["B"]
    off = case["offsets"]
    lo, hi = int(off[t * B]), int(off[(t + 1) * B])
    one = dict(case, T=1, idx=case["idx"][lo:hi], offsets=off[t * B:(t + 1) * B + 1] - lo)
    for k in ("G1", "G2", "G3"):
        one[k] = case[k][t:t + 1]
    if "dV" in case:
        one["dV"] = case["dV"][t:t + 1]
    return one


def _oracle_backward_by_table(orc, case, want):
    """orc.backward with slice masks, each table (independent of the others) as a case
    of its own on a thread pool; returns the three gradients stacked over tables."""
    from concurrent.futures import ThreadPoolExecutor

    T, n = case["T"], case["n"]

    def one(t):
        w = [m[t * n[k]:(t + 1) * n[k]] for k, m in enumerate(want)]
        if not any(x.any() for x in w):
            return None
        return orc.backward(_table_case(case, t), want=w)[:3]

    with ThreadPoolExecutor(min(T, 8)) as ex:
        parts = list(ex.map(one, range(T)))
    out = []
    for k in range(3):
        shape = (1,) + tuple(case[("G1", "G2", "G3")[k]].shape[1:])
        out.append(np.concatenate([np.zeros(shape) if p is None else p[k] for p in parts]))
    return out


def _hottest_slices(case, extra_tables=(0,), extra=2, seed=17):
    """Per core, the slice with the most occurrences in every table (the longest fp32
    sums of the gradient), plus `extra` random slices in the listed tables."""
    T, n, B = case["T"], case["n"], case["B"]
    bag = np.repeat(np.arange(T * B), np.diff(case["offsets"]))
    tab = bag // B
    dig = np.stack(np.unravel_index(case["idx"], n), 1)
    rng = np.random.default_rng(seed)
    want = [np.zeros(T * nk, np.uint8) for nk in n]
    for t in range(T):
        sel = tab == t
        for k in range(3):
            want[k][t * n[k] + np.bincount(dig[sel, k], minlength=n[k]).argmax()] = 1
            if t in extra_tables:
                want[k][t * n[k] + rng.choice(n[k], extra, replace=False)] = 1
    return want


def _sel(a, T, want_k):
    return a.reshape(T * a.shape[1], -1)[np.flatnonzero(want_k)]


@pytest.mark.parametrize("cfg", [5, 6])
def test_backward_full_hottest_slices(lib, orc, cfg):
    # The training workloads at full size (D = 128 and D = 32, both on the R = 32 MFMA
    # backward), in the launch sequence the benchmark times (forward with grouping,
    # then the backward reusing it): every table's most-used slice of each core (tens
    # of thousands of occurrences summed into one dG3 slice) plus random slices,
    # element by element against the oracle; then the fused backward-and-SGD call on
    # the same grouping, the call the benchmark times.
    case = ttgen.make(cfg)
    T, B, lr = case["T"], case["B"], case["lr"]
    M = int(case["idx"].size)
    want = _hottest_slices(case, extra_tables=(0, T - 1))
    _say(f"[bwd] config{cfg} full, hottest + random slices ({sum(int(w.sum()) for w in want)} slices)")
    emb = _make(lib, case)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], M)
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.forward(*G, idx, off, num_bags=B)
    grads = emb.backward(*G, idx, off, dV, num_bags=B, reuse_grouping=True)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    ref = _oracle_backward_by_table(orc, case, want)
    mag = _oracle_backward_by_table(orc, abs_case(case), want)
    for k in range(3):
        g = grads[k].cpu().numpy()
        assert_close(f"dG{k + 1} config{cfg} full (hottest slices)", _sel(g, T, want[k]), _sel(ref[k], T, want[k]),
                     _sel(mag[k], T, want[k]))
    del grads
    _say(f"[bwd+sgd] config{cfg} full, same slices")
    emb.backward_sgd(*G, idx, off, dV, lr, num_bags=B, reuse_grouping=True)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    for k, cname in enumerate(("G1", "G2", "G3")):
        new = _sel(G[k].cpu().numpy().astype(np.float64), T, want[k])
        exp = _sel(orc.sgd(case[cname], ref[k], lr), T, want[k])
        # gradient error scaled by lr plus one fp32 rounding of the updated value
        bound = TOL * lr * _sel(mag[k], T, want[k]) + 2.0 ** -23 * np.abs(exp)
        assert np.all(np.abs(new - exp) <= bound + 1e-30), cname


def _oracle_backward_by_slice(orc, case, want):
    """orc.backward with slice masks, one wanted slice per call on a thread pool (each
    call visits only the occurrences that touch its slice); returns the three
    gradients with the wanted slices filled in."""
    from concurrent.futures import ThreadPoolExecutor

    tasks = [(k, int(i)) for k, m in enumerate(want) for i in np.flatnonzero(m)]

    def one(task):
        k, i = task
        w = [np.zeros_like(m) for m in want]
        w[k][i] = 1
        return orc.backward(case, want=w)[k]

    with ThreadPoolExecutor(min(len(tasks), 16)) as ex:
        parts = list(ex.map(one, tasks))
    out = [np.zeros(case[("G1", "G2", "G3")[k]].shape) for k in range(3)]
    for (k, i), g in zip(tasks, parts):
        T = case["T"]
        out[k].reshape(T * out[k].shape[1], -1)[i] = g.reshape(T * g.shape[1], -1)[i]
    return out


def test_backward_config4_full_hottest_slices(lib, orc):
    # The hot-prefix workload at full size as a training step on the R = 64 MFMA
    # backward (forward with grouping, backward reusing it, then the fused update):
    # the most-used slice of each core (the hottest prefix's G1 and G2 slices and the
    # most-used G3 slice) plus two random slices per core, against the oracle.
    case = ttgen.make(4, with_grad=True)
    T, B, lr = case["T"], case["B"], 0.01
    M = int(case["idx"].size)
    want = _hottest_slices(case, extra_tables=(0,))
    _say(f"[bwd] config4 full, hottest + random slices ({sum(int(w.sum()) for w in want)} slices)")
    emb = _make(lib, case)
    assert lib.N.tt_emb_kernel_uses_mfma(emb.handle, lib.N.KERNELS["bwd_fused"], M)
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.forward(*G, idx, off, num_bags=B)
    grads = emb.backward(*G, idx, off, dV, num_bags=B, reuse_grouping=True)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    from concurrent.futures import ThreadPoolExecutor

    with ThreadPoolExecutor(2) as ex:  # the signed and the absolute case side by side
        ref_f = ex.submit(_oracle_backward_by_slice, orc, case, want)
        mag_f = ex.submit(_oracle_backward_by_slice, orc, abs_case(case), want)
        ref, mag = ref_f.result(), mag_f.result()
    for k in range(3):
        g = grads[k].cpu().numpy()
        assert_close(f"dG{k + 1} config4 full (hottest slices)", _sel(g, T, want[k]), _sel(ref[k], T, want[k]),
                     _sel(mag[k], T, want[k]))
    del grads
    _say("[bwd+sgd] config4 full, same slices")
    emb.backward_sgd(*G, idx, off, dV, lr, num_bags=B, reuse_grouping=True)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    for k, cname in enumerate(("G1", "G2", "G3")):
        new = _sel(G[k].cpu().numpy().astype(np.float64), T, want[k])
        exp = _sel(orc.sgd(case[cname], ref[k], lr), T, want[k])
        bound = TOL * lr * _sel(mag[k], T, want[k]) + 2.0 ** -23 * np.abs(exp)
        assert np.all(np.abs(new - exp) <= bound + 1e-30), cname


def test_sgd_step(lib, orc):
    case = ttgen.make(5, bags=32)
    _say("[sgd] config5 B=32")
    emb, G, grads, dV = gpu_train(lib, case)
    lr = case["lr"]
    emb.sgd(*G, *grads, lr)
    torch.cuda.synchronize()
    ref = orc.backward(case)[:3]
    mag = orc.backward(abs_case(case))[:3]
    for k, name in enumerate(("G1", "G2", "G3")):
        new = G[k].cpu().numpy().astype(np.float64)
        exp = orc.sgd(case[name], ref[k], lr)
        # gradient error scaled by lr plus one fp32 rounding of the updated value
        bound = TOL * lr * mag[k] + 2.0 ** -23 * np.abs(exp)
        assert np.all(np.abs(new - exp) <= bound + 1e-30), name


def _check_sgd(orc, case, G, lr, name):
    ref = orc.backward(case)[:3]
    mag = orc.backward(abs_case(case))[:3]
    for k, cname in enumerate(("G1", "G2", "G3")):
        new = G[k].cpu().numpy().astype(np.float64)
        exp = orc.sgd(case[cname], ref[k], lr)
        # gradient error scaled by lr plus one fp32 rounding of the updated value
        bound = TOL * lr * mag[k] + 2.0 ** -23 * np.abs(exp)
        assert np.all(np.abs(new - exp) <= bound + 1e-30), f"{cname} {name}"


@pytest.mark.parametrize("reuse", [True, False])
@pytest.mark.parametrize("k", [0, 4, 5, 7])
def test_backward_sgd_fused(lib, orc, k, reuse):
    # one call for backward + SGD leaves the cores where backward then sgd would
    # (the MFMA shapes update inside the reductions, the others via workspace gradients)
    c = dict(TINY[k])
    case = ttgen.tiny(5000 + k, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    _say(f"[bwd+sgd] tiny{k} reuse_grouping={reuse}")
    emb = _make(lib, case)
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    lr = 0.01
    if reuse:
        emb.group(idx, off, num_bags=case["B"])
    emb.backward_sgd(*G, idx, off, dV, lr, num_bags=case["B"], reuse_grouping=reuse)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    _check_sgd(orc, case, G, lr, f"tiny{k}")


def test_backward_sgd_fused_config5(lib, orc):
    case = ttgen.make(5, bags=32)
    _say("[bwd+sgd] config5 B=32")
    emb = _make(lib, case)
    G, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    emb.backward_sgd(*G, idx, off, dV, case["lr"], num_bags=case["B"], reuse_grouping=False)
    torch.cuda.synchronize()
    _check_sgd(orc, case, G, case["lr"], "config5 B=32")


def test_autograd_module(lib, orc):
    # torch autograd through the library: forward output and .grad of the three
    # core parameters against the oracle, for L = sum <dV, out>
    case = ttgen.tiny(6001, 2, (20, 30, 40), (4, 4, 8), 32, B=60, max_len=12, zipf=1.1)
    _say("[autograd] T=2 n=(20,30,40) d=(4,4,8) R=32")
    M = int(case["idx"].size)
    mod = lib.TTEmbeddingBag(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=M,
                             max_bags=case["B"])
    with torch.no_grad():
        for name in ("G1", "G2", "G3"):
            getattr(mod, name).copy_(torch.from_numpy(case[name]))
    _, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    out = mod(idx, off)
    # another lookup on the same handle in between: backward must regroup its own indices
    other = torch.randint(0, case["N"], (idx.numel(),), device=idx.device)
    mod.emb.group(other, off, num_bags=case["B"])
    (out * dV).sum().backward()
    torch.cuda.synchronize()
    D = int(np.prod(case["d"]))
    ref_v, _ = orc.forward(case)
    mag_v, _ = orc.forward(abs_case(case))
    assert_close("autograd out", out.detach().cpu().numpy().reshape(-1, D), ref_v, mag_v)
    ref = orc.backward(case)[:3]
    mag = orc.backward(abs_case(case))[:3]
    for k, name in enumerate(("G1", "G2", "G3")):
        assert_close(f"autograd {name}.grad", getattr(mod, name).grad.cpu().numpy(), ref[k], mag[k])
    # the fused training step on the module matches backward + sgd
    mod2 = lib.TTEmbeddingBag(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=M,
                              max_bags=case["B"])
    with torch.no_grad():
        for name in ("G1", "G2", "G3"):
            getattr(mod2, name).copy_(torch.from_numpy(case[name]))
    mod2(idx, off)
    mod2.step_fused(idx, off, dV, 0.01)
    torch.cuda.synchronize()
    _check_sgd(orc, case, [mod2.G1.data, mod2.G2.data, mod2.G3.data], 0.01, "module step_fused")


def _run_mode(lib, case, **kw):
    M = int(case["idx"].size)
    emb = lib.TTEmbedding(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=max(M, 1),
                          max_bags=max(int(case["B"]), 1), **kw)
    G, idx, off = _dev(case)
    out = emb.forward(*G, idx, off, num_bags=case["B"])
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = emb.backward(*G, idx, off, dV, num_bags=case["B"], reuse_grouping=True)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    D = int(np.prod(case["d"]))
    return out.cpu().numpy().reshape(-1, D), [g.cpu().numpy() for g in grads], emb


@pytest.mark.parametrize("which", ["hot_r64", "hot_generic", "mfma", "mfma_d32"])
def test_schedules_same_results(lib, orc, which):
    # Section 4.4 ablation modes compute the same function: static shares, stealing,
    # stealing with the checkpointed intermediate (hot prefix groups spanning
    # several chunks on the generic kernels), and the static prefix mapping (each
    # group one work unit)
    if which == "hot_r64":
        case = ttgen.make(4, bags=256, with_grad=True)
    elif which == "hot_generic":
        # d = (4, 4, 4), R = 16: generic kernels both ways, groups of about 60 slices
        case = _hot_prefix_case(7006, 1, (3, 2, 2000), B=300, hot=[(1, 1), (2, 0)], per_bag=24,
                                d=(4, 4, 4), R=16)
    elif which == "mfma_d32":
        # D = 32 = (4, 4, 2), R = 32: twelve prefixes of one (table, i2) run with nearly all
        # suffixes, groups of 7-8 slices across chunk ends (whole groups under "group")
        case = _hot_prefix_case(7008, 2, (12, 2, 250), B=400, hot=[(i1, 0) for i1 in range(12)], per_bag=20,
                                d=(4, 4, 2), R=32)
    else:
        c = dict(TINY[4])
        case = ttgen.tiny(7004, c.pop("T"), c.pop("n"), c.pop("d"), c.pop("R"), **c)
    ref_v, _ = orc.forward(case)
    mag_v, _ = orc.forward(abs_case(case))
    ref = orc.backward(case)[:3]
    mag = orc.backward(abs_case(case))[:3]
    for sched in ("steal", "static", "steal_ckpt", "group"):
        _say(f"[sched] {which} {sched}")
        V, grads, emb = _run_mode(lib, case, sched=sched)
        assert_close(f"forward {which} {sched}", V, ref_v, mag_v)
        for k in range(3):
            assert_close(f"dG{k + 1} {which} {sched}", grads[k], ref[k], mag[k])
        if which == "hot_generic" and sched == "steal_ckpt":
            # the workload must exercise the checkpoint: some prefix group spans chunks
            g = emb.debug_grouping(int(case["idx"].size))
            assert np.max(np.diff(g["pg_start"])) > 8 * 32
