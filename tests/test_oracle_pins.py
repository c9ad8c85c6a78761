"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Nothing here compares the oracle with itself: each test checks it against a
textbook routine, a closed form, an invariant of the operator, or brute force
over the fully reconstructed table.  The paper (FlowTT) prints no worked
numeric example, so no test uses numbers from it.
"""
import numpy as np
import pytest
import torch

import ttgen

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _full_table(case):
    """Brute force: every row of every table, W[t][g][D], by one einsum over the
    whole TT tensor (a library contraction; no digit arithmetic is written here:
    the C-order reshape enumerates rows and outputs)."""
    T, n, d = case["T"], case["n"], case["d"]
    G1 = case["G1"].astype(np.float64)  # [T][n1][d1][R]
    G2 = case["G2"].astype(np.float64)  # [T][n2][R][d2][R]
    G3 = case["G3"].astype(np.float64)  # [T][n3][R][d3]
    W = np.einsum("tpxa,tqayb,trbz->tpqrxyz", G1, G2, G3)
    D = d[0] * d[1] * d[2]
    return W.reshape(T, n[0] * n[1] * n[2], D)


def _bags(case):
    T, B = case["T"], case["B"]
    M = case["idx"].size
    if case["offsets"] is None:
        return np.arange(M)
    lens = np.diff(case["offsets"])
    return np.repeat(np.arange(T * B), lens)


def _brute_forward(case):
    W = _full_table(case)
    T, B, N = case["T"], case["B"], case["N"]
    D = W.shape[2]
    bag = _bags(case)
    V = np.zeros((T * B, D))
    for o, g in enumerate(case["idx"]):
        if 0 <= g < N:
            V[bag[o]] += W[bag[o] // B, g]
    return V


TINY_SHAPES = [
    dict(T=1, n=(3, 4, 5), d=(2, 3, 2), R=3),
    dict(T=2, n=(2, 3, 7), d=(1, 2, 4), R=5),
    dict(T=3, n=(1, 5, 2), d=(3, 1, 1), R=1),
    dict(T=1, n=(7, 1, 3), d=(2, 2, 2), R=4),
    dict(T=2, n=(4, 4, 4), d=(1, 1, 3), R=2),
]


@pytest.mark.parametrize("k", range(len(TINY_SHAPES)))
def test_forward_matches_brute_force(orc, k):
    sh = TINY_SHAPES[k]
    case = ttgen.tiny(100 + k, sh["T"], sh["n"], sh["d"], sh["R"], B=6, max_len=5)
    V, invalid = orc.forward(case)
    assert invalid == 0
    ref = _brute_forward(case)
    np.testing.assert_allclose(V, ref, rtol=1e-12, atol=1e-12)


def test_forward_with_padding_rows_and_invalid(orc):
    # N < n1*n2*n3: indices in [N, prod) and negatives are invalid and contribute nothing
    case = ttgen.tiny(7, 2, (3, 4, 5), (2, 2, 2), 3, B=5, max_len=6, N=50)
    idx = case["idx"].copy()
    sel = np.arange(idx.size)[::4]
    idx[sel] = np.choose(sel % 3, [55, -3, 50])  # 50 == N is the first invalid row
    case["idx"] = idx
    V, invalid = orc.forward(case)
    assert invalid == int(np.sum((idx < 0) | (idx >= 50)))
    ref = _brute_forward(case)
    np.testing.assert_allclose(V, ref, rtol=1e-12, atol=1e-12)


def test_digits_match_unravel_index(orc):
    rng = np.random.default_rng(3)
    for n in [(3, 4, 5), (1, 7, 2), (200, 200, 250), (400, 500, 500), (100, 100, 100), (5, 1, 1)]:
        N = n[0] * n[1] * n[2]
        g = rng.integers(0, N, size=2000)
        g[:3] = [0, N - 1, min(N - 1, n[2])]
        got = orc.digits(g, n)
        ref = np.stack(np.unravel_index(g, n), axis=1)
        assert np.array_equal(got, ref)


def _rank2_cores(T, n, d, R):
    """Rank-2 additive TT cores whose row g reconstructs to E[g][j] = g*D + j."""
    assert R >= 2
    n1, n2, n3 = n
    d1, d2, d3 = d
    D = d1 * d2 * d3
    G1 = np.zeros((T, n1, d1, R), np.float32)
    G2 = np.zeros((T, n2, R, d2, R), np.float32)
    G3 = np.zeros((T, n3, R, d3), np.float32)
    for i1 in range(n1):
        for j1 in range(d1):
            G1[:, i1, j1, 0] = i1 * n2 * n3 * D + j1 * d2 * d3
            G1[:, i1, j1, 1] = 1
    for i2 in range(n2):
        for j2 in range(d2):
            G2[:, i2, 0, j2, 0] = 1
            G2[:, i2, 1, j2, 0] = i2 * n3 * D + j2 * d3
            G2[:, i2, 1, j2, 1] = 1
    for i3 in range(n3):
        for j3 in range(d3):
            G3[:, i3, 0, j3] = 1
            G3[:, i3, 1, j3] = i3 * D + j3
    return G1, G2, G3


@pytest.mark.parametrize("shape", [((3, 4, 5), (2, 3, 2), 2), ((100, 100, 100), (2, 2, 4), 8),
                                   ((6, 1, 9), (1, 4, 1), 3)])
def test_rank2_closed_form_row(orc, shape):
    n, d, R = shape
    G1, G2, G3 = _rank2_cores(1, n, d, R)
    N = n[0] * n[1] * n[2]
    D = d[0] * d[1] * d[2]
    case = dict(T=1, N=N, n=n, d=d, R=R, B=1, G1=G1, G2=G2, G3=G3)
    rng = np.random.default_rng(5)
    gs = np.unique(np.concatenate([[0, N - 1], rng.integers(0, N, 50)]))
    for g in gs:
        E = orc.row(case, 0, int(g))
        assert np.array_equal(E, g * D + np.arange(D, dtype=np.float64)), g


def test_rank1_kronecker(orc):
    n, d = (3, 2, 4), (2, 3, 2)
    case = ttgen.tiny(11, 1, n, d, 1, B=1, max_len=1)
    for g in range(n[0] * n[1] * n[2]):
        i1, i2, i3 = np.unravel_index(g, n)
        a = case["G1"][0, i1, :, 0].astype(np.float64)
        b = case["G2"][0, i2, 0, :, 0].astype(np.float64)
        c = case["G3"][0, i3, 0, :].astype(np.float64)
        ref = np.kron(a, np.kron(b, c))
        np.testing.assert_allclose(orc.row(case, 0, g), ref, rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("k", range(len(TINY_SHAPES)))
def test_backward_matches_autograd(orc, k):
    sh = TINY_SHAPES[k]
    case = ttgen.tiny(200 + k, sh["T"], sh["n"], sh["d"], sh["R"], B=6, max_len=5)
    dG1, dG2, dG3, invalid = orc.backward(case)
    assert invalid == 0
    # independent path: torch float64 autograd through the full-table einsum and a bag sum
    G1 = torch.tensor(case["G1"], dtype=torch.float64, requires_grad=True)
    G2 = torch.tensor(case["G2"], dtype=torch.float64, requires_grad=True)
    G3 = torch.tensor(case["G3"], dtype=torch.float64, requires_grad=True)
    T, n, d, B = case["T"], case["n"], case["d"], case["B"]
    W = torch.einsum("tpxa,tqayb,trbz->tpqrxyz", G1, G2, G3).reshape(T, -1, d[0] * d[1] * d[2])
    bag = torch.tensor(_bags(case))
    idx = torch.tensor(case["idx"])
    rows = W[bag // B, idx]
    V = torch.zeros(T * B, W.shape[2], dtype=torch.float64).index_add(0, bag, rows)
    L = (V * torch.tensor(case["dV"], dtype=torch.float64).reshape(T * B, -1)).sum()
    L.backward()
    for got, ref in ((dG1, G1.grad), (dG2, G2.grad), (dG3, G3.grad)):
        np.testing.assert_allclose(got, ref.numpy(), rtol=1e-11, atol=1e-12)


def test_euler_identity(orc):
    # V is linear in each core, so <dG_k, G_k> = <dV, V> for every k
    case = ttgen.tiny(31, 2, (4, 5, 6), (2, 2, 3), 4, B=9, max_len=6, zipf=1.1)
    V, _ = orc.forward(case)
    dG1, dG2, dG3, _ = orc.backward(case)
    lhs = float(np.sum(case["dV"].reshape(V.shape).astype(np.float64) * V))
    for dG, G in ((dG1, case["G1"]), (dG2, case["G2"]), (dG3, case["G3"])):
        rhs = float(np.sum(dG * G.astype(np.float64)))
        assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs)), (lhs, rhs)


def test_single_entry_gradients_are_exact_differences(orc):
    # L is affine in any single core entry x: dL/dx = L(x=1) - L(x=0)
    case = ttgen.tiny(41, 2, (3, 3, 4), (2, 1, 2), 3, B=5, max_len=4)
    dG = orc.backward(case)[:3]
    dV = case["dV"].reshape(case["T"] * case["B"], -1).astype(np.float64)
    rng = np.random.default_rng(0)

    def loss(c):
        V, _ = orc.forward(c)
        return float(np.sum(V * dV))

    for k, name in enumerate(("G1", "G2", "G3")):
        for _ in range(4):
            pos = tuple(int(rng.integers(0, s)) for s in case[name].shape)
            c1 = dict(case)
            c0 = dict(case)
            c1[name] = case[name].copy()
            c0[name] = case[name].copy()
            c1[name][pos] = 1.0
            c0[name][pos] = 0.0
            fd = loss(c1) - loss(c0)
            assert abs(fd - dG[k][pos]) <= 1e-11 * max(1.0, abs(fd)), (name, pos, fd, dG[k][pos])


def test_linearity_and_symmetries(orc):
    case = ttgen.tiny(51, 2, (3, 4, 2), (2, 2, 2), 3, B=7, max_len=5)
    dG = orc.backward(case)[:3]
    c2 = dict(case)
    c2["dV"] = case["dV"] * 2.0
    dG2x = orc.backward(c2)[:3]
    for a, b in zip(dG, dG2x):
        assert np.array_equal(2.0 * a, b)
    V, _ = orc.forward(case)
    # permuting occurrences inside each bag leaves V unchanged (up to rounding)
    off = case["offsets"]
    idx = case["idx"].copy()
    for gb in range(len(off) - 1):
        idx[off[gb]:off[gb + 1]] = idx[off[gb]:off[gb + 1]][::-1]
    cp = dict(case)
    cp["idx"] = idx
    np.testing.assert_allclose(orc.forward(cp)[0], V, rtol=1e-13, atol=1e-14)
    # duplicating every occurrence doubles V
    lens = np.diff(off)
    cd = dict(case)
    cd["idx"] = np.repeat(case["idx"], 2)
    cd["offsets"] = np.concatenate([[0], np.cumsum(2 * lens)])
    np.testing.assert_allclose(orc.forward(cd)[0], 2 * V, rtol=1e-13, atol=1e-14)
    # bag sums of a concatenation of single-row bags equal the rows
    V1, _ = orc.forward(dict(case, offsets=None, B=case["idx"].size // case["T"],
                             idx=case["idx"][: (case["idx"].size // case["T"]) * case["T"]]))
    assert V1.shape[0] == (case["idx"].size // case["T"]) * case["T"]


def test_sgd_step(orc):
    # one SGD step on the linear loss <dG, G> lowers it by exactly lr*|dG|^2 (up to rounding)
    rng = np.random.default_rng(9)
    G = rng.standard_normal(1000).astype(np.float32)
    dG = rng.standard_normal(1000)
    out = orc.sgd(G, dG, 0.01)
    before = float(np.dot(dG, G.astype(np.float64)))
    after = float(np.dot(dG, out))
    assert abs((before - after) - 0.01 * float(np.dot(dG, dG))) < 1e-10
    assert np.array_equal(orc.sgd(G, dG, 0.0), G.astype(np.float64))


def _numpy_grouping(case):
    T, B, N, n = case["T"], case["B"], case["N"], case["n"]
    idx = case["idx"]
    bag = _bags(case)
    tab = bag // B
    valid = (idx >= 0) & (idx < N)
    pos = np.flatnonzero(valid)
    keys = tab[pos] * N + idx[pos]
    order = np.argsort(keys, kind="stable")
    uniq, first, inv_v = np.unique(keys, return_index=True, return_inverse=True)
    inv = np.full(idx.size, -1, np.int64)
    inv[pos] = inv_v
    counts = np.bincount(inv_v, minlength=uniq.size)
    occ_start = np.concatenate([[0], np.cumsum(counts)])
    ut, ug = np.divmod(uniq, N)
    d = np.stack(np.unravel_index(ug, n), axis=1) if ug.size else np.zeros((0, 3), np.int64)
    pref = ut * (n[0] * n[1]) + d[:, 0] * n[1] + d[:, 1]
    heads = np.flatnonzero(np.concatenate([[True], np.diff(pref) != 0])) if pref.size else np.zeros(0, np.int64)
    return dict(uniq_t=ut, uniq_g=ug, inv=inv, occ_start=occ_start, occ_pos=pos[order],
                pg_start=np.concatenate([heads, [uniq.size]]), pg_t=ut[heads],
                pg_q=d[heads, 0] * n[1] + d[heads, 1])


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_grouping_matches_numpy(orc, seed):
    case = ttgen.tiny(300 + seed, 3, (4, 3, 5), (1, 1, 1), 1, B=40, max_len=6, zipf=1.2, grad=False)
    if seed == 3:
        case["idx"][::7] = -1
    got = orc.grouping(case)
    ref = _numpy_grouping(case)
    for key in ref:
        assert np.array_equal(got[key], ref[key]), key


def test_grouping_prefix_groups_split_at_table_boundaries(orc):
    # n1 = n2 = 1: every row has prefix 0, so each table is exactly one prefix group
    case = ttgen.tiny(12, 3, (1, 1, 6), (1, 1, 1), 1, B=8, max_len=3, empty_bags=False, grad=False)
    got = orc.grouping(case)
    assert got["P"] == 3
    assert np.array_equal(got["pg_t"], [0, 1, 2])
    ref = _numpy_grouping(case)
    for key in ref:
        assert np.array_equal(got[key], ref[key]), key


def test_grouping_single_index_bags(orc):
    case = ttgen.tiny(9, 2, (5, 5, 5), (1, 1, 1), 1, B=64, single=True, grad=False, zipf=1.05)
    got = orc.grouping(case)
    ref = _numpy_grouping(case)
    for key in ref:
        assert np.array_equal(got[key], ref[key]), key


# ---------------------------------------------------------------------------
# The oracle's subset options, which the full-size GPU checks rely on: a bag
# list computes exactly those bags of the full forward, and slice masks keep
# every occurrence that adds to a wanted slice (in the same order), so the
# wanted slices' gradients are those of the full backward, bit for bit.
# ---------------------------------------------------------------------------
def _dup_invalid_case(seed, T=3, n=(4, 3, 5), d=(2, 1, 3), R=3, B=9):
    case = ttgen.tiny(seed, T, n, d, R, B=B, max_len=6, N=n[0] * n[1] * n[2] - 3)
    idx = case["idx"].copy()
    idx[::7] = idx[0]             # repeated rows inside and across bags
    idx[3::11] = case["N"] + 1    # padding rows: invalid
    idx[5::13] = -1
    case["idx"] = idx
    return case


@pytest.mark.parametrize("seed", [61, 62])
def test_forward_bag_subset_is_the_full_forward_on_those_bags(orc, seed):
    case = _dup_invalid_case(seed)
    V, inv_all = orc.forward(case)
    nb = case["T"] * case["B"]
    rng = np.random.default_rng(seed)
    bags = np.concatenate([rng.choice(nb, 7, replace=False), [nb - 1, 0, 3, 3]])  # unsorted, repeated
    Vs, _ = orc.forward(case, bags=bags)
    assert np.array_equal(Vs, V[bags])
    assert inv_all > 0


def _masks(rng, T, n, count):
    out = []
    for nk in n:
        m = np.zeros(T * nk, np.uint8)
        m[rng.choice(T * nk, min(count, T * nk), replace=False)] = 1
        out.append(m)
    return out


@pytest.mark.parametrize("seed", [71, 72, 73])
def test_backward_slice_masks_keep_the_wanted_slices_exact(orc, seed):
    case = _dup_invalid_case(seed)
    T, n = case["T"], case["n"]
    full = orc.backward(case)
    rng = np.random.default_rng(seed)
    want = _masks(rng, T, n, 2)
    if seed == 73:
        want[1] = None  # a core with no mask: only the others select
    part = orc.backward(case, want=want)
    assert part[3] == full[3]
    for k in range(3):
        if want[k] is None:
            continue
        sel = np.flatnonzero(want[k])
        g = part[k].reshape(T * n[k], -1)[sel]
        r = full[k].reshape(T * n[k], -1)[sel]
        assert np.array_equal(g, r), k
    # occurrences touching no wanted slice were skipped: some unwanted slice differs
    diffs = [np.any(part[k] != full[k]) for k in range(3)]
    assert any(diffs)


@pytest.mark.parametrize("seed,L", [(81, 4), (82, 5), (83, 2)])
def test_backward_n_slice_masks_keep_the_wanted_slices_exact(orc, seed, L):
    n = {2: (6, 5), 4: (3, 2, 4, 3), 5: (2, 3, 2, 2, 3)}[L]
    d = {2: (2, 3), 4: (2, 1, 2, 2), 5: (1, 2, 1, 2, 2)}[L]
    case = ttgen.tiny_n(seed, 2, n, d, 3, 11, max_len=6)
    full, _ = orc.backward_n(case)
    rng = np.random.default_rng(seed)
    T = case["T"]
    want = _masks(rng, T, n, 1)
    part, _ = orc.backward_n(case, want=want)
    for k in range(L):
        sel = np.flatnonzero(want[k])
        g = part[k].reshape(T * n[k], -1)[sel]
        r = full[k].reshape(T * n[k], -1)[sel]
        assert np.array_equal(g, r), k
    # a list of no masks selects nothing away: the full backward
    none, _ = orc.backward_n(case, want=[None] * L)
    assert all(np.array_equal(none[k], full[k]) for k in range(L))
    with pytest.raises(ValueError):
        orc.backward_n(case, want=want[:-1])
