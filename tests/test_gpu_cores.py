"""GPU parity of the L-core calls (tt_emb_forward_n / backward_n / sgd_n) against
the L-core oracle: L = 2 .. 8, the MFMA view shape, L = 3 against the three-core
calls, edge cases, a full-size L = 4 workload on sampled bags and, for its
gradients, the Euler identity <dG_k, G_k> = <dV, V> of a function linear in
each core."""
import sys

import numpy as np
import pytest
import torch

import ttgen
from tests._util import TOL, assert_close

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


def _abs_n(case):
    c = dict(case)
    c["cores"] = [np.abs(G) for G in case["cores"]]
    if "dV" in case:
        c["dV"] = np.abs(case["dV"])
    return c


def _make(lib, case, **kw):
    M = int(case["idx"].size)
    return lib.TTEmbedding(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=max(M, 1),
                           max_bags=max(int(case["B"]), 1), **kw)


def _dev(case):
    cores = [torch.from_numpy(np.ascontiguousarray(G)).cuda() for G in case["cores"]]
    idx = torch.from_numpy(np.ascontiguousarray(case["idx"], dtype=np.int64)).cuda()
    off = None if case["offsets"] is None else torch.from_numpy(np.ascontiguousarray(case["offsets"])).cuda()
    return cores, idx, off


def _run(lib, case, **kw):
    emb = _make(lib, case, **kw)
    cores, idx, off = _dev(case)
    out = emb.forward_n(cores, idx, off, num_bags=case["B"])
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = emb.backward_n(cores, idx, off, dV, num_bags=case["B"], reuse_grouping=True)
    torch.cuda.synchronize()
    D = int(np.prod(case["d"]))
    return emb, out.cpu().numpy().reshape(-1, D), [g.cpu().numpy() for g in grads]


def _check(orc, case, V, grads, name):
    ref, _ = orc.forward_n(case)
    mag, _ = orc.forward_n(_abs_n(case))
    assert_close(f"{name} forward", V, ref, mag)
    dref, _ = orc.backward_n(case)
    dmag, _ = orc.backward_n(_abs_n(case))
    for k in range(len(grads)):
        assert_close(f"{name} dG{k + 1}", grads[k], dref[k], dmag[k])


CASES = [
    dict(T=2, n=(30, 40), d=(4, 8), R=16, B=50, max_len=8),
    dict(T=1, n=(7, 5), d=(3, 1), R=3, B=20, max_len=5),
    dict(T=2, n=(3, 4, 5, 6), d=(2, 1, 3, 2), R=5, B=40, max_len=6),
    dict(T=2, n=(5, 4, 20, 30), d=(2, 2, 4, 8), R=32, B=200, max_len=16, zipf=1.1),  # MFMA view (4, 4, 8), R = 32
    dict(T=2, n=(4, 5, 6, 7), d=(2, 2, 2, 4), R=64, B=60, max_len=10),  # R = 64
    dict(T=2, n=(2, 3, 4, 5, 6), d=(1, 2, 2, 2, 2), R=8, B=60, max_len=8),
    dict(T=1, n=(2, 2, 3, 2, 3, 4), d=(2, 1, 2, 1, 2, 2), R=4, B=30, max_len=6),
    dict(T=2, n=(2,) * 8, d=(1, 2, 1, 2, 1, 2, 1, 2), R=3, B=25, max_len=5),
    dict(T=2, n=(2, 2, 2, 3, 4), d=(4, 4, 2, 1, 1), R=16, B=40, max_len=6),  # wide merged core: d1' = 32
    dict(T=2, n=(5, 4, 3, 2, 2), d=(1, 2, 1, 2, 2), R=2, B=40, max_len=6),  # 20 parents: several per-level chunks
    dict(T=1, n=(2, 2, 2, 2, 2), d=(4, 4, 2, 1, 1), R=64, B=20, max_len=4),  # R = 64: split chunks of 2 parents
    dict(T=2, n=(5, 4, 20, 30), d=(2, 2, 4, 2), R=32, B=200, max_len=16, zipf=1.1),  # MFMA view (4, 4, 2): D = 32
]


@pytest.mark.parametrize("k", range(len(CASES)))
def test_forward_backward_n(lib, orc, k):
    p = CASES[k]
    case = ttgen.tiny_n(7000 + k, p["T"], p["n"], p["d"], p["R"], p["B"], max_len=p["max_len"], zipf=p.get("zipf"))
    _say(f"[cores] L={len(p['n'])} T={p['T']} n={p['n']} d={p['d']} R={p['R']} B={p['B']} M={case['idx'].size}")
    emb, V, grads = _run(lib, case)
    assert emb.check_errors() == 0
    _check(orc, case, V, grads, f"L={len(p['n'])}")


@pytest.mark.parametrize("sched", ["static", "steal_ckpt"])
@pytest.mark.parametrize("reuse", ["prefix", "none"])
def test_modes_n(lib, orc, sched, reuse):
    case = ttgen.tiny_n(7100, 2, (3, 4, 5, 6), (2, 1, 3, 2), 5, 40, max_len=6)
    _say(f"[cores modes] sched={sched} reuse={reuse}")
    _, V, grads = _run(lib, case, sched=sched, reuse=reuse)
    _check(orc, case, V, grads, f"L=4 {sched} {reuse}")


def test_three_cores_through_n_calls_match_the_three_core_calls(lib, orc):
    case = ttgen.tiny_n(7200, 2, (20, 30, 40), (4, 4, 8), 32, 60, max_len=12, zipf=1.1)
    _say("[cores L=3] n=(20,30,40) d=(4,4,8) R=32")
    emb, V, grads = _run(lib, case)
    emb3 = _make(lib, case)
    cores, idx, off = _dev(case)
    V3 = emb3.forward(*cores, idx, off, num_bags=case["B"])
    torch.cuda.synchronize()
    assert np.array_equal(V, V3.cpu().numpy().reshape(V.shape))
    _check(orc, case, V, grads, "L=3")


def test_empty_batch_and_untouched_rows(lib):
    # no index at all: zero output and zero gradients for every core
    case = ttgen.tiny_n(7300, 2, (3, 4, 5, 6), (2, 1, 3, 2), 5, 10, max_len=0)
    assert case["idx"].size == 0
    _say("[cores edge] empty batch L=4")
    emb = lib.TTEmbedding(2, case["N"], case["n"], case["d"], 5, max_indices=16, max_bags=10)
    cores, idx, off = _dev(case)
    out = emb.forward_n(cores, idx, off, num_bags=10)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = [torch.full(G.shape, 7.0, device="cuda") for G in cores]
    emb.backward_n(cores, idx, off, dV, num_bags=10, grads=grads, reuse_grouping=True)
    torch.cuda.synchronize()
    assert not out.any()
    assert all(not g.any() for g in grads)


def test_invalid_indices_n(lib, orc):
    # N below the product of the factors: indices in [N, prod) are flagged and skipped
    case = ttgen.tiny_n(7400, 2, (3, 4, 5, 6), (2, 1, 3, 2), 5, 40, max_len=6)
    prod = case["N"]
    case = dict(case, N=prod - 50)
    idx = case["idx"] % (prod - 50)
    idx[::7] = prod - 1 - (np.arange(idx[::7].size) % 50)
    case["idx"] = idx
    _say("[cores edge] invalid indices L=4")
    emb, V, grads = _run(lib, case)
    assert emb.check_errors() == lib.N.TT_EMB_ERANGE
    ref, inv = orc.forward_n(case)
    assert inv == idx[::7].size
    _check(orc, case, V, grads, "invalid")


def _sub_bags(case, per_table, seed):
    """The bags picked (the same count per table) as a case of their own."""
    rng = np.random.default_rng(seed)
    T, B = case["T"], case["B"]
    off = case["offsets"]
    idx, lens, dV = [], [], []
    for t in range(T):
        for b in np.sort(rng.choice(B, per_table, replace=False)):
            gb = t * B + int(b)
            idx.append(case["idx"][off[gb]:off[gb + 1]])
            lens.append(off[gb + 1] - off[gb])
            dV.append(case["dV"][t, b])
    o = np.zeros(T * per_table + 1, np.int64)
    np.cumsum(lens, out=o[1:])
    sub = dict(case, B=per_table, idx=np.concatenate(idx), offsets=o,
               dV=np.stack(dV).reshape(T, per_table, -1))
    return sub


def test_full_size_four_cores(lib, orc):
    # the 8-table training workload with its 10^7 rows split over four cores:
    # n = (20, 10, 200, 250), d = (2, 2, 4, 8), R = 32 (view (200, 200, 250), (4, 4, 8))
    base = ttgen.make(5, with_grad=True)
    n, d, R, T = (20, 10, 200, 250), (2, 2, 4, 8), 32, base["T"]
    rng = np.random.default_rng(7500)
    cores = [(rng.standard_normal(s) * 0.5).astype(np.float32) for s in ttgen.core_shapes_n(T, n, d, R)]
    case = dict(T=T, N=base["N"], L=4, n=n, d=d, R=R, B=base["B"], cores=cores, idx=base["idx"],
                offsets=base["offsets"], dV=base["dV"])
    _say(f"[cores full] T={T} n={n} d={d} R={R} B={case['B']} M={case['idx'].size}")
    emb = _make(lib, case)
    dcores, idx, off = _dev(case)
    out = emb.forward_n(dcores, idx, off, num_bags=case["B"])
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = emb.backward_n(dcores, idx, off, dV, num_bags=case["B"])
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    # sampled bags against the oracle
    sub = _sub_bags(case, 24, 7501)
    ref, _ = orc.forward_n(sub)
    mag, _ = orc.forward_n(_abs_n(sub))
    picked = []
    rng = np.random.default_rng(7501)
    for t in range(T):
        for b in np.sort(rng.choice(case["B"], 24, replace=False)):
            picked.append(t * case["B"] + int(b))
    V = out.cpu().numpy().reshape(T * case["B"], -1)
    assert_close("full L=4 sampled bags", V[picked], ref, mag)
    # gradients: <dG_k, G_k> = <dV, V> for every core (V linear in each core)
    Vd = out.double()
    lhs = float((dV.double().reshape(Vd.shape) * Vd).sum())
    for k in range(4):
        rhs = float((grads[k].double() * dcores[k].double()).sum())
        scale = float((grads[k].double().abs() * dcores[k].double().abs()).sum())
        assert abs(lhs - rhs) <= TOL * scale, (k, lhs, rhs, scale)
    # and element by element on sampled slices of every core: the most-used slice of
    # each core in the first and last table, and a random one in the first table
    want = _sampled_slices_n(case, (0, T - 1), seed=7502)
    _say(f"[cores full] L=4 gradients on {[int(w.sum()) for w in want]} slices per core")
    ref = _oracle_backward_n_by_table(orc, case, want)
    mag = _oracle_backward_n_by_table(orc, _abs_n(case), want)
    for k in range(4):
        sel = np.flatnonzero(want[k])
        g = grads[k].cpu().numpy()
        assert_close(f"full L=4 dG{k + 1} (sampled slices)", g.reshape(T * n[k], -1)[sel],
                      ref[k].reshape(T * n[k], -1)[sel], mag[k].reshape(T * n[k], -1)[sel])


def _part_case_n(case, t, b0, b1):
    """Bags [b0, b1) of table t of an L-core case as a one-table case of its own."""
    B = case["B"]
    off = case["offsets"]
    lo, hi = int(off[t * B + b0]), int(off[t * B + b1])
    return dict(case, T=1, B=b1 - b0, idx=case["idx"][lo:hi], offsets=off[t * B + b0:t * B + b1 + 1] - lo,
                cores=[G[t:t + 1] for G in case["cores"]], dV=case["dV"][t:t + 1, b0:b1])


def _oracle_backward_n_by_table(orc, case, want, splits=4):
    """orc.backward_n with slice masks on a thread pool: each table with a wanted slice
    (tables are independent) in `splits` bag ranges, each a case of its own; the
    ranges' gradients are added in double and stacked over tables."""
    from concurrent.futures import ThreadPoolExecutor

    T, n, L, B = case["T"], case["n"], len(case["n"]), case["B"]
    jobs = []
    for t in range(T):
        w = [m[t * n[k]:(t + 1) * n[k]] for k, m in enumerate(want)]
        if any(x.any() for x in w):
            cuts = [B * j // splits for j in range(splits + 1)]
            jobs += [(t, cuts[j], cuts[j + 1], w) for j in range(splits) if cuts[j + 1] > cuts[j]]

    def one(job):
        t, b0, b1, w = job
        return t, orc.backward_n(_part_case_n(case, t, b0, b1), want=w)[0]

    out = [np.zeros(G.shape) for G in case["cores"]]
    with ThreadPoolExecutor(8) as ex:
        for t, g in ex.map(one, jobs):
            for k in range(L):
                out[k][t] += g[k][0]
    return out


def _sampled_slices_n(case, tables, seed):
    T, n, B = case["T"], case["n"], case["B"]
    bag = np.repeat(np.arange(T * B), np.diff(case["offsets"]))
    tab = bag // B
    dig = np.stack(np.unravel_index(case["idx"], n), 1)
    rng = np.random.default_rng(seed)
    want = [np.zeros(T * nk, np.uint8) for nk in n]
    for t in tables:
        sel = tab == t
        for k in range(len(n)):
            want[k][t * n[k] + np.bincount(dig[sel, k], minlength=n[k]).argmax()] = 1
    for k in range(len(n)):
        want[k][tables[0] * n[k] + int(rng.integers(0, n[k]))] = 1
    return want


@pytest.mark.parametrize("n,d,R", [((3, 4, 5, 6), (2, 1, 2, 2), 5), ((2, 3, 2, 4, 5), (1, 2, 2, 1, 3), 4)])
def test_gradients_n_deterministic(lib, n, d, R):
    # every gradient of a generic view is a fixed-order sum (segment sums in the view's
    # backward, chunk and child partials in the split): two runs give the same bits
    case = ttgen.tiny_n(7650 + len(n), 2, n, d, R, 40, max_len=6, zipf=1.1)
    _say(f"[cores determinism] L={len(n)} n={n} d={d} R={R}")
    runs = []
    for _ in range(2):
        emb = _make(lib, case)
        cores, idx, off = _dev(case)
        dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
        emb.forward_n(cores, idx, off, num_bags=case["B"])
        grads = emb.backward_n(cores, idx, off, dV, num_bags=case["B"])
        torch.cuda.synchronize()
        runs.append([g.cpu().numpy() for g in grads])
    for k, (a, b) in enumerate(zip(*runs)):
        assert np.array_equal(a, b), k


def test_autograd_module_n(lib, orc):
    case = ttgen.tiny_n(7600, 2, (5, 4, 20, 30), (2, 2, 4, 8), 32, 60, max_len=12, zipf=1.1)
    _say("[cores autograd] L=4 n=(5,4,20,30) d=(2,2,4,8) R=32")
    M = int(case["idx"].size)
    mod = lib.TTEmbeddingBag(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=M,
                             max_bags=case["B"])
    with torch.no_grad():
        for G, src in zip(mod.cores, case["cores"]):
            G.copy_(torch.from_numpy(src))
    _, idx, off = _dev(case)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    out = mod(idx, off)
    (out * dV).sum().backward()
    torch.cuda.synchronize()
    D = int(np.prod(case["d"]))
    grads = [G.grad.cpu().numpy() for G in mod.cores]
    _check(orc, case, out.detach().cpu().numpy().reshape(-1, D), grads, "autograd L=4")
    # the training step (backward_n + sgd_n) leaves G - lr dG
    lr = 0.01
    before = [G.detach().clone() for G in mod.cores]
    mod.step_fused(idx, off, dV, lr)
    torch.cuda.synchronize()
    dref, _ = orc.backward_n(case)
    dmag, _ = orc.backward_n(_abs_n(case))
    for k, G in enumerate(mod.cores):
        got = (before[k] - G.detach()).cpu().numpy() / lr
        # the difference of two nearby floats adds |G| * 2^-24 / lr of rounding
        slack = np.abs(before[k].cpu().numpy()) * 2.0 ** -23 / lr
        assert_close(f"step dG{k + 1}", got, dref[k], dmag[k] + slack / TOL)


def _random_shape(rng):
    L = int(rng.integers(2, 8))
    while True:
        n = tuple(int(x) for x in rng.integers(1, 6, size=L))
        d = tuple(int(x) for x in rng.integers(1, 4, size=L))
        if np.prod(n) >= 2 and np.prod(d) <= 64:
            break
    R = int(rng.choice([1, 2, 3, 5, 8, 16]))
    T = int(rng.integers(1, 4))
    B = int(rng.integers(1, 40))
    return T, n, d, R, B


@pytest.mark.parametrize("seed", range(12))
def test_random_shapes_n(lib, orc, seed):
    # seeded random L, factors (including 1), ranks and bag mixes; every third case
    # regroups in the backward instead of reusing the forward's grouping
    rng = np.random.default_rng([7700, seed])
    T, n, d, R, B = _random_shape(rng)
    case = ttgen.tiny_n(7700 + seed, T, n, d, R, B, max_len=int(rng.integers(0, 9)),
                        zipf=1.2 if seed % 2 else None)
    _say(f"[cores random {seed}] L={len(n)} T={T} n={n} d={d} R={R} B={B} M={case['idx'].size}")
    emb = _make(lib, case)
    cores, idx, off = _dev(case)
    out = emb.forward_n(cores, idx, off, num_bags=B)
    dV = torch.from_numpy(np.ascontiguousarray(case["dV"])).cuda()
    grads = emb.backward_n(cores, idx, off, dV, num_bags=B, reuse_grouping=seed % 3 != 0)
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    D = int(np.prod(d))
    _check(orc, case, out.cpu().numpy().reshape(-1, D), [g.cpu().numpy() for g in grads], f"random {seed}")
