"""Seeded synthetic workloads for the TT-embedding gather.

This module only draws random inputs: TT cores, row indices, bag offsets and
upstream gradients.  It holds none of the gather's arithmetic (no digit
decomposition, no contraction, no pooling), so both the oracle side and the
GPU side can take their inputs from here without sharing any of the method.

Layouts produced (float32, row-major, tables contiguous):
    G1 [T][n1][d1][R]      first core,  rank profile (1, R)
    G2 [T][n2][R][d2][R]   middle core, rank profile (R, R)
    G3 [T][n3][R][d3]      last core,   rank profile (R, 1)
    idx     int64 [M]      row ids of all tables concatenated (table-major)
    offsets int64 [T*B+1]  CSR bag boundaries over idx, or None (one row per bag)
    dV      float32 [T][B][D] upstream gradient of the pooled output

The workloads stand in for the paper's benchmark (Meta's synthetic DLRM
embedding-bag traces, evaluation section), which is not available here.  The
recipes follow the paper's operating regime: three cores, equal inner ranks,
batch 32,768, long-tailed (Zipf) row popularity.

Samplers, each a published method:
  * uniform / normal / Poisson / permutation: numpy's PCG64 Generator
    (permutation is a Fisher-Yates shuffle);
  * bounded Zipf P(k) ~ k^-a on {1..n}: rejection-inversion of Hormann and
    Derflinger, "Rejection-inversion to generate variates from monotone
    discrete distributions" (ACM TOMACS 6(3), 1996).
"""
from __future__ import annotations

import math

import numpy as np

BASE_SEED = 20261202

# purpose codes for independent random streams
_S_CORES, _S_IDX, _S_LEN, _S_PERM, _S_HOT, _S_DV = 1, 2, 3, 4, 5, 6


def _rng(seed: int, cfg: int, table: int, purpose: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(cfg), int(table), int(purpose)])


# ----------------------------------------------------------------------------
# bounded Zipf by rejection-inversion
# ----------------------------------------------------------------------------
def _H(x, s):
    """Antiderivative of x^-s with H(1) = 0."""
    lx = np.log(x)
    t = (1.0 - s) * lx
    # (exp(t) - 1) / t, evaluated stably near t = 0
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(np.abs(t) > 1e-8, np.expm1(t) / np.where(t == 0, 1.0, t), 1.0 + 0.5 * t)
    return r * lx


def _Hinv(y, s):
    t = y * (1.0 - s)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(np.abs(t) > 1e-8, np.log1p(t) / np.where(t == 0, 1.0, t), 1.0 - 0.5 * t)
    return np.exp(r * y)


def zipf_bounded(rng: np.random.Generator, alpha: float, n: int, size: int) -> np.ndarray:
    """Draw `size` ranks k in [1, n] with P(k) proportional to k^-alpha."""
    s = float(alpha)
    h = lambda x: np.exp(-s * np.log(x))  # noqa: E731
    hx1 = float(_H(np.float64(1.5), s)) - 1.0
    hn = float(_H(np.float64(n + 0.5), s))
    squeeze = 2.0 - float(_Hinv(_H(np.float64(2.5), s) - h(np.float64(2.0)), s))
    out = np.empty(size, dtype=np.int64)
    todo = np.arange(size)
    while todo.size:
        u = hn + rng.random(todo.size) * (hx1 - hn)
        x = _Hinv(u, s)
        k = np.clip(np.floor(x + 0.5), 1, n)
        ok = (k - x <= squeeze) | (u >= _H(k + 0.5, s) - h(k))
        out[todo[ok]] = k[ok].astype(np.int64)
        todo = todo[~ok]
    return out


# ----------------------------------------------------------------------------
# workload recipes
# ----------------------------------------------------------------------------
CONFIGS = {
    1: dict(workload="tt-gather-1e6rows-d16-r8-uniform4096", T=1, n=(100, 100, 100), d=(2, 2, 4), R=8,
            sigma=0.1, B=4096, bags="single", dist=("uniform",), train=False),
    2: dict(workload="tt-gather-1e7rows-d64-r16-zipf1.05-b32768", T=1, n=(200, 200, 250), d=(4, 4, 4), R=16,
            sigma=0.05, B=32768, bags="single", dist=("zipf", 1.05), train=False),
    3: dict(workload="tt-embbag-8x1e7rows-d128-r32-zipf1.1-pois20-b32768", T=8, n=(200, 200, 250), d=(4, 4, 8),
            R=32, sigma=0.05, B=32768, bags="poisson", bag_mean=20.0, bag_min=1, bag_max=64,
            dist=("zipf", 1.1), train=False),
    4: dict(workload="tt-embbag-1e8rows-d128-r64-zipf1.2-hotprefix-b32768x32", T=1, n=(400, 500, 500),
            d=(4, 4, 8), R=64, sigma=0.05, B=32768, bags="fixed", bag_len=32,
            dist=("hotprefix", 1.2, 2000, 0.5), train=False),
    5: dict(workload="tt-embbag-train-8x1e7rows-d128-r32-zipf1.1-pois20-b32768-sgd", T=8, n=(200, 200, 250),
            d=(4, 4, 8), R=32, sigma=0.05, B=32768, bags="poisson", bag_mean=20.0, bag_min=1, bag_max=64,
            dist=("zipf", 1.1), train=True, lr=0.01),
    # the paper's operating point (D = 32, R = 32, three cores; its factorisation of D is not
    # stated: (4, 4, 2) here) on the 8-table index recipe above
    6: dict(workload="tt-embbag-train-8x1e7rows-d32-r32-zipf1.1-pois20-b32768-sgd", T=8, n=(200, 200, 250),
            d=(4, 4, 2), R=32, sigma=0.05, B=32768, bags="poisson", bag_mean=20.0, bag_min=1, bag_max=64,
            dist=("zipf", 1.1), train=True, lr=0.01),
}


def draw_cores(rng: np.random.Generator, T, n, d, R, sigma):
    n1, n2, n3 = n
    d1, d2, d3 = d
    G1 = (rng.standard_normal((T, n1, d1, R)) * sigma).astype(np.float32)
    G2 = (rng.standard_normal((T, n2, R, d2, R)) * sigma).astype(np.float32)
    G3 = (rng.standard_normal((T, n3, R, d3)) * sigma).astype(np.float32)
    return G1, G2, G3


def make(cfg: int, seed: int = BASE_SEED, bags: int | None = None, with_grad: bool | None = None) -> dict:
    """Build workload `cfg` (1..6).  `bags` overrides the per-table bag count
    (parity tests run the same recipe at a smaller batch)."""
    c = dict(CONFIGS[cfg])
    T, n, d, R = c["T"], c["n"], c["d"], c["R"]
    N = int(n[0]) * int(n[1]) * int(n[2])
    B = int(bags) if bags is not None else int(c["B"])
    G1, G2, G3 = draw_cores(_rng(seed, cfg, 0, _S_CORES), T, n, d, R, c["sigma"])

    lens = []
    for t in range(T):
        if c["bags"] == "single":
            lens.append(np.ones(B, dtype=np.int64))
        elif c["bags"] == "fixed":
            lens.append(np.full(B, c["bag_len"], dtype=np.int64))
        else:
            lr = _rng(seed, cfg, t, _S_LEN)
            lens.append(np.clip(lr.poisson(c["bag_mean"], B), c["bag_min"], c["bag_max"]).astype(np.int64))

    idx_parts = []
    hot_share = []
    for t in range(T):
        m = int(lens[t].sum())
        ri = _rng(seed, cfg, t, _S_IDX)
        kind = c["dist"][0]
        if kind == "uniform":
            g = ri.integers(0, N, size=m, dtype=np.int64)
        elif kind == "zipf":
            perm = _rng(seed, cfg, t, _S_PERM).permutation(N)
            g = perm[zipf_bounded(ri, c["dist"][1], N, m) - 1]
        elif kind == "hotprefix":
            alpha, nhot, p_hot = c["dist"][1], c["dist"][2], c["dist"][3]
            block = int(n[2])                      # rows sharing one (first, second) factor pair
            nblocks = N // block
            hot_blocks = _rng(seed, cfg, t, _S_HOT).permutation(nblocks)[:nhot]
            is_hot = ri.random(m) < p_hot
            g = np.empty(m, dtype=np.int64)
            nh = int(is_hot.sum())
            hb = hot_blocks[zipf_bounded(ri, alpha, nhot, nh) - 1]
            g[is_hot] = hb * block + ri.integers(0, block, size=nh, dtype=np.int64)
            perm = _rng(seed, cfg, t, _S_PERM).permutation(N)
            g[~is_hot] = perm[zipf_bounded(ri, alpha, N, m - nh) - 1]
            hot_share.append(nh / max(m, 1))
        else:
            raise ValueError(kind)
        idx_parts.append(g.astype(np.int64))
    idx = np.concatenate(idx_parts) if idx_parts else np.zeros(0, np.int64)

    if c["bags"] == "single":
        offsets = None
    else:
        all_lens = np.concatenate(lens)
        offsets = np.zeros(T * B + 1, dtype=np.int64)
        np.cumsum(all_lens, out=offsets[1:])

    out = dict(cfg=cfg, workload=c["workload"], T=T, N=N, n=tuple(n), d=tuple(d), R=R, B=B,
               G1=G1, G2=G2, G3=G3, idx=idx, offsets=offsets, seed=seed)
    if hot_share:
        out["hot_share"] = float(np.mean(hot_share))
    train = c["train"] if with_grad is None else with_grad
    if train:
        D = d[0] * d[1] * d[2]
        out["dV"] = _rng(seed, cfg, 0, _S_DV).standard_normal((T, B, D)).astype(np.float32)
        out["lr"] = float(c.get("lr", 0.01))
    return out


def tiny(seed: int, T: int, n, d, R: int, B: int, max_len: int = 4, N: int | None = None,
         empty_bags: bool = True, sigma: float = 0.5, single: bool = False, grad: bool = True,
         zipf: float | None = None) -> dict:
    """A small random case with arbitrary factors (tests and edge cases)."""
    rng = np.random.default_rng([int(seed), 777])
    n = tuple(int(x) for x in n)
    d = tuple(int(x) for x in d)
    full = n[0] * n[1] * n[2]
    N = full if N is None else int(N)
    G1, G2, G3 = draw_cores(rng, T, n, d, R, sigma)
    if single:
        lens = np.ones(T * B, dtype=np.int64)
    else:
        lens = rng.integers(0 if empty_bags else 1, max_len + 1, size=T * B).astype(np.int64)
    m = int(lens.sum())
    if zipf is not None and N > 1:
        idx = (zipf_bounded(rng, zipf, N, m) - 1).astype(np.int64)
    else:
        idx = rng.integers(0, N, size=m, dtype=np.int64)
    offsets = None
    if not single:
        offsets = np.zeros(T * B + 1, dtype=np.int64)
        np.cumsum(lens, out=offsets[1:])
    D = d[0] * d[1] * d[2]
    out = dict(cfg=0, workload="tiny", T=T, N=N, n=n, d=d, R=R, B=B, G1=G1, G2=G2, G3=G3, idx=idx,
               offsets=offsets, seed=seed)
    if grad:
        out["dV"] = rng.standard_normal((T, B, D)).astype(np.float32)
        out["lr"] = 0.01
    return out


def bag_lengths(offsets: np.ndarray | None, T: int, B: int) -> np.ndarray:
    if offsets is None:
        return np.ones(T * B, dtype=np.int64)
    return np.diff(offsets)


def sample_bags(seed: int, T: int, B: int, count: int) -> np.ndarray:
    """Seeded sample of global bag ids (t*B + b) for spot checks at full size."""
    rng = np.random.default_rng([int(seed), 4242])
    count = min(count, T * B)
    return np.sort(rng.choice(T * B, size=count, replace=False)).astype(np.int64)


def math_check_zipf_mass(alpha: float, n: int) -> float:
    """Probability of rank 1 under bounded Zipf (used to sanity-check the sampler)."""
    ks = np.arange(1, n + 1, dtype=np.float64)
    return float(1.0 / np.sum(ks ** -alpha))


__all__ = ["BASE_SEED", "CONFIGS", "make", "tiny", "zipf_bounded", "draw_cores", "bag_lengths",
           "sample_bags", "math_check_zipf_mass"]
_ = math


def core_shapes_n(T: int, n, d, R: int):
    """Shapes of the L cores of a TT table: core k is [T][n_k][r_k][d_k][r_{k+1}]
    with r_0 = r_L = 1 (the unit ranks dropped from the shape) and the others R."""
    L = len(n)
    shapes = []
    for k in range(L):
        s = [T, int(n[k])]
        if k > 0:
            s.append(R)
        s.append(int(d[k]))
        if k < L - 1:
            s.append(R)
        shapes.append(tuple(s))
    return shapes


def tiny_n(seed: int, T: int, n, d, R: int, B: int, max_len: int = 4, sigma: float = 0.5,
           zipf: float | None = None, grad: bool = True) -> dict:
    """A small random case with L = len(n) cores (random data only)."""
    rng = np.random.default_rng([int(seed), 778])
    n = tuple(int(x) for x in n)
    d = tuple(int(x) for x in d)
    N = int(np.prod(n))
    cores = [(rng.standard_normal(s) * sigma).astype(np.float32) for s in core_shapes_n(T, n, d, R)]
    lens = rng.integers(0, max_len + 1, size=T * B).astype(np.int64)
    m = int(lens.sum())
    if zipf is not None and N > 1:
        idx = (zipf_bounded(rng, zipf, N, m) - 1).astype(np.int64)
    else:
        idx = rng.integers(0, N, size=m, dtype=np.int64)
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    out = dict(workload="tiny_n", T=T, N=N, L=len(n), n=n, d=d, R=R, B=B, cores=cores, idx=idx, offsets=offsets,
               seed=seed)
    if grad:
        out["dV"] = rng.standard_normal((T, B, int(np.prod(d)))).astype(np.float32)
        out["lr"] = 0.01
    return out
