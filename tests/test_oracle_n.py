"""Pins of the L-core oracle (CPU): the L = 3 oracle, an exact closed form, a
reduction of L = 4 to L = 3, an independent float64 torch computation with
autograd, and the Euler identity of a function linear in each core."""
import numpy as np
import pytest
import torch

import oracle
import ttgen


def _as3(case_n):
    """The same L = 3 case in the three-core oracle's format."""
    G1, G2, G3 = case_n["cores"]
    return dict(T=case_n["T"], N=case_n["N"], n=case_n["n"], d=case_n["d"], R=case_n["R"], B=case_n["B"], G1=G1,
                G2=G2, G3=G3, idx=case_n["idx"], offsets=case_n["offsets"], dV=case_n["dV"])


def test_three_cores_match_the_three_core_oracle():
    c = ttgen.tiny_n(11, 2, (3, 4, 5), (2, 3, 2), 4, 9, max_len=5)
    V, _ = oracle.forward_n(c)
    V3, _ = oracle.forward(_as3(c))
    np.testing.assert_allclose(V, V3, rtol=1e-12, atol=1e-12)
    dG, _ = oracle.backward_n(c)
    ref = oracle.backward(_as3(c))[:3]
    for k in range(3):
        np.testing.assert_allclose(dG[k], ref[k], rtol=1e-12, atol=1e-12)


def _additive(T, n, d, R):
    """Rank-2 additive TT (zero-padded to rank R): E[g][j] = g*D + j exactly."""
    L = len(n)
    D = int(np.prod(d))
    cores = [np.zeros(s, np.float32) for s in ttgen.core_shapes_n(T, n, d, R)]
    for k in range(L):
        pn = int(np.prod(n[k + 1:])) if k + 1 < L else 1
        pd = int(np.prod(d[k + 1:])) if k + 1 < L else 1
        for i in range(n[k]):
            for j in range(d[k]):
                val = i * pn * D + j * pd
                if k == 0:
                    cores[k][:, i, j, 0] = val
                    cores[k][:, i, j, 1] = 1
                elif k == L - 1:
                    cores[k][:, i, 0, j] = 1
                    cores[k][:, i, 1, j] = val
                else:
                    cores[k][:, i, 0, j, 0] = 1
                    cores[k][:, i, 1, j, 0] = val
                    cores[k][:, i, 1, j, 1] = 1
    return cores


@pytest.mark.parametrize("n,d", [((5, 7), (3, 2)), ((3, 4, 2, 3), (2, 1, 3, 2)), ((2, 3, 2, 2, 3), (1, 2, 2, 1, 3))])
def test_additive_rank2_closed_form(n, d):
    # pins the digit order of Eq. 2, the output digit order and the chain of
    # contractions at once, for L = 2, 4, 5
    T, R = 1, 3
    N = int(np.prod(n))
    D = int(np.prod(d))
    idx = np.arange(N, dtype=np.int64)
    case = dict(T=T, N=N, L=len(n), n=n, d=d, R=R, B=N, cores=_additive(T, n, d, R), idx=idx, offsets=None)
    V, inv = oracle.forward_n(case)
    assert inv == 0
    expect = np.arange(N)[:, None] * D + np.arange(D)[None, :]
    assert np.array_equal(V, expect.astype(np.float64))


def test_identity_core_reduces_four_cores_to_three():
    # a middle core with one row, one output digit and the identity as its slice
    # leaves the function of the other three cores unchanged
    c3 = ttgen.tiny_n(21, 2, (3, 4, 5), (2, 3, 2), 4, 8, max_len=4)
    G1, G2, G3 = c3["cores"]
    Ident = np.broadcast_to(np.eye(4, dtype=np.float32)[None, None, :, None, :], (2, 1, 4, 1, 4)).copy()
    c4 = dict(c3, L=4, n=(3, 4, 1, 5), d=(2, 3, 1, 2), cores=[G1, G2, Ident, G3])
    V4, _ = oracle.forward_n(c4)
    V3, _ = oracle.forward_n(c3)
    np.testing.assert_allclose(V4, V3, rtol=1e-12, atol=1e-12)
    dG4, _ = oracle.backward_n(c4)
    dG3, _ = oracle.backward_n(c3)
    for a, b in ((0, 0), (1, 1), (3, 2)):
        np.testing.assert_allclose(dG4[a], dG3[b], rtol=1e-12, atol=1e-12)


def _torch_table(cores, n, d):
    """Every row of every table from float64 torch ops: the core slices of each digit
    combination multiplied as a chain (independent of the oracle's C code)."""
    L = len(n)
    T = cores[0].shape[0]
    rows = []
    for t in range(T):
        for g in range(int(np.prod(n))):
            dig = []
            r = g
            for k in reversed(range(L)):
                dig.append(r % n[k])
                r //= n[k]
            dig = dig[::-1]
            X = cores[0][t, dig[0]]  # d0 x R
            for k in range(1, L):
                S = cores[k][t, dig[k]]
                S = S.reshape(S.shape[0], -1)  # r_k x (d_k r_{k+1})
                X = (X.reshape(-1, S.shape[0]) @ S)
            rows.append(X.reshape(-1))
    return torch.stack(rows).reshape(T, int(np.prod(n)), -1)


@pytest.mark.parametrize("n,d,R", [((4, 3), (2, 3), 3), ((2, 3, 2, 3), (2, 2, 1, 3), 3), ((2, 2, 2, 2, 2), (1, 2, 1, 2, 2), 2)])
def test_brute_force_and_autograd(n, d, R):
    c = ttgen.tiny_n(31, 2, n, d, R, 6, max_len=5)
    cores = [torch.tensor(G, dtype=torch.float64, requires_grad=True) for G in c["cores"]]
    W = _torch_table(cores, n, d)
    T, B = c["T"], c["B"]
    off = c["offsets"]
    V = []
    for gb in range(T * B):
        t = gb // B
        lo, hi = off[gb], off[gb + 1]
        rows = [W[t, int(g)] for g in c["idx"][lo:hi]]
        V.append(torch.stack(rows).sum(0) if rows else torch.zeros(W.shape[-1], dtype=torch.float64))
    V = torch.stack(V)
    Vo, _ = oracle.forward_n(c)
    np.testing.assert_allclose(Vo, V.detach().numpy(), rtol=1e-12, atol=1e-12)
    (V * torch.tensor(c["dV"].reshape(T * B, -1), dtype=torch.float64)).sum().backward()
    dG, _ = oracle.backward_n(c)
    for k in range(len(n)):
        np.testing.assert_allclose(dG[k], cores[k].grad.numpy(), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("n,d", [((6, 5), (2, 4)), ((3, 4, 3, 2), (2, 2, 2, 2)), ((2, 3, 2, 2, 3), (2, 1, 2, 2, 1))])
def test_euler_identity(n, d):
    # V is linear in each core, so <dG_k, G_k> = <dV, V> for every k
    c = ttgen.tiny_n(41, 2, n, d, 3, 10, max_len=6)
    V, _ = oracle.forward_n(c)
    dG, _ = oracle.backward_n(c)
    lhs = float(np.sum(c["dV"].reshape(V.shape).astype(np.float64) * V))
    for k in range(len(n)):
        rhs = float(np.sum(dG[k] * c["cores"][k].astype(np.float64)))
        assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))
