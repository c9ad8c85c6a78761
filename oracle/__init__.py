"""Python access to the plain CPU oracle (oracle/tt_oracle.c).

TEST INFRASTRUCTURE ONLY: the correctness reference for the GPU library.
Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  It imports nothing from the GPU library and the GPU library
imports nothing from it; the two share only the seeded input generators
(package `ttgen`), which hold none of the operator's arithmetic.

Each function cites the passage of the paper (FlowTT, ICCAD'26) it follows;
see the header of tt_oracle.c for layouts and conventions.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tt_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile tt_oracle.c with gcc into oracle/liboracle.so (IEEE double, no contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _ShapeN(C.Structure):
    _fields_ = [("T", C.c_int), ("N", C.c_int64), ("L", C.c_int), ("n", C.c_int32 * 8), ("d", C.c_int32 * 8),
                ("R", C.c_int), ("B", C.c_int64)]


class _Shape(C.Structure):
    _fields_ = [("T", C.c_int), ("N", C.c_int64), ("n", C.c_int32 * 3), ("d", C.c_int32 * 3), ("R", C.c_int),
                ("B", C.c_int64)]


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("TT_ORACLE_LIB")  # another build of tt_oracle.c (the sanitizer test's)
        if not path:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            path = _LIB
        lib = C.CDLL(path)
        P = C.c_void_p
        lib.orc_digits.argtypes = [P, C.c_int64, P, P]
        lib.orc_digits.restype = None
        lib.orc_row.argtypes = [C.POINTER(_Shape), P, P, P, C.c_int64, C.c_int64, P]
        lib.orc_row.restype = None
        lib.orc_forward.argtypes = [C.POINTER(_Shape), P, P, P, P, C.c_int64, P, P, C.c_int64, P]
        lib.orc_forward.restype = C.c_int64
        lib.orc_backward.argtypes = [C.POINTER(_Shape), P, P, P, P, C.c_int64, P, P, P, P, P, P, P, P]
        lib.orc_backward.restype = C.c_int64
        lib.orc_forward_n.argtypes = [C.POINTER(_ShapeN), P, P, C.c_int64, P, P]
        lib.orc_forward_n.restype = C.c_int64
        lib.orc_backward_n.argtypes = [C.POINTER(_ShapeN), P, P, C.c_int64, P, P, P, P]
        lib.orc_backward_n.restype = C.c_int64
        lib.orc_sgd.argtypes = [P, P, C.c_int64, C.c_double, P]
        lib.orc_sgd.restype = None
        lib.orc_grouping.argtypes = [C.POINTER(_Shape), P, C.c_int64, P, P, P, P, P, P, P, P, P, P]
        lib.orc_grouping.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _shape(case) -> _Shape:
    s = _Shape()
    s.T = int(case["T"])
    s.N = int(case["N"])
    for k in range(3):
        s.n[k] = int(case["n"][k])
        s.d[k] = int(case["d"][k])
    s.R = int(case["R"])
    s.B = int(case["B"])
    return s


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int64)


def digits(g, n) -> np.ndarray:
    """Eq. 2 (Section 3.3): mixed-radix digits (i1, i2, i3) of each row id."""
    g = _i64(np.atleast_1d(g))
    nn = np.ascontiguousarray(n, dtype=np.int32)
    out = np.zeros((g.size, 3), dtype=np.int64)
    _load().orc_digits(_ptr(g), g.size, _ptr(nn), _ptr(out))
    return out


def row(case, t: int, g: int) -> np.ndarray:
    """One reconstructed embedding row E_g of table t (Section 3.2: C = A.B, E = C.D)."""
    D = int(np.prod(case["d"]))
    out = np.zeros(D, dtype=np.float64)
    s = _shape(case)
    _load().orc_row(C.byref(s), _ptr(_f32(case["G1"])), _ptr(_f32(case["G2"])), _ptr(_f32(case["G3"])), int(t),
                    int(g), _ptr(out))
    return out


def forward(case, bags=None):
    """Sum-pooled TT gather (Section 3.2): V[gb] = sum over the bag of E_idx.
    Returns (V, invalid_count); V is [T*B][D] or [len(bags)][D]."""
    D = int(np.prod(case["d"]))
    s = _shape(case)
    idx = _i64(case["idx"])
    off = _i64(case["offsets"])
    bl = _i64(bags)
    count = (int(case["T"]) * int(case["B"])) if bl is None else bl.size
    V = np.zeros((count, D), dtype=np.float64)
    inv = _load().orc_forward(C.byref(s), _ptr(_f32(case["G1"])), _ptr(_f32(case["G2"])), _ptr(_f32(case["G3"])),
                              _ptr(idx), idx.size, _ptr(off), _ptr(bl), 0 if bl is None else bl.size, _ptr(V))
    return V, int(inv)


def backward(case, dV=None, want=None):
    """Core gradients of L = sum <dV, V> (Section 3.2, Eq. 1 before regrouping).
    `want` = optional (mask1, mask2, mask3) of per-slice booleans [T*n_k]: only
    the wanted slices are then guaranteed exact.  Returns (dG1, dG2, dG3, invalid)."""
    T, n, d, R = int(case["T"]), case["n"], case["d"], int(case["R"])
    dV = _f32(case["dV"] if dV is None else dV)
    s = _shape(case)
    idx = _i64(case["idx"])
    off = _i64(case["offsets"])
    dG1 = np.zeros((T, n[0], d[0], R), dtype=np.float64)
    dG2 = np.zeros((T, n[1], R, d[1], R), dtype=np.float64)
    dG3 = np.zeros((T, n[2], R, d[2]), dtype=np.float64)
    masks = [None, None, None]
    if want is not None:
        masks = [None if w is None else np.ascontiguousarray(w, dtype=np.uint8) for w in want]
    inv = _load().orc_backward(C.byref(s), _ptr(_f32(case["G1"])), _ptr(_f32(case["G2"])), _ptr(_f32(case["G3"])),
                               _ptr(idx), idx.size, _ptr(off), _ptr(dV), _ptr(dG1), _ptr(dG2), _ptr(dG3),
                               _ptr(masks[0]), _ptr(masks[1]), _ptr(masks[2]))
    return dG1, dG2, dG3, int(inv)


def sgd(G, dG, lr: float) -> np.ndarray:
    """Plain SGD step G - lr*dG, in double."""
    G = _f32(G)
    dG = np.ascontiguousarray(dG, dtype=np.float64)
    out = np.zeros(G.shape, dtype=np.float64)
    _load().orc_sgd(_ptr(G), _ptr(dG), G.size, float(lr), _ptr(out))
    return out


def grouping(case) -> dict:
    """Prefix-based index grouping (Section 3.3, Fig. 4) as canonical arrays."""
    s = _shape(case)
    idx = _i64(case["idx"])
    off = _i64(case["offsets"])
    M = idx.size
    m1 = max(M, 1)
    uniq_t = np.zeros(m1, np.int64)
    uniq_g = np.zeros(m1, np.int64)
    inv = np.zeros(m1, np.int64)
    occ_start = np.zeros(m1 + 1, np.int64)
    occ_pos = np.zeros(m1, np.int64)
    pg_start = np.zeros(m1 + 1, np.int64)
    pg_t = np.zeros(m1, np.int64)
    pg_q = np.zeros(m1, np.int64)
    counts = np.zeros(3, np.int64)
    _load().orc_grouping(C.byref(s), _ptr(idx), M, _ptr(off), _ptr(uniq_t), _ptr(uniq_g), _ptr(inv),
                         _ptr(occ_start), _ptr(occ_pos), _ptr(pg_start), _ptr(pg_t), _ptr(pg_q), _ptr(counts))
    U, P, nv = (int(x) for x in counts)
    return dict(uniq_t=uniq_t[:U], uniq_g=uniq_g[:U], inv=inv[:M], occ_start=occ_start[:U + 1],
                occ_pos=occ_pos[:nv], pg_start=pg_start[:P + 1], pg_t=pg_t[:P], pg_q=pg_q[:P], U=U, P=P,
                nvalid=nv)


__all__ = ["build", "digits", "row", "forward", "backward", "sgd", "grouping"]


def _shape_n(case) -> _ShapeN:
    s = _ShapeN()
    s.T, s.N, s.L, s.R, s.B = int(case["T"]), int(case["N"]), int(case["L"]), int(case["R"]), int(case["B"])
    if not 2 <= s.L <= 8:
        raise ValueError("2 <= L <= 8 cores")
    for k in range(s.L):
        s.n[k] = int(case["n"][k])
        s.d[k] = int(case["d"][k])
    return s


def _ptr_array(arrays):
    a = (C.c_void_p * len(arrays))(*[x.ctypes.data for x in arrays])
    return a


def forward_n(case):
    """Sum-pooled gather with L = len(case["n"]) cores: each row is the chain of its
    L core slices (Eq. 2 digits, Section 3.2 contraction extended to L cores).
    Returns (V [T*B][D], invalid_count)."""
    s = _shape_n(case)
    cores = [_f32(G) for G in case["cores"]]
    idx = _i64(case["idx"])
    off = _i64(case["offsets"])
    V = np.zeros((int(case["T"]) * int(case["B"]), int(np.prod(case["d"]))), dtype=np.float64)
    inv = _load().orc_forward_n(C.byref(s), C.cast(_ptr_array(cores), C.c_void_p), _ptr(idx), idx.size, _ptr(off),
                                _ptr(V))
    return V, int(inv)


def backward_n(case, dV=None, want=None):
    """Core gradients with L cores of L = sum <dV, V>: the chain rule through the chain
    of slices, per occurrence (for L = 3 exactly Eq. 1).  `want` = optional list of L
    per-slice boolean masks [T*n_k] (or None entries): only the wanted slices are then
    guaranteed exact.  Returns ([dG_k], invalid)."""
    s = _shape_n(case)
    cores = [_f32(G) for G in case["cores"]]
    dV = _f32(case["dV"] if dV is None else dV)
    idx = _i64(case["idx"])
    off = _i64(case["offsets"])
    dG = [np.zeros(G.shape, dtype=np.float64) for G in cores]
    wp = None
    if want is not None:
        masks = [None if w is None else np.ascontiguousarray(w, dtype=np.uint8) for w in want]
        if len(masks) != s.L:
            raise ValueError("one mask (or None) per core")
        wp = (C.c_void_p * s.L)(*[None if m is None else m.ctypes.data for m in masks])
    inv = _load().orc_backward_n(C.byref(s), C.cast(_ptr_array(cores), C.c_void_p), _ptr(idx), idx.size, _ptr(off),
                                 _ptr(dV), C.cast(_ptr_array(dG), C.c_void_p),
                                 None if wp is None else C.cast(wp, C.c_void_p))
    return dG, int(inv)
