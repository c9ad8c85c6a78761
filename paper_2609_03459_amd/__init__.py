"""MI355X-native Tensor-Train embedding gather (FlowTT, ICCAD'26).

`TTEmbedding` drives the C-ABI library libttemb.so (include/tt_emb.h) on
torch-allocated device memory and torch's current HIP stream.  Torch provides
memory and streams only; every step of the gather runs in the library's HIP
kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _native as N

__all__ = ["TTEmbedding", "N"]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


class TTEmbedding:
    """One handle plus its device workspace for tables of one TT shape.

    Cores: G1 [T][n1][d1][R], G2 [T][n2][R][d2][R], G3 [T][n3][R][d3] (float32).
    Indices int64 [M] (tables concatenated), offsets int64 [T*B+1] or None.
    """

    def __init__(self, num_tables, num_rows, row_factors, dim_factors, rank, max_indices, max_bags,
                 device="cuda", reuse="prefix"):
        d = N.tt_emb_desc()
        d.num_tables = int(num_tables)
        d.num_rows = int(num_rows)
        for k in range(3):
            d.row_factors[k] = int(row_factors[k])
            d.dim_factors[k] = int(dim_factors[k])
        d.rank = int(rank)
        d.max_indices = int(max_indices)
        d.max_bags = int(max_bags)
        self.desc = d
        self.T, self.N, self.R = int(num_tables), int(num_rows), int(rank)
        self.n = tuple(int(x) for x in row_factors)
        self.d = tuple(int(x) for x in dim_factors)
        self.D = self.d[0] * self.d[1] * self.d[2]
        self.handle = N.tt_emb_create(d)
        # reuse level (Section 4.5 ablation): "prefix" (default), "unique" or "none"
        N.tt_emb_set_reuse(self.handle, N.REUSE[reuse])
        self.reuse = reuse
        self.ws_bytes = N.tt_emb_workspace_size(self.handle)
        # 256-byte aligned workspace carved from one torch allocation
        raw = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        shift = (-raw.data_ptr()) % 256
        self._raw = raw
        self.workspace = raw[shift:shift + self.ws_bytes]
        self.device = device

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            N.tt_emb_destroy(h)
            self.handle = None

    # shapes
    def core_shapes(self):
        T, (n1, n2, n3), (d1, d2, d3), R = self.T, self.n, self.d, self.R
        return (T, n1, d1, R), (T, n2, R, d2, R), (T, n3, R, d3)

    def _nb(self, idx, offsets, num_bags):
        if num_bags is not None:
            return int(num_bags)
        if offsets is None:
            return idx.numel() // self.T
        return (offsets.numel() - 1) // self.T

    def group(self, idx, offsets=None, num_bags=None):
        nb = self._nb(idx, offsets, num_bags)
        N.tt_emb_group(self.handle, _ptr(idx), idx.numel(), _ptr(offsets), nb, _ptr(self.workspace), self.ws_bytes,
                       _stream())

    def forward(self, G1, G2, G3, idx, offsets=None, num_bags=None, out=None, reuse_grouping=False):
        nb = self._nb(idx, offsets, num_bags)
        if out is None:
            out = torch.empty((self.T, nb, self.D), dtype=torch.float32, device=G1.device)
        N.tt_emb_forward(self.handle, _ptr(G1), _ptr(G2), _ptr(G3), _ptr(idx), idx.numel(), _ptr(offsets), nb,
                         _ptr(out), reuse_grouping, _ptr(self.workspace), self.ws_bytes, _stream())
        return out

    def backward(self, G1, G2, G3, idx, offsets, grad_out, num_bags=None, grads=None, reuse_grouping=True):
        nb = self._nb(idx, offsets, num_bags)
        if grads is None:
            grads = tuple(torch.empty(s, dtype=torch.float32, device=G1.device) for s in self.core_shapes())
        dG1, dG2, dG3 = grads
        N.tt_emb_backward(self.handle, _ptr(G1), _ptr(G2), _ptr(G3), _ptr(idx), idx.numel(), _ptr(offsets), nb,
                          _ptr(grad_out), _ptr(dG1), _ptr(dG2), _ptr(dG3), reuse_grouping, _ptr(self.workspace),
                          self.ws_bytes, _stream())
        return grads

    def sgd(self, G1, G2, G3, dG1, dG2, dG3, lr):
        N.tt_emb_sgd(self.handle, _ptr(G1), _ptr(G2), _ptr(G3), _ptr(dG1), _ptr(dG2), _ptr(dG3), lr, _stream())

    def check_errors(self) -> int:
        return N.tt_emb_check_errors(self.handle, _ptr(self.workspace), _stream())

    def counts(self):
        """U, P, nvalid and slice count of the last grouping (synchronises)."""
        counts = np.zeros(4, np.int64)
        N.check("tt_emb_debug_grouping",
                N.lib.tt_emb_debug_grouping(self.handle, _ptr(self.workspace), None, None, None, None, None, None,
                                            None, counts.ctypes.data, _stream()))
        return dict(U=int(counts[0]), P=int(counts[1]), nvalid=int(counts[2]), nslices=int(counts[3]))

    def debug_grouping(self, num_indices):
        """Grouping arrays of the last grouped call, on the host (synchronises)."""
        import ctypes as C

        counts = np.zeros(4, np.int64)
        N.check("tt_emb_debug_grouping",
                N.lib.tt_emb_debug_grouping(self.handle, _ptr(self.workspace), None, None, None, None, None, None,
                                            None, counts.ctypes.data, _stream()))
        U, P, nv, ns = (int(x) for x in counts)
        m1 = max(num_indices, 1)
        uk = np.zeros(max(U, 1), np.int64)
        dg = np.zeros((max(U, 1), 3), np.int32)
        inv = np.zeros(m1, np.int32)
        os_ = np.zeros(U + 1, np.int32)
        op = np.zeros(max(nv, 1), np.int32)
        ps = np.zeros(P + 1, np.int32)
        pk = np.zeros(max(P, 1), np.int64)
        N.check("tt_emb_debug_grouping",
                N.lib.tt_emb_debug_grouping(self.handle, _ptr(self.workspace), uk.ctypes.data, dg.ctypes.data,
                                            inv.ctypes.data, os_.ctypes.data, op.ctypes.data, ps.ctypes.data,
                                            pk.ctypes.data, counts.ctypes.data, _stream()))
        del C
        return dict(uniq_keys=uk[:U], digits=dg[:U], inv=inv[:num_indices], occ_start=os_, occ_pos=op[:nv],
                    pg_start=ps, pg_keys=pk[:P], U=U, P=P, nvalid=nv, nslices=ns)
