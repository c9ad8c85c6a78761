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

__all__ = ["TTEmbedding", "TTEmbeddingBag", "tt_embedding_bag", "tt_embedding_bag_n", "N"]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


class TTEmbedding:
    """One handle plus its device workspace for tables of one TT shape.

    Three cores: G1 [T][n1][d1][R], G2 [T][n2][R][d2][R], G3 [T][n3][R][d3] (float32),
    used by forward / backward / sgd / backward_sgd.  Any number L >= 2 of factors:
    core k is [T][n_k][r_k][d_k][r_{k+1}] with r_0 = r_L = 1 and the other ranks R,
    used by forward_n / backward_n / sgd_n (which also accept L = 3).
    Indices int64 [M] (tables concatenated), offsets int64 [T*B+1] or None.
    """

    def __init__(self, num_tables, num_rows, row_factors, dim_factors, rank, max_indices, max_bags,
                 device="cuda", reuse="prefix", sched="steal"):
        L = len(row_factors)
        if len(dim_factors) != L:
            raise ValueError("row_factors and dim_factors must have the same length")
        self.L = L
        if L == 3:
            d = N.tt_emb_desc()
        else:
            d = N.tt_emb_desc_n()
            d.num_cores = L
        d.num_tables = int(num_tables)
        d.num_rows = int(num_rows)
        for k in range(min(L, N.MAX_CORES)):
            d.row_factors[k] = int(row_factors[k])
            d.dim_factors[k] = int(dim_factors[k])
        d.rank = int(rank)
        d.max_indices = int(max_indices)
        d.max_bags = int(max_bags)
        self.desc = d
        self.T, self.N, self.R = int(num_tables), int(num_rows), int(rank)
        self.n = tuple(int(x) for x in row_factors)
        self.d = tuple(int(x) for x in dim_factors)
        self.D = int(np.prod(self.d))
        if L == 3:
            self.handle = N.tt_emb_create(d)
        elif L < 2 or L > N.MAX_CORES:
            raise ValueError(f"number of cores must be in [2, {N.MAX_CORES}]")
        else:
            self.handle = N.tt_emb_create_n(d)
        # reuse level (Section 4.5 ablation): "prefix" (default), "unique" or "none"
        N.tt_emb_set_reuse(self.handle, N.REUSE[reuse])
        self.reuse = reuse
        # work distribution (Section 4.4 ablation): "steal" (default), "static" or "steal_ckpt"
        self.set_schedule(sched)
        # a workspace that serves every call up to the maxima
        self.ws_bytes = N.tt_emb_workspace_size(self.handle, int(max_indices), int(max_bags))
        # 256-byte aligned workspace carved from one torch allocation
        raw = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        shift = (-raw.data_ptr()) % 256
        self._raw = raw
        self.workspace = raw[shift:shift + self.ws_bytes]
        self.device = device

    def set_schedule(self, sched):
        N.tt_emb_set_schedule(self.handle, N.SCHED[sched])
        self.sched = sched

    def __del__(self):
        # at interpreter exit the binding's module globals may already be gone
        h = getattr(self, "handle", None)
        self.handle = None
        if h and N is not None and getattr(N, "lib", None) is not None:
            try:
                N.tt_emb_destroy(h)
            except Exception:
                pass

    # shapes
    def core_shapes(self):
        T, R, L = self.T, self.R, self.L
        shapes = []
        for k in range(L):
            shape = [T, self.n[k]] + ([R] if k > 0 else []) + [self.d[k]] + ([R] if k < L - 1 else [])
            shapes.append(tuple(shape))
        return tuple(shapes)

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

    def backward_sgd(self, G1, G2, G3, idx, offsets, grad_out, lr, num_bags=None, reuse_grouping=True):
        """Backward pass with the SGD step fused in: G_k -= lr * dG_k in place, no gradient arrays."""
        nb = self._nb(idx, offsets, num_bags)
        N.tt_emb_backward_sgd(self.handle, _ptr(G1), _ptr(G2), _ptr(G3), _ptr(idx), idx.numel(), _ptr(offsets), nb,
                              _ptr(grad_out), lr, reuse_grouping, _ptr(self.workspace), self.ws_bytes, _stream())

    def forward_n(self, cores, idx, offsets=None, num_bags=None, out=None, reuse_grouping=False):
        nb = self._nb(idx, offsets, num_bags)
        if out is None:
            out = torch.empty((self.T, nb, self.D), dtype=torch.float32, device=cores[0].device)
        N.tt_emb_forward_n(self.handle, [_ptr(G) for G in cores], _ptr(idx), idx.numel(), _ptr(offsets), nb,
                           _ptr(out), reuse_grouping, _ptr(self.workspace), self.ws_bytes, _stream())
        return out

    def backward_n(self, cores, idx, offsets, grad_out, num_bags=None, grads=None, reuse_grouping=True):
        nb = self._nb(idx, offsets, num_bags)
        if grads is None:
            grads = tuple(torch.empty(sh, dtype=torch.float32, device=cores[0].device) for sh in self.core_shapes())
        N.tt_emb_backward_n(self.handle, [_ptr(G) for G in cores], _ptr(idx), idx.numel(), _ptr(offsets), nb,
                            _ptr(grad_out), [_ptr(g) for g in grads], reuse_grouping, _ptr(self.workspace),
                            self.ws_bytes, _stream())
        return grads

    def sgd_n(self, cores, grads, lr):
        N.tt_emb_sgd_n(self.handle, [_ptr(G) for G in cores], [_ptr(g) for g in grads], lr, _stream())

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


class _TTEmbeddingBagFn(torch.autograd.Function):
    """Autograd node of the pooled TT gather: forward groups the indices and runs the
    fused forward; backward reuses that grouping (regrouping if another call on the
    same handle replaced it) and returns the three dense core gradients."""

    @staticmethod
    def forward(ctx, G1, G2, G3, emb, idx, offsets, num_bags):
        out = emb.forward(G1, G2, G3, idx, offsets, num_bags=num_bags)
        ctx.emb, ctx.idx, ctx.offsets, ctx.num_bags = emb, idx, offsets, num_bags
        ctx.save_for_backward(G1, G2, G3)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        G1, G2, G3 = ctx.saved_tensors
        emb = ctx.emb
        g = grad_out.contiguous().to(torch.float32)
        try:
            grads = emb.backward(G1, G2, G3, ctx.idx, ctx.offsets, g, num_bags=ctx.num_bags, reuse_grouping=True)
        except N.TTEmbError as e:
            if e.code != N.TT_EMB_EINVAL:
                raise
            grads = emb.backward(G1, G2, G3, ctx.idx, ctx.offsets, g, num_bags=ctx.num_bags, reuse_grouping=False)
        return grads[0], grads[1], grads[2], None, None, None, None


def tt_embedding_bag(G1, G2, G3, emb, idx, offsets=None, num_bags=None):
    """Differentiable pooled lookup: out [T][B][D], gradients flow to G1, G2, G3."""
    return _TTEmbeddingBagFn.apply(G1, G2, G3, emb, idx, offsets, emb._nb(idx, offsets, num_bags))


class _TTEmbeddingBagNFn(torch.autograd.Function):
    """Autograd node of the pooled gather with any number of cores (forward_n /
    backward_n; the grouping is reused as in the three-core node)."""

    @staticmethod
    def forward(ctx, emb, idx, offsets, num_bags, *cores):
        out = emb.forward_n(cores, idx, offsets, num_bags=num_bags)
        ctx.emb, ctx.idx, ctx.offsets, ctx.num_bags = emb, idx, offsets, num_bags
        ctx.save_for_backward(*cores)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        cores = ctx.saved_tensors
        emb = ctx.emb
        g = grad_out.contiguous().to(torch.float32)
        try:
            grads = emb.backward_n(cores, ctx.idx, ctx.offsets, g, num_bags=ctx.num_bags, reuse_grouping=True)
        except N.TTEmbError as e:
            if e.code != N.TT_EMB_EINVAL:
                raise
            grads = emb.backward_n(cores, ctx.idx, ctx.offsets, g, num_bags=ctx.num_bags, reuse_grouping=False)
        return (None, None, None, None, *grads)


def tt_embedding_bag_n(cores, emb, idx, offsets=None, num_bags=None):
    """Differentiable pooled lookup over L cores: out [T][B][D], gradients flow to every core."""
    return _TTEmbeddingBagNFn.apply(emb, idx, offsets, emb._nb(idx, offsets, num_bags), *cores)


class TTEmbeddingBag(torch.nn.Module):
    """T sum-pooled embedding tables of one TT shape, the cores as parameters
    G1 .. GL (L = len(row_factors); G1, G2, G3 for three cores).

    forward(idx, offsets) returns [T][B][D]; loss.backward() fills the cores' .grad.
    step_fused(idx, offsets, grad_out, lr) is the training step without autograd:
    for three cores backward and SGD in one library call (no gradient tensors);
    for other L, backward_n into temporary gradients and sgd_n.
    """

    def __init__(self, num_tables, num_rows, row_factors, dim_factors, rank, max_indices, max_bags, init_std=0.05,
                 reuse="prefix", device="cuda", generator=None):
        super().__init__()
        self.emb = TTEmbedding(num_tables, num_rows, row_factors, dim_factors, rank, max_indices, max_bags,
                               device=device, reuse=reuse)

        def init(shape):
            return torch.nn.Parameter(
                (torch.randn(shape, generator=generator, dtype=torch.float32) * init_std).to(device))

        for k, shape in enumerate(self.emb.core_shapes()):
            setattr(self, f"G{k + 1}", init(shape))

    @property
    def cores(self):
        return [getattr(self, f"G{k + 1}") for k in range(self.emb.L)]

    def forward(self, idx, offsets=None, num_bags=None):
        if self.emb.L == 3:
            return tt_embedding_bag(self.G1, self.G2, self.G3, self.emb, idx, offsets, num_bags)
        return tt_embedding_bag_n(self.cores, self.emb, idx, offsets, num_bags)

    @torch.no_grad()
    def step_fused(self, idx, offsets, grad_out, lr, num_bags=None, reuse_grouping=True):
        if self.emb.L == 3:
            self.emb.backward_sgd(self.G1.data, self.G2.data, self.G3.data, idx, offsets, grad_out.contiguous(), lr,
                                  num_bags=num_bags, reuse_grouping=reuse_grouping)
            return
        cores = [G.data for G in self.cores]
        grads = self.emb.backward_n(cores, idx, offsets, grad_out.contiguous(), num_bags=num_bags,
                                    reuse_grouping=reuse_grouping)
        self.emb.sgd_n(cores, grads, lr)
