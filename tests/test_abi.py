"""The C-ABI library loads on the CPU and exports every symbol the header declares;
host-side argument checks reject bad calls before anything is launched."""
import ctypes as C

import pytest


@pytest.fixture(scope="module")
def N():
    from paper_2609_03459_amd import _native

    return _native


def _desc(N, T=2, n=(3, 4, 5), d=(2, 2, 2), R=4, M=100, B=10, rows=None):
    x = N.tt_emb_desc()
    x.num_tables = T
    x.num_rows = rows if rows is not None else n[0] * n[1] * n[2]
    for k in range(3):
        x.row_factors[k] = n[k]
        x.dim_factors[k] = d[k]
    x.rank = R
    x.max_indices = M
    x.max_bags = B
    return x


def test_every_header_symbol_is_exported(N):
    names = N.header_symbols()
    assert len(names) >= 10
    for name in names:
        assert hasattr(N.lib, name), name


def test_create_destroy_and_workspace(N):
    h = N.tt_emb_create(_desc(N))
    ws = N.tt_emb_workspace_size(h, 100, 10)
    assert ws > 0 and ws % 256 == 0
    h2 = N.tt_emb_create(_desc(N, M=1000))
    assert N.tt_emb_workspace_size(h2, 1000, 10) > ws
    # sized per call: the same handle needs less for a smaller call, and as much
    # as a handle made for that size
    assert N.tt_emb_workspace_size(h2, 100, 10) == ws
    assert N.tt_emb_workspace_size(h2, 0, 0) < ws
    n = C.c_size_t()
    E = N.TT_EMB_EINVAL
    assert N.lib.tt_emb_workspace_size(h2, 1001, 10, C.byref(n)) == E  # beyond max_indices
    assert N.lib.tt_emb_workspace_size(h2, 10, 11, C.byref(n)) == E    # beyond max_bags
    assert N.lib.tt_emb_workspace_size(h2, -1, 10, C.byref(n)) == E
    assert N.lib.tt_emb_workspace_size(h2, 10, 10, None) == E
    assert N.lib.tt_emb_workspace_size(None, 10, 10, C.byref(n)) == E
    N.tt_emb_destroy(h)
    N.tt_emb_destroy(h2)


def test_workspace_of_the_training_workload(N):
    # 8 tables of 200 x 200 x 250 rows, d = (4, 4, 8), R = 32, 5,246,700 indices in
    # 32,768 bags per table: the bound on work slices (indices / 32 + prefix slots)
    # keeps the workspace near its E rows (2.69 GB) instead of one slice per index
    M, B = 5246700, 32768
    h = N.tt_emb_create(_desc(N, T=8, n=(200, 200, 250), d=(4, 4, 8), R=32, M=M, B=B))
    ws = N.tt_emb_workspace_size(h, M, B)
    rows = 4 * M * 128
    assert rows < ws < rows + 1.4e9, ws
    # and per call: a quarter of the batch needs well under half of it
    assert N.tt_emb_workspace_size(h, M // 4, B // 4) < ws / 2
    N.tt_emb_destroy(h)
    assert N.lib.tt_emb_destroy(None) == N.TT_EMB_OK
    assert N.status_string(N.TT_EMB_ERANGE).startswith("index")


@pytest.mark.parametrize("kw,code", [
    (dict(T=0), 1), (dict(R=0), 1), (dict(n=(3, 0, 5)), 1), (dict(d=(1, -1, 1)), 1),
    (dict(rows=61), 1), (dict(M=-1), 1),
    (dict(R=65), 5), (dict(T=100, n=(1000, 1000, 100)), 5), (dict(d=(64, 64, 2)), 5),
])
def test_create_rejects_bad_shapes(N, kw, code):
    h = C.c_void_p()
    assert N.lib.tt_emb_create(C.byref(_desc(N, **kw)), C.byref(h)) == code
    assert not h.value
    assert N.lib.tt_emb_create(None, C.byref(h)) == N.TT_EMB_EINVAL


def test_calls_reject_bad_arguments_without_launching(N):
    h = N.tt_emb_create(_desc(N, T=2, M=100, B=10))
    ws_bytes = N.tt_emb_workspace_size(h, 100, 10)
    ws_call = N.tt_emb_workspace_size(h, 20, 10)  # what a training call of 20 indices needs
    fake = 1 << 20  # aligned non-null addresses; nothing may be dereferenced
    off = fake
    E = N.TT_EMB_EINVAL
    f = N.lib.tt_emb_forward
    # null handle, null workspace, small workspace
    assert f(None, fake, fake, fake, fake, 20, None, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake, 20, None, 10, fake, 0, None, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake, 20, None, 10, fake, 0, fake, 256, None) == E
    # NULL offsets require num_indices == T*B
    assert f(h, fake, fake, fake, fake, 19, None, 10, fake, 0, fake, ws_bytes, None) == E
    # beyond capacities
    assert f(h, fake, fake, fake, fake, 101, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake, 20, off, 11, fake, 0, fake, ws_bytes, None) == E
    # indices without bags
    assert f(h, fake, fake, fake, fake, 5, off, 0, fake, 0, fake, ws_bytes, None) == E
    # null cores / output, misaligned pointers
    assert f(h, None, fake, fake, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake, 20, off, 10, None, 0, fake, ws_bytes, None) == E
    assert f(h, fake + 4, fake, fake, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake + 4, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, fake, fake, fake, fake, 20, off, 10, fake, 0, fake + 64, ws_bytes, None) == E
    # reuse of a grouping that was never made
    assert f(h, fake, fake, fake, fake, 20, off, 10, fake, 1, fake, ws_bytes, None) == E
    b = N.lib.tt_emb_backward
    assert b(h, fake, fake, fake, fake, 20, off, 10, fake, None, fake, fake, 0, fake, ws_bytes, None) == E
    assert b(h, fake, fake, fake, fake, 20, off, 10, fake, fake, fake, fake, 1, fake, ws_bytes, None) == E
    assert N.lib.tt_emb_sgd(h, fake, fake, None, fake, fake, fake, C.c_float(0.1), None) == E
    bs = N.lib.tt_emb_backward_sgd
    lr = C.c_float(0.1)
    assert bs(h, None, fake, fake, fake, 20, off, 10, fake, lr, 0, fake, ws_bytes, None) == E  # null core
    assert bs(h, fake, fake, fake + 4, fake, 20, off, 10, fake, lr, 0, fake, ws_bytes, None) == E  # misaligned
    assert bs(h, fake, fake, fake, fake, 20, off, 10, None, lr, 0, fake, ws_bytes, None) == E  # null grad_out
    assert bs(h, fake, fake, fake, fake, 20, off, 10, fake, lr, 1, fake, ws_bytes, None) == E  # no grouping yet
    assert bs(h, fake, fake, fake, fake, 20, off, 10, fake, lr, 0, fake, ws_call - 1, None) == E
    assert b(h, fake, fake, fake, fake, 20, off, 10, fake, fake, fake, fake, 0, fake, ws_call - 1, None) == E
    assert N.lib.tt_emb_group(h, fake, 20, off, 10, fake, 256, None) == E
    assert N.lib.tt_emb_group(h, None, 20, off, 10, fake, ws_bytes, None) == E
    assert N.lib.tt_emb_set_schedule(h, 4) == E and N.lib.tt_emb_set_schedule(h, -1) == E
    assert N.lib.tt_emb_set_schedule(None, 0) == E
    assert N.lib.tt_emb_set_schedule(h, 2) == N.TT_EMB_OK and N.lib.tt_emb_set_schedule(h, 0) == N.TT_EMB_OK
    assert N.lib.tt_emb_debug_grouping(h, fake, None, None, None, None, None, None, None, None, None) == E
    N.tt_emb_destroy(h)


def test_reuse_levels_and_workspace(N):
    h = N.tt_emb_create(_desc(N, T=2, M=1000, B=100))
    base = N.tt_emb_workspace_size(h, 1000, 100)
    assert N.lib.tt_emb_set_reuse(h, 3) == N.TT_EMB_EINVAL
    assert N.lib.tt_emb_set_reuse(h, -1) == N.TT_EMB_EINVAL
    assert N.lib.tt_emb_set_reuse(None, 0) == N.TT_EMB_EINVAL
    sizes = {}
    for name, level in N.REUSE.items():
        N.tt_emb_set_reuse(h, level)
        sizes[name] = N.tt_emb_workspace_size(h, 1000, 100)
    assert sizes["prefix"] == base
    # one slice per row (and per occurrence without dedup) needs more room
    assert sizes["unique"] >= base and sizes["none"] >= sizes["unique"]
    N.tt_emb_destroy(h)



@pytest.mark.parametrize("n,d,R,M,num,fwd,bwd", [
    ((200, 200, 250), (4, 4, 8), 32, 1 << 20, 1 << 20, 1, 1),   # both MFMA kernels
    ((400, 500, 500), (4, 4, 8), 64, 1 << 20, 1 << 20, 1, 1),   # both MFMA kernels at R = 64
    ((100, 100, 100), (4, 4, 4), 16, 1 << 20, 1 << 20, 0, 0),   # generic both ways
    ((6, 5, 252), (4, 4, 8), 32, 1000, 1000, 1, 1),             # the backward's LDS accumulator fills
    ((6, 5, 253), (4, 4, 8), 32, 1000, 1000, 1, 0),             # one row past it
    ((10, 10, 10), (4, 4, 8), 32, 1 << 24, 1 << 24, 0, 0),      # E offsets would pass 2^31
    ((10, 10, 10), (4, 4, 8), 32, 1 << 24, 1000, 1, 1),         # small call: both decide per call
    # 32-bit G2 offsets (T n2 4096 floats) or G1 offsets (T n1 128 floats) would pass 2^31: generic kernels
    ((1, 300000, 2), (4, 4, 8), 32, 1000, 1000, 0, 0),
    ((9000000, 1, 2), (4, 4, 8), 32, 1000, 1000, 0, 0),
    ((1, 70000, 2), (4, 4, 8), 64, 1000, 1000, 0, 0),
    # D = 32 = (4, 4, 2) at R = 32: both MFMA kernels, the backward within the same n3 bound
    ((200, 200, 250), (4, 4, 2), 32, 1 << 20, 1 << 20, 1, 1),
    ((6, 5, 252), (4, 4, 2), 32, 1000, 1000, 1, 1),
    ((6, 5, 253), (4, 4, 2), 32, 1000, 1000, 1, 0),
    ((10, 10, 10), (4, 4, 2), 32, 1 << 24, 1 << 24, 0, 0),
    ((10, 10, 10), (4, 4, 2), 64, 1000, 1000, 0, 0),            # D = 32 at R = 64: generic
    ((10, 10, 10), (4, 4, 1), 32, 1000, 1000, 0, 0),            # d3 = 1: generic
])
def test_kernel_uses_mfma(N, n, d, R, M, num, fwd, bwd):
    h = N.tt_emb_create(_desc(N, T=2, n=n, d=d, R=R, M=M, B=10))
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["fwd_fused"], num) == bool(fwd)
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["bwd_fused"], num) == bool(bwd)
    assert not N.tt_emb_kernel_uses_mfma(h, N.KERNELS["pool"], num)
    flag = C.c_int()
    E = N.TT_EMB_EINVAL
    assert N.lib.tt_emb_kernel_uses_mfma(h, 8, 0, C.byref(flag)) == E
    assert N.lib.tt_emb_kernel_uses_mfma(h, 2, M + 1, C.byref(flag)) == E
    assert N.lib.tt_emb_kernel_uses_mfma(h, 2, -1, C.byref(flag)) == E
    assert N.lib.tt_emb_kernel_uses_mfma(h, 2, 0, None) == E
    assert N.lib.tt_emb_kernel_uses_mfma(None, 2, 0, C.byref(flag)) == E
    N.tt_emb_destroy(h)


def test_r64_kernels_keep_one_tables_third_core_in_one_descriptor(N):
    # at R = 64 a table's third core takes n3 x 2,048 bytes, addressed through one buffer
    # descriptor of 32-bit extent: from n3 = 2^21 on the generic kernels serve
    for n3, mfma in ((1 << 21, False), ((1 << 21) - 1, True)):
        h = N.tt_emb_create(_desc(N, T=1, n=(1, 1, n3), d=(4, 4, 8), R=64, M=1000, B=10))
        assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["fwd_fused"], 1000) == mfma
        assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["bwd_fused"], 1000) == mfma
        N.tt_emb_destroy(h)


def _desc_n(N, L=4, T=2, n=(3, 4, 5, 2), d=(2, 2, 2, 1), R=4, M=100, B=10, rows=None):
    x = N.tt_emb_desc_n()
    x.num_tables = T
    x.num_cores = L
    x.num_rows = rows if rows is not None else int(__import__("numpy").prod(n[:L]))
    for k in range(min(len(n), N.MAX_CORES)):
        x.row_factors[k] = n[k]
        x.dim_factors[k] = d[k]
    x.rank = R
    x.max_indices = M
    x.max_bags = B
    return x


def test_create_n_shapes_and_workspace(N):
    # L = 3 through create_n is the three-core handle
    h3 = N.tt_emb_create(_desc(N))
    h3n = N.tt_emb_create_n(_desc_n(N, L=3, n=(3, 4, 5), d=(2, 2, 2)))
    assert N.tt_emb_workspace_size(h3, 100, 10) == N.tt_emb_workspace_size(h3n, 100, 10)
    # L = 4 and L = 2 need room for the merged / identity core and its gradient
    h4 = N.tt_emb_create_n(_desc_n(N))
    h2 = N.tt_emb_create_n(_desc_n(N, L=2, n=(12, 10), d=(4, 2)))
    assert N.tt_emb_workspace_size(h4, 100, 10) > 0 and N.tt_emb_workspace_size(h2, 100, 10) > 0
    h8 = N.tt_emb_create_n(_desc_n(N, L=8, n=(2,) * 8, d=(1, 2, 1, 2, 1, 2, 1, 2)))
    # wide merged cores are served too (their chain runs level by level in the workspace)
    h5 = N.tt_emb_create_n(_desc_n(N, L=5, n=(2, 2, 2, 2, 2), d=(8, 8, 2, 1, 1), R=64))
    assert N.tt_emb_workspace_size(h5, 100, 10) > N.tt_emb_workspace_size(h8, 100, 10)
    for h in (h3, h3n, h4, h2, h8, h5):
        N.tt_emb_destroy(h)


def test_kernel_uses_mfma_on_the_three_core_view(N):
    # four cores d = (2, 2, 4, 8) view as d = (4, 4, 8): the MFMA kernels serve them
    h = N.tt_emb_create_n(_desc_n(N, L=4, n=(10, 20, 10, 30), d=(2, 2, 4, 8), R=32, M=1000))
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["fwd_fused"], 1000)
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["bwd_fused"], 1000)
    assert not N.tt_emb_kernel_uses_mfma(h, N.KERNELS["merge"], 1000)
    N.tt_emb_destroy(h)
    # four cores d = (2, 2, 4, 2) view as d = (4, 4, 2), D = 32: the MFMA kernels too
    h = N.tt_emb_create_n(_desc_n(N, L=4, n=(10, 20, 10, 30), d=(2, 2, 4, 2), R=32, M=1000))
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["fwd_fused"], 1000)
    assert N.tt_emb_kernel_uses_mfma(h, N.KERNELS["bwd_fused"], 1000)
    N.tt_emb_destroy(h)
    # two cores d = (16, 8) view as d = (16, 1, 8) around an identity core: generic kernels
    h = N.tt_emb_create_n(_desc_n(N, L=2, n=(100, 100), d=(16, 8), R=32, M=1000))
    assert not N.tt_emb_kernel_uses_mfma(h, N.KERNELS["fwd_fused"], 1000)
    N.tt_emb_destroy(h)


@pytest.mark.parametrize("kw,code", [
    (dict(L=1), 1), (dict(L=9), 1), (dict(L=0), 1), (dict(T=0), 1), (dict(R=0), 1),
    (dict(n=(3, 0, 5, 2)), 1), (dict(d=(1, 1, -1, 1)), 1), (dict(rows=121), 1),
    (dict(n=(1000, 1000, 1000, 10)), 5), (dict(d=(16, 16, 16, 2)), 5), (dict(R=65), 5),
    # merged row product n0 n1 of 2^28 or more
    (dict(T=1, n=(1 << 14, 1 << 14, 2, 2), d=(1, 1, 2, 2)), 5),
])
def test_create_n_rejects_bad_shapes(N, kw, code):
    h = C.c_void_p()
    assert N.lib.tt_emb_create_n(C.byref(_desc_n(N, **kw)), C.byref(h)) == code
    assert not h.value
    assert N.lib.tt_emb_create_n(None, C.byref(h)) == N.TT_EMB_EINVAL


def test_calls_n_reject_bad_arguments_without_launching(N):
    h = N.tt_emb_create_n(_desc_n(N, T=2, M=100, B=10))
    ws_bytes = N.tt_emb_workspace_size(h, 100, 10)
    fake = 1 << 20
    off = fake
    E = N.TT_EMB_EINVAL
    cores = N.ptr_array([fake] * 4)
    short = N.ptr_array([fake, fake, None, fake])
    mis = N.ptr_array([fake, fake, fake + 4, fake])
    f = N.lib.tt_emb_forward_n
    assert f(h, None, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, short, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, mis, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert f(h, cores, fake, 20, off, 10, None, 0, fake, ws_bytes, None) == E
    assert f(h, cores, fake, 20, off, 10, fake, 0, fake, 256, None) == E
    assert f(h, cores, fake, 20, off, 10, fake, 1, fake, ws_bytes, None) == E  # no grouping yet
    b = N.lib.tt_emb_backward_n
    assert b(h, cores, fake, 20, off, 10, fake, None, 0, fake, ws_bytes, None) == E
    assert b(h, cores, fake, 20, off, 10, fake, short, 0, fake, ws_bytes, None) == E
    assert b(h, cores, fake, 20, off, 10, None, cores, 0, fake, ws_bytes, None) == E
    assert b(h, cores, fake, 20, off, 10, fake, cores, 0, fake, N.tt_emb_workspace_size(h, 20, 10) - 1, None) == E
    assert N.lib.tt_emb_sgd_n(h, cores, mis, C.c_float(0.1), None) == E
    assert N.lib.tt_emb_sgd_n(None, cores, cores, C.c_float(0.1), None) == E
    # the three-core calls refuse a handle with four cores
    lr = C.c_float(0.1)
    assert N.lib.tt_emb_forward(h, fake, fake, fake, fake, 20, off, 10, fake, 0, fake, ws_bytes, None) == E
    assert N.lib.tt_emb_backward(h, fake, fake, fake, fake, 20, off, 10, fake, fake, fake, fake, 0, fake,
                                 ws_bytes, None) == E
    assert N.lib.tt_emb_backward_sgd(h, fake, fake, fake, fake, 20, off, 10, fake, lr, 0, fake, ws_bytes,
                                     None) == E
    assert N.lib.tt_emb_sgd(h, fake, fake, fake, fake, fake, fake, lr, None) == E
    N.tt_emb_destroy(h)


def test_noalloc_forward_host_checks(N):
    # host-side refusals of the allocation-free forward, before any device call
    E = N.TT_EMB_EINVAL
    fake = 1 << 20
    h = N.tt_emb_create(_desc(N, T=8, n=(200, 200, 250), d=(4, 4, 8), R=32, M=1 << 20, B=32768))
    f = N.lib.tt_emb_forward_noalloc
    assert f(None, fake, fake, fake, fake, 20, fake, 10, fake, None) == E
    assert f(h, fake, fake, fake, fake, (1 << 20) + 1, fake, 10, fake, None) == E  # beyond max_indices
    assert f(h, fake, fake, fake, fake, 20, fake, 32769, fake, None) == E          # beyond max_bags
    assert f(h, fake, fake, fake, fake, -1, fake, 10, fake, None) == E
    # 10^6 indices of 128 floats need far more than the 64 MiB scratch
    assert f(h, fake, fake, fake, fake, 1 << 20, fake, 32768, fake, None) == N.TT_EMB_ESCRATCH
    assert "scratch" in N.status_string(N.TT_EMB_ESCRATCH)
    N.tt_emb_destroy(h)
    h4 = N.tt_emb_create_n(_desc_n(N))
    assert f(h4, fake, fake, fake, fake, 20, fake, 10, fake, None) == E  # four cores: not a three-core call
    N.tt_emb_destroy(h4)


def test_group_schedule_sizes_its_own_work_list(N):
    # the static prefix mapping cuts one chunk per prefix group: more chunk partials
    h = N.tt_emb_create(_desc(N, T=2, n=(20, 30, 40), d=(4, 4, 8), R=32, M=5000, B=100))
    base = N.tt_emb_workspace_size(h, 5000, 100)
    N.tt_emb_set_schedule(h, N.SCHED["group"])
    assert N.tt_emb_workspace_size(h, 5000, 100) > base
    N.tt_emb_set_schedule(h, N.SCHED["static"])
    assert N.tt_emb_workspace_size(h, 5000, 100) == base
    N.tt_emb_destroy(h)
