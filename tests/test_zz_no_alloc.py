"""The allocation-free forward (tt_emb_forward_noalloc): through the C ABI, two
calls in a row on one GPU (the second smaller, so it runs on what the first
left in the static scratch) give exactly what tt_emb_forward gives on a
caller-owned workspace, and the oracle's result to the scaled-error bound; a
call too large for the scratch is refused before anything is launched."""
import sys

import numpy as np
import pytest
import torch

import ttgen
from tests._util import abs_case, assert_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_03459_amd as P

    return P


def _dev(case):
    G = [torch.from_numpy(np.ascontiguousarray(case[k])).cuda() for k in ("G1", "G2", "G3")]
    idx = torch.from_numpy(np.ascontiguousarray(case["idx"], dtype=np.int64)).cuda()
    off = None if case["offsets"] is None else torch.from_numpy(np.ascontiguousarray(case["offsets"])).cuda()
    return G, idx, off


def _noalloc(lib, emb, case):
    G, idx, off = _dev(case)
    T, B, D = case["T"], case["B"], int(np.prod(case["d"]))
    out = torch.full((T, B, D), float("nan"), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    lib.N.tt_emb_forward_noalloc(emb.handle, G[0].data_ptr(), G[1].data_ptr(), G[2].data_ptr(), idx.data_ptr(),
                                 idx.numel(), None if off is None else off.data_ptr(), B, out.data_ptr(), stream)
    ref = emb.forward(*G, idx, off, num_bags=B)  # the same computation on a caller-owned workspace
    torch.cuda.synchronize()
    assert emb.check_errors() == 0
    return out.cpu().numpy().reshape(T * B, D), ref.cpu().numpy().reshape(T * B, D)


@pytest.mark.parametrize("cfg,bags", [(3, (400, 96)), (6, (400, 96)), (2, (20000, 3000))])
def test_noalloc_forward_two_calls(lib, orc, cfg, bags):
    first = ttgen.make(cfg, bags=bags[0], with_grad=False)
    second = ttgen.make(cfg, seed=ttgen.BASE_SEED + 1, bags=bags[1], with_grad=False)
    M = max(first["idx"].size, second["idx"].size)
    emb = lib.TTEmbedding(first["T"], first["N"], first["n"], first["d"], first["R"], max_indices=M,
                          max_bags=bags[0])
    for k, case in enumerate((first, second)):
        print(f"[noalloc] config {cfg} call {k + 1}: {case['B']} bags, {case['idx'].size} indices", flush=True)
        sys.stdout.flush()
        got, ref = _noalloc(lib, emb, case)
        assert np.array_equal(got, ref), f"call {k + 1} differs from tt_emb_forward"
        bags_s = ttgen.sample_bags(cfg, case["T"], case["B"], 64)
        r, _ = orc.forward(case, bags=bags_s)
        m, _ = orc.forward(abs_case(case), bags=bags_s)
        assert_close(f"noalloc config {cfg} call {k + 1}", got[bags_s], r, m)


def test_noalloc_refuses_calls_beyond_the_scratch(lib):
    case = ttgen.make(3, bags=4096, with_grad=False)  # about 650k indices: several hundred MB of workspace
    emb = lib.TTEmbedding(case["T"], case["N"], case["n"], case["d"], case["R"], max_indices=case["idx"].size,
                          max_bags=case["B"])
    G, idx, off = _dev(case)
    out = torch.zeros((case["T"], case["B"], 128), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    code = lib.N.lib.tt_emb_forward_noalloc(emb.handle, G[0].data_ptr(), G[1].data_ptr(), G[2].data_ptr(),
                                            idx.data_ptr(), idx.numel(), off.data_ptr(), case["B"], out.data_ptr(),
                                            stream)
    assert code == lib.N.TT_EMB_ESCRATCH
    assert "static scratch" in lib.N.status_string(code)
    torch.cuda.synchronize()
    assert float(out.abs().sum()) == 0.0  # nothing was launched
