"""usp_spmm_noalloc (the entry point for callers that cannot allocate) against
usp_spmm, through the C ABI: bit for bit the same output on two calls in a row,
the second with a smaller input, both within the oracle's tolerance; a product
needing more workspace than the device scratch is refused with nothing
enqueued."""
import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu


def test_noalloc_matches_spmm_two_calls():
    import torch
    from paper_2607_08786_amd import usp
    assert torch.cuda.is_available()
    lib = usp.load_library()
    # First a split product (partials and arrival counters in the scratch), then a smaller one
    # through another kernel, then the four-wavefront and the shared-decode kernels (the latter
    # with packed X in the scratch too), then the first again: each equals usp_spmm bit for bit.
    cases = [wl.make_random(5120, 5120, 16, 0.5, seed=601), wl.make_random(1024, 1024, 8, 0.5, seed=602),
             wl.make_random(4101, 1000, 48, 0.5, seed=603), wl.make_random(5120, 5120, 128, 0.5, seed=605)]
    for i, (W, mask, X) in enumerate(cases + cases[:1]):
        print(f"case {i}: M={W.shape[0]} K={W.shape[1]} N={X.shape[0]}", flush=True)
        A = usp.SparseMatrix(W, mask)
        need = A.workspace_size(X.shape[0])
        print(f"  {A.plan(X.shape[0])}, workspace {need} bytes", flush=True)
        assert need <= usp.NOALLOC_SCRATCH_BYTES, need
        Xd = torch.from_numpy(X.view(np.float16)).cuda()
        Yn = torch.full((X.shape[0], A.M), float("nan"), dtype=torch.float16, device="cuda")
        usp.usp_spmm_noalloc(A.handle, Xd, Yn)
        Yr = A.spmm(Xd)
        torch.cuda.synchronize()
        assert torch.equal(Yn.view(torch.int16), Yr.view(torch.int16)), i
        Yref, Aref = oracle.masked_gemm(W, mask, X)
        res = oracle.check_tolerance(Yn.cpu().numpy().astype(np.float64), Yref, Aref)
        assert res["ok"], (i, res)
        A.free()
    del lib


def test_noalloc_refuses_oversized_products():
    import torch
    from paper_2607_08786_amd import usp
    W, mask, X = wl.make_small_int(36880, 8088, 256, 0.5, seed=604, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    need = A.workspace_size(256)
    print(f"workspace for 256 tokens: {need} bytes", flush=True)
    Xd = torch.from_numpy(X.view(np.float16)).cuda()
    Y = torch.zeros((256, A.M), dtype=torch.float16, device="cuda")
    if need <= usp.NOALLOC_SCRATCH_BYTES:
        pytest.skip("this product fits the scratch")
    with pytest.raises(usp.UspError) as e:
        usp.usp_spmm_noalloc(A.handle, Xd, Y)
    assert e.value.status == 2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert int(Y.count_nonzero().item()) == 0  # nothing was enqueued
    A.free()
