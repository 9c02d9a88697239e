"""GPU parity of the sparse product against the CPU oracle, through the C ABI.

Bit-exact where the arithmetic is exact (decode, densify, small-integer
products, identity columns, zero mask); elsewhere the acceptance bound
|Y - Yref| <= 1e-2 * (|W||X|) + 1e-3 elementwise and relative Frobenius error
<= 1e-3, with fp32 accumulation and fp16 output.
"""
import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture(scope="module")
def usp(torch):
    from paper_2607_08786_amd import usp as mod
    mod.load_library()
    return mod


def to_dev(torch, bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.float16)).cuda()


def run(torch, usp, W, mask, X, ldx_extra=0, offset=0):
    """Y (N x M float64) from the GPU path; X given as N x K fp16 bits."""
    A = usp.SparseMatrix(W, mask)
    N, K = X.shape
    if ldx_extra or offset:
        buf = torch.zeros(N * (K + ldx_extra) + offset + 8, dtype=torch.float16, device="cuda")
        Xv = buf[offset:offset + N * (K + ldx_extra)].view(N, K + ldx_extra)[:, :K]
        Xv.copy_(to_dev(torch, X))
    else:
        Xv = to_dev(torch, X)
    Y = A.spmm(Xv)
    torch.cuda.synchronize()
    A.free()
    return Y.cpu().numpy().astype(np.float64)


def assert_close(Y, W, mask, X, rows=None):
    Yref, Aref = oracle.masked_gemm(W, mask, X, rows=rows)
    res = oracle.check_tolerance(Y, Yref, Aref)
    assert res["ok"], res
    return res


@pytest.mark.parametrize("M,K,N", [(16, 256, 16), (64, 512, 16), (48, 768, 32), (37, 300, 7),
                                   (128, 1024, 64), (20, 600, 100), (1, 1, 1)])
def test_small_integers_exact(torch, usp, M, K, N):
    """Integer W in [-3, 3], X in [-1, 1]: every partial sum and the fp16 output are exact."""
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=1)
    X = (X.view(np.float16).astype(np.float64).clip(-1, 1)).astype(np.float16).view(np.uint16)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


@pytest.mark.parametrize("M,K", [(16, 256), (64, 1024), (37, 300), (100, 513), (5, 7)])
def test_densify_bit_exact(torch, usp, M, K):
    rng = np.random.default_rng(M + K)
    W = rng.integers(0, 1 << 16, size=(M, K)).astype(np.uint16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    A = usp.SparseMatrix(W, mask)
    Wd = A.densify()
    torch.cuda.synchronize()
    got = Wd.cpu().numpy().view(np.uint16)
    A.free()
    assert np.array_equal(got, oracle.masked_bits(W, mask))


def test_decode_roundtrip_through_device(torch, usp):
    rng = np.random.default_rng(3)
    W = rng.integers(0, 1 << 16, size=(50, 700)).astype(np.uint16)
    mask = (rng.random(W.shape) < 0.4).astype(np.uint8)
    A = usp.SparseMatrix(W, mask)
    Wo, mo = A.decode()
    info = A.info()
    A.free()
    assert np.array_equal(Wo, oracle.masked_bits(W, mask))
    assert np.array_equal(mo, mask)
    assert info["nnz"] == int(mask.sum()) and info["format_version"] == 2


def test_tiny_workload_parity(torch, usp):
    inst = wl.make_instance("tiny", 16)
    Y = run(torch, usp, inst.W, inst.mask, inst.X)
    assert_close(Y, inst.W, inst.mask, inst.X)


@pytest.mark.parametrize("N", [1, 7, 8, 15, 16, 17, 33, 64, 65, 128, 255, 256])
def test_n_sweep(torch, usp, N):
    W, mask, X = wl.make_random(96, 1280, N, 0.5, seed=N)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


@pytest.mark.parametrize("density", [0.0, 0.3, 0.4, 0.5, 0.6, 0.7, 1.0])
def test_density_sweep(torch, usp, density):
    W, mask, X = wl.make_random(80, 2048, 24, density, seed=int(density * 10))
    Y = run(torch, usp, W, mask, X)
    if density == 0.0:
        assert np.all(Y == 0)
    assert_close(Y, W, mask, X)


def test_identity_columns_recover_w(torch, usp):
    """X = [e_j1 ... e_jN] over every column j: Y reproduces W (masked) exactly."""
    M, K = 128, 1024
    W, mask, _ = wl.make_random(M, K, 1, 0.5, seed=11)
    A = usp.SparseMatrix(W, mask)
    Wm = oracle.masked_bits(W, mask)
    for j0 in range(0, K, 256):
        X = np.zeros((256, K), dtype=np.float16)
        X[np.arange(256), j0 + np.arange(256)] = 1.0
        Y = A.spmm(to_dev(torch, X.view(np.uint16)))
        torch.cuda.synchronize()
        got = Y.cpu().numpy()  # (256 tokens, M)
        exp = Wm[:, j0:j0 + 256].view(np.float16).T
        assert np.array_equal(got.astype(np.float64), exp.astype(np.float64)), j0
    A.free()


def test_deterministic_across_runs(torch, usp):
    W, mask, X = wl.make_random(320, 5120, 16, 0.5, seed=2)
    A = usp.SparseMatrix(W, mask)
    Xd = to_dev(torch, X)
    Y1 = A.spmm(Xd).clone()
    Y2 = A.spmm(Xd).clone()
    torch.cuda.synchronize()
    A.free()
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))


def test_strided_and_unaligned_x(torch, usp):
    W, mask, X = wl.make_random(64, 777, 9, 0.5, seed=4)
    Y = run(torch, usp, W, mask, X, ldx_extra=3, offset=1)
    assert_close(Y, W, mask, X)


def test_special_values_follow_ieee(torch, usp):
    M, K, N = 16, 256, 16
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=5)
    W = W.copy()
    mask = mask.copy()
    W[0, 3], mask[0, 3] = 0x7C00, 1  # +Inf kept
    W[1, 5], mask[1, 5] = 0x7E00, 1  # NaN kept
    W[2, 9], mask[2, 9] = 0x7C00, 0  # Inf pruned: no effect
    W[3, 0], mask[3, 0] = 0x0001, 1  # smallest subnormal kept
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(np.isnan(Y), np.isnan(Yref))
    fin = ~np.isnan(Yref)
    assert np.array_equal(np.isinf(Y[fin]), np.isinf(Yref[fin]))
    ok = np.isfinite(Yref)
    assert np.allclose(Y[ok], Yref[ok], rtol=1e-2, atol=1e-3)


def test_zero_mask_gives_exact_zero(torch, usp):
    W, _, X = wl.make_random(64, 512, 16, 0.5, seed=6)
    Y = run(torch, usp, W, np.zeros(W.shape, np.uint8), X)
    assert np.all(Y == 0)


def test_workspace_contract(torch, usp):
    W, mask, X = wl.make_random(64, 4096, 16, 0.5, seed=7)
    A = usp.SparseMatrix(W, mask)
    need = A.workspace_size(16)
    if need:
        with pytest.raises(usp.UspError):
            usp.usp_spmm(A.handle, to_dev(torch, X), torch.empty((16, 64), dtype=torch.float16, device="cuda"),
                         None)
    A.free()


# Passes of 128 tokens (small matrices): 200 tokens on 4101 x 1000 run one pass
# of 128 and one of 72 (last row block ragged, K ends in a partial tile), exact
# on small integers; 128 tokens on a 13B attention-size random matrix,
# tolerance.
def test_wide_token_passes(torch, usp):
    W, mask, X = wl.make_small_int(4101, 1000, 200, 0.5, seed=81, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)
    W, mask, X = wl.make_random(5120, 5120, 128, 0.5, seed=82)
    A = usp.SparseMatrix(W, mask)
    Y = A.spmm(to_dev(torch, X))
    torch.cuda.synchronize()
    A.free()
    rows = np.sort(np.random.default_rng(3).choice(5120, 256, replace=False))
    got = Y.cpu().numpy().astype(np.float64)[:, rows]
    assert_close(got, W, mask, X, rows=rows)


# One zero-filled workspace shared by handles of different sizes, calls
# alternating: partials a call leaves behind must never be read as another
# handle's arrival counters (4101 x 3000 splits its row blocks through the
# column-chunk kernel, 36880 x 8088 through the direct-to-LDS kernel, and
# 4101 x 1000 at 48 tokens through the four-wavefront kernel). Exact small
# integers, every output.
def test_workspace_shared_between_handles(torch, usp):
    cases = [wl.make_small_int(4101, 3000, 16, 0.5, seed=71, lo=-1, hi=1),
             wl.make_small_int(36880, 8088, 16, 0.5, seed=72, lo=-1, hi=1),
             wl.make_small_int(4101, 1000, 48, 0.5, seed=73, lo=-1, hi=1)]
    mats = [usp.SparseMatrix(W, m) for W, m, _ in cases]
    need = max(A.workspace_size(X.shape[0]) for A, (_, _, X) in zip(mats, cases))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    refs = [oracle.masked_gemm(W, m, X)[0] for W, m, X in cases]
    for it in range(2):
        for A, (W, m, X), Yref in zip(mats, cases, refs):
            Y = A.spmm(to_dev(torch, X), workspace=ws)
            torch.cuda.synchronize()
            assert np.array_equal(Y.cpu().numpy().astype(np.float64), Yref), (it, A.M, A.K, X.shape[0])
    for A in mats:
        A.free()


# Full-size workloads, sampled output rows (the oracle computes them one by one),
# in the same launch configuration the benchmark times.
@pytest.mark.parametrize("name,N,s", [("attn13b", 16, 50), ("attn13b", 8, 50), ("attn13b", 32, 50), ("ffn13b_up", 64, 50),
                                      ("ffn13b_down", 16, 50), ("ffn70b", 16, 50), ("ffn70b", 256, 40),
                                      ("ffn70b", 32, 70), ("ffn66b", 16, 60)])
def test_workload_sampled_rows(torch, usp, name, N, s):
    inst = wl.make_instance(name, N, s)
    A = usp.SparseMatrix(inst.W, inst.mask)
    Y = A.spmm(to_dev(torch, inst.X))
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    rows = np.sort(np.unique(np.concatenate([rng.choice(inst.M, 192, replace=False),
                                             [0, 15, 16, inst.M - 1]])))
    got = Y.cpu().numpy().astype(np.float64)[:, rows]
    A.free()
    assert_close(got, inst.W, inst.mask, inst.X, rows=rows)


# Matrices large enough that the planner picks the direct-to-LDS kernel (every
# wavefront gets at least 8 units of 4 row blocks), checked on every output:
# M = 36880 leaves the last set of 4 row blocks one block short, K = 8088 ends
# in a partial column tile. Small integers in {-1, 0, 1} keep every partial sum
# exact in fp32 and the outputs exact in fp16, so that case is bit-exact.
def test_dma_kernel_exact_full(torch, usp):
    W, mask, X = wl.make_small_int(36880, 8088, 16, 0.5, seed=21, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


@pytest.mark.parametrize("density,N", [(0.7, 11), (0.95, 8)])
def test_dma_kernel_dense_records_full(torch, usp, density, N):
    W, mask, X = wl.make_random(36880, 8088, N, density, seed=22)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# Two blocks of 16 tokens through the direct-to-LDS kernel (each decoded step
# feeds two MFMAs): exact on small integers at 32 tokens, tolerance at 27.
def test_dma_kernel_two_token_blocks_exact(torch, usp):
    W, mask, X = wl.make_small_int(36880, 8088, 32, 0.5, seed=23, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


def test_dma_kernel_two_token_blocks_ragged(torch, usp):
    W, mask, X = wl.make_random(36880, 8088, 27, 0.5, seed=24)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# Records of fully dense tiles (8 KB of values) exceed the shared-decode
# kernel's 8 KB slots once the mask is added, so from 33 tokens such a layer
# stays on the direct-to-LDS kernel with 3-4 blocks per wavefront (the mask by
# its own load) and token groups above 64: tolerance at 48 and 100 tokens.
@pytest.mark.parametrize("N,route", [(48, "dma nb=3 tg=1"), (100, "dma nb=4 tg=2")])
def test_dma_kernel_dense_records_token_groups(torch, usp, N, route):
    W, mask, X = wl.make_random(36880, 8088, N, 1.0, seed=33 + N)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(N)
    A.free()
    print(f"case N={N}: {plan}", flush=True)
    assert plan.startswith(route), plan
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# The shared-decode kernel (33 to 256 tokens on large layers: four
# wavefronts decode one record each into LDS, each multiplies all four by its
# quarter of the tokens, X packed in product order first). Exact on small
# integers, every output, at 48 and 64 tokens (one block per wavefront, the
# last wavefronts partly or wholly without tokens), 128 (two), 176 (three, the
# last wavefront's third block empty) and 256 (four; at three and four the
# pipelined variant, which decodes the next unit while multiplying this one);
# tolerance at 40, 100 and 250 tokens. M = 36880 leaves the last set of 4 row blocks one block
# short, K = 8088 ends in a partial column tile (zeros in the packed X).
@pytest.mark.parametrize("N", [48, 64, 128, 176, 256])
def test_share_kernel_exact(torch, usp, N):
    W, mask, X = wl.make_small_int(36880, 8088, N, 0.5, seed=27 + N, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(N)
    A.free()
    print(f"case N={N}: {plan}", flush=True)
    assert plan.startswith("share"), plan
    assert ("pipelined" in plan) == (N > 128), plan  # 3-4 blocks per wavefront
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# 448 row sets on 512 resident workgroups (28672 x 5120 at 128 tokens): one
# whole row set per workgroup, no partials. Exact on small integers.
def test_share_kernel_whole_sets(torch, usp):
    W, mask, X = wl.make_small_int(28672, 5120, 128, 0.5, seed=35, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(128)
    A.free()
    print(f"case: {plan}", flush=True)
    assert plan.startswith("share nb=2 grid=448"), plan
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# The pipelined variant at two blocks per wavefront, which the planner takes
# on layers of fewer than 32 units per CU (5120 x 5120: 1600 units): exact at
# 128 tokens, tolerance at 100 (the last wavefront's second block partly past
# N).
@pytest.mark.parametrize("N,exact", [(128, True), (100, False)])
def test_share_kernel_pipelined_two_blocks(torch, usp, N, exact):
    if exact:
        W, mask, X = wl.make_small_int(5120, 5120, N, 0.5, seed=31, lo=-1, hi=1)
    else:
        W, mask, X = wl.make_random(5120, 5120, N, 0.5, seed=32)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(N)
    A.free()
    print(f"case N={N}: {plan}", flush=True)
    assert plan.startswith("share nb=2") and "pipelined" in plan, plan
    Y = run(torch, usp, W, mask, X)
    if exact:
        Yref, _ = oracle.masked_gemm(W, mask, X)
        assert np.array_equal(Y, Yref)
    else:
        assert_close(Y, W, mask, X)


@pytest.mark.parametrize("N", [40, 100, 250])
def test_share_kernel_ragged(torch, usp, N):
    W, mask, X = wl.make_random(36880, 8088, N, 0.5, seed=28 + N)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# A call the wave kernels cannot take (X not 16-byte aligned, ldx odd) on a
# shape that the shared-decode kernel serves otherwise: the passes of the
# four-wavefront kernel run in the workspace sized for both routes.
def test_share_shape_unaligned_x_passes(torch, usp):
    W, mask, X = wl.make_small_int(36880, 8088, 64, 0.5, seed=29, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X, ldx_extra=3, offset=1)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# 33 to 64 tokens on a matrix whose last row group has one real row block (257
# row blocks) and whose K ends in a partial tile, every output checked: exact
# on small integers at 48 tokens, tolerance at 33.
def test_mid_tokens_ragged_exact(torch, usp):
    W, mask, X = wl.make_small_int(4101, 1000, 48, 0.5, seed=31)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


def test_mid_tokens_random(torch, usp):
    W, mask, X = wl.make_random(4101, 3000, 33, 0.45, seed=32)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# Fused epilogue (usp_spmm_ex): Y = act(W X + bias) + residual against the
# oracle's product through the same epilogue, with the error scale carried
# through the activation's largest slope. Every kernel: the row-block kernel
# (1024 x 1024, 16 tokens), the column-chunk kernel (4101 x 1000, 16; two
# token blocks: 4101 x 3800 at 27 tokens, split over 4 chunks, and 16300 x
# 1000 at 17, unsplit), the four-wavefront kernel (48 tokens), the
# direct-to-LDS kernel (36880 x 8088: 16 tokens, 27 tokens, 100 tokens in
# token groups).
EPI_SMALL = [(1024, 1024, 16), (4101, 1000, 16), (4101, 3800, 27), (16300, 1000, 17), (4101, 1000, 48)]
EPI_LARGE = [((36880, 8088, 16), "gelu_tanh"), ((36880, 8088, 27), "silu"), ((36880, 8088, 100), "relu")]


def _epilogue_case(torch, usp, M, K, N, act, seed, rows=None, inplace=False, use_bias=True, use_res=True):
    W, mask, X = wl.make_random(M, K, N, 0.5, seed=seed)
    rng = np.random.default_rng(seed + 1)
    bias = rng.normal(0, 0.5, M).astype(np.float16).view(np.uint16)
    res = rng.normal(0, 1.0, (N, M)).astype(np.float16).view(np.uint16)
    A = usp.SparseMatrix(W, mask)
    Xd = to_dev(torch, X)
    bd = to_dev(torch, bias) if use_bias else None
    rd = to_dev(torch, res) if use_res else None
    if inplace:
        Y = rd.clone()
        A.spmm(Xd, Y=Y, bias=bd, residual=Y, activation=act)
    else:
        Y = A.spmm(Xd, bias=bd, residual=rd, activation=act)
    torch.cuda.synchronize()
    A.free()
    got = Y.cpu().numpy().astype(np.float64)
    Yref, Aref = oracle.masked_gemm(W, mask, X, rows=rows)
    cols = np.arange(M) if rows is None else rows
    got = got[:, cols]
    b64 = oracle.f16_to_f64(bias)[cols] if use_bias else None
    r64 = oracle.f16_to_f64(res)[:, cols] if use_res else None
    y, scale = oracle.linear_epilogue(Yref, Aref, oracle.ACTIVATIONS[act], bias=b64, residual=r64)
    out = oracle.check_tolerance(got, y, scale)
    assert out["ok"], (M, K, N, act, out)


@pytest.mark.parametrize("shape", EPI_SMALL)
@pytest.mark.parametrize("act", ["none", "relu", "gelu_tanh", "silu"])
def test_fused_epilogue_small(torch, usp, shape, act):
    M, K, N = shape
    _epilogue_case(torch, usp, M, K, N, act, seed=40 + M % 7 + N)


@pytest.mark.parametrize("case", EPI_LARGE)
def test_fused_epilogue_large(torch, usp, case):
    (M, K, N), act = case
    rows = np.sort(np.unique(np.concatenate([np.random.default_rng(2).choice(M, 200, replace=False),
                                             [0, 15, 16, M - 16, M - 1]])))
    _epilogue_case(torch, usp, M, K, N, act, seed=50 + N, rows=rows)


def test_fused_epilogue_inplace_residual_and_parts(torch, usp):
    # Residual read from Y itself (in-place add); bias alone; residual alone.
    _epilogue_case(torch, usp, 4101, 1000, 16, "silu", seed=61, inplace=True)
    _epilogue_case(torch, usp, 4101, 1000, 48, "gelu_tanh", seed=62, inplace=True)
    _epilogue_case(torch, usp, 1024, 1024, 16, "none", seed=63, use_res=False)
    _epilogue_case(torch, usp, 4101, 1000, 16, "none", seed=64, use_bias=False)


def test_sparse_linear_module(torch, usp):
    # The nn.Linear drop-in: 3-D input (2 x 8 tokens), fused ReLU and residual.
    from paper_2607_08786_amd.linear import SparseLinear
    torch.manual_seed(0)
    lin = torch.nn.Linear(1000, 4101).to("cuda", torch.float16)
    rng = np.random.default_rng(7)
    mask = (rng.random((4101, 1000)) < 0.5).astype(np.uint8)
    mod = SparseLinear.from_linear(lin, mask, activation="relu")
    x = torch.randn(2, 8, 1000, device="cuda", dtype=torch.float16)
    r = torch.randn(2, 8, 4101, device="cuda", dtype=torch.float16)
    y = mod(x, residual=r)
    y2 = mod(x, residual=r)
    torch.cuda.synchronize()
    assert y.shape == (2, 8, 4101) and torch.equal(y, y2)
    W = lin.weight.detach().cpu().numpy().view(np.uint16)
    X = x.reshape(16, 1000).cpu().numpy().view(np.uint16)
    Yref, Aref = oracle.masked_gemm(W, mask, X)
    b64 = oracle.f16_to_f64(lin.bias.detach().cpu().numpy().view(np.uint16))
    r64 = oracle.f16_to_f64(r.reshape(16, 4101).cpu().numpy().view(np.uint16))
    yref, scale = oracle.linear_epilogue(Yref, Aref, 1, bias=b64, residual=r64)
    out = oracle.check_tolerance(y.reshape(16, 4101).cpu().numpy().astype(np.float64), yref, scale)
    assert out["ok"], out
    # One workspace for every token count: 48 tokens (split row groups) and then
    # 16 and 48 again through the same module equal a fresh module's results.
    x48 = torch.randn(48, 1000, device="cuda", dtype=torch.float16)
    ya = mod(x48)
    yb = mod(x)
    yc = mod(x48)
    fresh = SparseLinear.from_linear(lin, mask, activation="relu")
    torch.cuda.synchronize()
    assert torch.equal(ya, yc) and torch.equal(ya, fresh(x48)) and torch.equal(yb, fresh(x))


# Every instance of the workload set (6 layers x sparsities x token counts, 38
# in all), at full size and in the benchmark's launch configuration: the
# encoding round-trips bit-exactly through the device copy, sampled output rows
# (including the first and last row blocks) meet the tolerance, and a second
# call reproduces the first bit for bit.
@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_every_instance(torch, usp, name):
    cfg = wl.CONFIGS[name]
    W = wl.draw_weights(cfg["cfg_id"], cfg["M"], cfg["K"], cfg["dist"], cfg["scale"])
    rng = np.random.default_rng(1)
    rows = np.sort(np.unique(np.concatenate([rng.choice(cfg["M"], 160, replace=False),
                                             [0, 15, 16, cfg["M"] - 16, cfg["M"] - 1]])))
    for s in cfg["sparsity"]:
        mask = wl.make_mask(cfg, W, s)
        A = usp.SparseMatrix(W, mask)
        Wd, md = A.decode()
        assert np.array_equal(md, mask)  # the generators' masks are 0/1
        assert np.array_equal(Wd, oracle.masked_bits(W, mask))
        del Wd, md
        for N in cfg["Ns"]:
            X = wl.make_x(cfg["cfg_id"], cfg["K"], N)
            Xd = to_dev(torch, X)
            Y1 = A.spmm(Xd)
            Y2 = A.spmm(Xd)
            torch.cuda.synchronize()
            assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16)), (name, s, N)
            got = Y1.cpu().numpy().astype(np.float64)[:, rows]
            Yref, Aref = oracle.masked_gemm(W, mask, X, rows=rows)
            res = oracle.check_tolerance(got, Yref, Aref)
            assert res["ok"], (name, s, N, res)
        A.free()


# More row blocks than CUs but few tiles: the column-chunk kernel (workgroups
# of 4 row blocks x 4 column tiles); 257 row blocks (the last one ragged, its
# row group mostly past M), K ending in a partial tile (one chunk), every
# output checked.
def test_chunk_kernel_exact_full(torch, usp):
    W, mask, X = wl.make_small_int(4101, 1000, 16, 0.5, seed=25)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Three chunks per row block, summed through the workspace; 13 tokens.
def test_chunk_kernel_split_random_full(torch, usp):
    W, mask, X = wl.make_random(4101, 3000, 13, 0.45, seed=26)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# 17 to 32 tokens on small matrices with more row blocks than CUs (the
# four-wavefront kernel): K of 2, 9 and 6 column tiles, ragged tokens; exact on
# small integers.
@pytest.mark.parametrize("M,K,N", [(4101, 512, 32), (5000, 2200, 20), (4101, 1300, 27)])
def test_two_token_blocks_small_exact(torch, usp, M, K, N):
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=M + 3 * K + N, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# More than 256 tokens on a large matrix: passes of 64 tokens of the
# four-wavefront kernel reusing one workspace, the row groups split across
# workgroups in every pass (300 tokens: 4 passes of 64 and one of 44); exact on
# small integers for 512 sampled rows, and the last row group (ragged, 1 real
# row block).
def test_many_passes_large_matrix_exact(torch, usp):
    W, mask, X = wl.make_small_int(36880, 8088, 300, 0.5, seed=93, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([rng.choice(36864, 512, replace=False), np.arange(36864, 36880)]))
    Yref, _ = oracle.masked_gemm(W, mask, X, rows=rows)
    assert np.array_equal(Y[:, rows], Yref)


# One GPU's share of the 70B FFN under 8-way row sharding (3584 x 8192: fewer
# row blocks than CUs, so the K dimension is split), every output against the
# oracle's tolerance.
@pytest.mark.parametrize("N", [16, 32, 64])
def test_sharded_layer_full(torch, usp, N):
    inst = wl.make_instance("ffn70b_shard8", N)
    Y = run(torch, usp, inst.W, inst.mask, inst.X)
    assert_close(Y, inst.W, inst.mask, inst.X)


# Column-chunk kernel with more workgroups than stay resident at once (13B FFN
# up shape: 216 row groups x 5 chunks), exact on small integers.
def test_chunk_kernel_many_workgroups_exact(torch, usp):
    W, mask, X = wl.make_small_int(13824, 5120, 16, 0.5, seed=91, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Column-chunk kernel at two blocks of 16 tokens (the chunk's X for 32 tokens
# in LDS, two MFMAs per decoded step; taken when one round of workgroups of 8
# row blocks covers at least half the CUs): the 13B attention shape, a ragged
# last row group with a short last chunk (15 column tiles: 4, 4, 4, 3) and
# ragged tokens, and no split (4 column tiles, 1019 row blocks); exact on small
# integers, every output.
@pytest.mark.parametrize("M,K,N", [(5120, 5120, 32), (4101, 3800, 27), (16300, 1000, 17)])
def test_chunk_kernel_two_blocks_exact(torch, usp, M, K, N):
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=M + 5 * K + N, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(N)
    A.free()
    assert plan.startswith("chunk") and "nb=2" in plan, plan
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Column-chunk kernel at two token blocks on random fp16 data: four chunks per
# row block summed through the workspace, 29 tokens, every output against the
# oracle's tolerance.
def test_chunk_kernel_two_blocks_random_full(torch, usp):
    W, mask, X = wl.make_random(4101, 4000, 29, 0.55, seed=27)
    Y = run(torch, usp, W, mask, X)
    assert_close(Y, W, mask, X)


# Column-chunk kernel with a short last chunk: 6 column tiles (chunks of 4 and
# 2) and 9 (4, 4 and 1), tokens 16, 7 and 11; exact on small integers.
@pytest.mark.parametrize("M,K,N", [(4101, 1300, 16), (4101, 1300, 7), (5000, 2200, 11)])
def test_chunk_kernel_short_last_chunk_exact(torch, usp, M, K, N):
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=M + K + N, lo=-1, hi=1)
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Capture in a HIP graph (as the benchmark does): two products per graph with
# their own workspace, replayed five times with eager work (an X update and an
# eager product) in between; every replay must equal the eager result bit for
# bit. The graph holds only the library's kernels (no memset node), and split
# products must leave their arrival counters at zero for the next replay. Every
# kernel: row-block (1024 x 1024, 16), column-chunk (5120 x 5120, 16 and, with
# two token blocks, 32; 5 chunks per row block), direct-to-LDS (36880 x 8088 at
# 16 tokens), shared-decode (36880 x 8088 at 100 tokens: the X-packing kernel,
# then the product) and four-wavefront (4101 x 1000, 48).
@pytest.mark.parametrize("M,K,N", [(1024, 1024, 16), (5120, 5120, 16), (5120, 5120, 32), (36880, 8088, 16),
                                   (36880, 8088, 100), (4101, 1000, 48)])
def test_graph_capture_replays(torch, usp, M, K, N):
    W, mask, X = wl.make_random(M, K, N, 0.5, seed=M + N)
    A = usp.SparseMatrix(W, mask)
    Xd = to_dev(torch, X)
    ws = A.make_workspace(N)
    Yg = torch.empty((N, M), dtype=torch.float16, device="cuda")
    Ye = torch.empty_like(Yg)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        A.spmm(Xd, Yg, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        A.spmm(Xd, Yg, workspace=ws)
        A.spmm(Xd, Yg, workspace=ws)
    ws_eager = A.make_workspace(N)
    for rep in range(5):
        Xd.mul_(-1.0 if rep % 2 else 1.0)  # eager work between replays (exact: sign flips)
        g.replay()
        A.spmm(Xd, Ye, workspace=ws_eager)
        torch.cuda.synchronize()
        assert torch.equal(Yg, Ye), (M, K, N, rep)
    if ws is not None:  # arrival counters (4 bytes per row block, rounded to sets of 4) back at zero
        RB = (M + 15) // 16
        assert int(ws[: 16 * ((RB + 3) // 4)].count_nonzero().item()) == 0
    A.free()


# The planner's routes on MI355X (256 CUs), one per rule it documents: the row
# kernel for few row blocks with few column tiles or few tokens; the
# column-chunk kernel for small layers at 9-16 tokens unless a row block would
# split into more than 8 chunks, and at 17-32 tokens when one round of its
# workgroups of 8 row blocks covers at least half the CUs; the direct-to-LDS
# kernel for large layers up to 32 tokens; the shared-decode kernel from 33 to
# 256 tokens on layers with at least 4 units of 4 row blocks per CU (the 70B
# FFN down projection, 13B attention at 128); the four-wavefront kernel
# otherwise, in passes above 256 tokens. The route depends only on the shape, the token count and
# the largest record, so a 50% Bernoulli mask over constant weights stands in.
# The column-chunk kernel takes 8 row blocks per workgroup when all its
# workgroups are resident at once, else 4.
ROUTES = [
    ((1024, 1024, 16), "row"), ((3584, 8192, 8), "row"),
    ((5120, 5120, 16), "chunk S=5 W=8"), ((5120, 5120, 8), "chunk S=5 W=8"), ((13824, 5120, 16), "chunk S=5 W=4"),
    ((3584, 8192, 16), "chunk S=8 W=8"),
    ((5120, 5120, 32), "chunk S=5 W=8 nb=2"), ((3584, 8192, 32), "chunk S=8 W=8 nb=2"),
    ((13824, 5120, 32), "fourwave passes=1 nt=2"), ((1024, 1024, 32), "fourwave passes=1 nt=2"),
    ((5120, 13824, 16), "fourwave passes=1 nt=1"),
    ((4101, 1000, 48), "fourwave passes=1 nt=3"), ((4101, 1000, 200), "fourwave passes=2 nt=8"),
    ((8192, 28672, 64), "share nb=1"), ((36880, 8088, 300), "fourwave passes=5 nt=4"),
    ((36880, 8088, 16), "dma nb=1 tg=1"), ((36880, 8088, 32), "dma nb=2 tg=1"),
    ((36880, 8088, 48), "share nb=1"), ((36880, 8088, 64), "share nb=1"), ((36880, 8088, 100), "share nb=2"),
    ((8192, 28672, 128), "share nb=2"), ((28672, 8192, 256), "share nb=4"), ((5120, 5120, 128), "share nb=2"),
    ((13824, 5120, 64), "share nb=1 grid=432"),
]


def test_planner_routes(torch, usp):
    rng = np.random.default_rng(11)
    cache = {}
    got = []
    for (M, K, N), want in ROUTES:
        if (M, K) not in cache:
            W = np.full((M, K), 0x3C00, dtype=np.uint16)
            mask = (rng.random((M, K), dtype=np.float32) < 0.5).astype(np.uint8)
            cache[(M, K)] = usp.SparseMatrix(W, mask)
        plan = cache[(M, K)].plan(N)
        got.append(((M, K, N), plan))
        assert plan.startswith(want), got
    for A in cache.values():
        A.free()


# Random shapes (fixed seeds): M, K from 1 to several thousand, N from 1 to 300,
# densities from 0 to 1, through whatever kernel the planner picks; exact on
# small integers, every output. Each case prints its shape and route first.
def _random_cases(count=32, seed=2607):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        M = int(rng.choice([1, 7, 16, 33, 250, 1023, 2049, 4101, 6000, 9000]))
        K = int(rng.choice([1, 9, 255, 256, 512, 704, 1504, 3000, 5120]))  # mostly multiples of 8
        N = int(rng.choice([1, 3, 8, 16, 17, 31, 48, 64, 65, 100, 129, 256, 300]))
        d = float(rng.choice([0.0, 0.05, 0.3, 0.5, 0.7, 1.0]))
        out.append((M, K, N, d, 100 + i))
    return out


@pytest.mark.parametrize("M,K,N,density,seed", _random_cases())
def test_random_shapes_exact(torch, usp, M, K, N, density, seed):
    W, mask, X = wl.make_small_int(M, K, N, density, seed=seed, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    print(f"case M={M} K={K} N={N} density={density}: {A.plan(N)}", flush=True)
    A.free()
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Concurrent host threads, each with its own handle, stream and workspace (the
# contract for concurrent calls), ten products each through the planner's
# different kernels; every result equals the single-threaded one bit for bit.
def test_concurrent_host_threads(torch, usp):
    import threading
    shapes = [(5120, 2048, 16), (4101, 1000, 48), (1024, 1024, 16), (36880, 8088, 16)]
    cases = []
    for i, (M, K, N) in enumerate(shapes):
        W, mask, X = wl.make_random(M, K, N, 0.5, seed=300 + i)
        A = usp.SparseMatrix(W, mask)
        Xd = to_dev(torch, X)
        ref = A.spmm(Xd)
        cases.append((A, Xd, ref))
    torch.cuda.synchronize()
    errors = []

    def work(A, Xd, ref):
        try:
            st = torch.cuda.Stream()
            ws = A.make_workspace(Xd.shape[0], stream=st)  # zeroed on st, before the products
            with torch.cuda.stream(st):
                for _ in range(10):
                    Y = A.spmm(Xd, workspace=ws)
            st.synchronize()
            if not torch.equal(Y, ref):
                errors.append((A.M, A.K))
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=c) for c in cases]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    for A, _, _ in cases:
        A.free()
    assert not errors, errors


# Long row blocks with few tokens: the row-block kernel serves them only while a
# wavefront's stretch of the offset table fits one 64-lane load (at most 126
# column tiles); 16 x 140000 at 4 tokens (547 column tiles) goes to another
# kernel. Exact on small integers, every output.
@pytest.mark.parametrize("M,K,N,route", [(16, 32256, 4, "row"), (16, 140000, 4, "fourwave"), (40, 90000, 8, "fourwave")])
def test_long_row_blocks_exact(torch, usp, M, K, N, route):
    W, mask, X = wl.make_small_int(M, K, N, 0.5, seed=K + N, lo=-1, hi=1)
    A = usp.SparseMatrix(W, mask)
    plan = A.plan(N)
    print(f"case M={M} K={K} N={N}: {plan}", flush=True)
    A.free()
    assert plan.startswith(route), plan
    Y = run(torch, usp, W, mask, X)
    Yref, _ = oracle.masked_gemm(W, mask, X)
    assert np.array_equal(Y, Yref)


# Handle lifetime: a freed handle is rejected by every entry point (it is looked
# up among the live handles, never dereferenced), and a second free is an error.
def test_freed_handle_rejected(torch, usp):
    W, mask, X = wl.make_random(64, 512, 16, 0.5, seed=8)
    A = usp.SparseMatrix(W, mask)
    h = A.handle
    usp.usp_free(h)
    A.handle = None
    lib = usp.load_library()
    Xd = to_dev(torch, X)
    Y = torch.empty((16, 64), dtype=torch.float16, device="cuda")
    assert lib.usp_spmm(h, Xd.data_ptr(), 512, Y.data_ptr(), 64, 16, None, 0, None) == 1
    assert "freed" in usp.usp_last_error()
    assert lib.usp_free(h) == 1
    assert lib.usp_workspace_size(h, 16) == 0


# Stress of the split-K protocol (partials stored with device-coherent stores,
# an arrival counter, the last arrival summing every slot in order): one graph
# holding a split product is replayed 2000 times for each split route, each
# replay compared bit for bit with the eager result, stopping at the first
# mismatch (checked on the device after every replay, read back every 250
# replays). Routes: column-chunk (5120 x 5120 at 16 tokens: 5 chunks per row
# block; at 32 tokens with two token blocks), direct-to-LDS (28672 x 8192 at 16
# and 64 tokens, row sets split over wavefronts), four-wavefront (4101 x 1000 at
# 48 tokens, row groups split over workgroups).
@pytest.mark.parametrize("M,K,N", [(5120, 5120, 16), (5120, 5120, 32), (28672, 8192, 16), (28672, 8192, 64),
                                   (4101, 1000, 48)])
def test_split_protocol_stress(torch, usp, M, K, N):
    W, mask, X = wl.make_random(M, K, N, 0.5, seed=700 + N)
    A = usp.SparseMatrix(W, mask)
    print(f"case M={M} K={K} N={N}: {A.plan(N)}", flush=True)
    assert A.workspace_size(N) > 0  # a split route
    Xd = to_dev(torch, X)
    ws = A.make_workspace(N)
    Ye = A.spmm(Xd, workspace=A.make_workspace(N))
    Yg = torch.empty_like(Ye)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        A.spmm(Xd, Yg, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        A.spmm(Xd, Yg, workspace=ws)
    ok = torch.ones((), dtype=torch.bool, device="cuda")
    for rep in range(2000):
        Yg.zero_()  # eager work between replays; a replay that skipped an output would leave a zero
        g.replay()
        ok &= (Yg.view(torch.int16) == Ye.view(torch.int16)).all()
        if rep % 250 == 249:
            torch.cuda.synchronize()
            assert bool(ok), (M, K, N, rep)
    torch.cuda.synchronize()
    assert bool(ok)
    A.free()
