"""Host encoder/decoder of the compressed format: bit-exact round trips and the
closed-form record size, on the CPU (the product's encoder source built with g++)."""
import numpy as np
import pytest

import native_host
import oracle
import workloads as wl


@pytest.fixture(scope="module")
def hlib(tmp_path_factory):
    return native_host.build(str(tmp_path_factory.mktemp("hostenc")))


def expected_bytes(mask: np.ndarray) -> int:
    """512 mask bytes per 16 x 256 tile plus 2 bytes per kept value, each record padded to 16 bytes."""
    M, K = mask.shape
    RB, KT = -(-M // 16), -(-K // 256)
    mp = np.zeros((RB * 16, KT * 256), dtype=np.int64)
    mp[:M, :K] = mask != 0
    per_tile = mp.reshape(RB, 16, KT, 256).sum(axis=(1, 3))
    return int(np.sum(512 + (2 * per_tile + 15) // 16 * 16))


def check(hlib, W, mask):
    Wo, mo, nnz, sb, tiles = native_host.roundtrip(hlib, W, mask)
    assert np.array_equal(Wo, oracle.masked_bits(W, mask))
    assert np.array_equal(mo, (mask != 0).astype(np.uint8))
    assert nnz == int(np.count_nonzero(mask))
    assert sb == expected_bytes(mask)
    assert tiles == -(-W.shape[0] // 16) * -(-W.shape[1] // 256)


SPECIAL_BITS = np.array([0x0000, 0x8000, 0x0001, 0x03FF, 0x8001, 0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF,
                         0x3C00, 0xBC00, 0x7BFF], dtype=np.uint16)


def adversarial_masks(M, K, rng):
    yield "zero", np.zeros((M, K), np.uint8)
    yield "ones", np.ones((M, K), np.uint8)
    one = np.zeros((M, K), np.uint8)
    one[M // 2, K // 3] = 1
    yield "one", one
    yield "checker", ((np.arange(M)[:, None] + np.arange(K)[None, :]) % 2).astype(np.uint8)
    row = np.zeros((M, K), np.uint8)
    row[min(5, M - 1)] = 1
    yield "dense_row", row
    col = np.zeros((M, K), np.uint8)
    col[:, min(7, K - 1)] = 1
    yield "dense_col", col
    win = np.zeros((M, K), np.uint8)
    win[:, 0::8] = win[:, 1::8] = win[:, 2::8] = win[:, 3::8] = 1  # full then empty 4-windows
    yield "full_empty_windows", win
    yield "nonbool_values", (rng.random((M, K)) < 0.5).astype(np.uint8) * rng.integers(1, 256, (M, K)).astype(np.uint8)
    for d in (0.05, 0.3, 0.5, 0.7, 0.95):
        yield f"bern{d}", (rng.random((M, K)) < d).astype(np.uint8)


@pytest.mark.parametrize("shape", [(16, 256), (1, 1), (3, 5), (17, 257), (37, 300), (64, 1000), (100, 513)])
def test_roundtrip_adversarial(hlib, shape):
    M, K = shape
    rng = np.random.default_rng(M * 1000 + K)
    W = rng.integers(0, 1 << 16, size=(M, K)).astype(np.uint16)  # arbitrary bit patterns incl. NaN payloads
    W[:, ::3] = SPECIAL_BITS[np.arange(W[:, ::3].size) % SPECIAL_BITS.size].reshape(W[:, ::3].shape)
    for name, mask in adversarial_masks(M, K, rng):
        check(hlib, W, mask)


def test_roundtrip_workloads(hlib):
    for name in ("tiny", "attn13b"):
        inst = wl.make_instance(name, 8)
        check(hlib, inst.W, inst.mask)


def test_record_layout_matches_definition(hlib):
    """Decode one record by hand from its documented layout: lane-major mask bytes; values in
    blocks of (step, nibble half), lanes in order within a block."""
    import ctypes
    rng = np.random.default_rng(5)
    M, K = 16, 256
    W = rng.integers(1, 1 << 15, size=(M, K)).astype(np.uint16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    size = expected_bytes(mask)
    stream = np.zeros(size, np.uint8)
    off = np.zeros(2, np.uint32)
    hlib.usp_test_records(W.ctypes.data, mask.ctypes.data, M, K, stream.ctypes.data, off.ctypes.data)
    assert off[0] == 0 and off[1] * 16 == size
    vals = stream[512:].view(np.uint16)
    v = 0
    for s in range(8):
        for lane in range(64):
            r, g = lane % 16, lane // 16
            byte = stream[8 * lane + s]
            for j in range(8):
                assert ((byte >> j) & 1) == mask[r, 32 * s + 8 * g + j]
        for h in range(2):
            for lane in range(64):
                r, g = lane % 16, lane // 16
                for j in range(4 * h, 4 * h + 4):
                    k = 32 * s + 8 * g + j
                    if mask[r, k]:
                        assert vals[v] == W[r, k]
                        v += 1
    assert v == mask.sum()
    assert np.all(stream[512 + 2 * v:] == 0)


def test_roundtrip_under_sanitizers(tmp_path):
    """Random round trips in a standalone driver built with AddressSanitizer and UBSan."""
    import os
    import subprocess
    root = native_host.ROOT
    exe = os.path.join(str(tmp_path), "encode_fuzz")
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    "-fno-sanitize-recover=all", "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "native", "encode_fuzz_main.cpp"),
                    os.path.join(root, "paper_2607_08786_amd", "csrc", "usp_encode.cpp"),
                    "-o", exe, "-lpthread"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="verify_asan_link_order=0")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("ok")
