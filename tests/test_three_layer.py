"""The CPU model of the paper's three-layer format (Section 3.2, Algorithm 1).

Pinned by the worked example of Section 3.2, by brute force over every window
pattern, by the closed forms of the layer sizes for independent keep
decisions, by exact round trips against the oracle's masked bits, and by the
format's structural invariants (2:4 layers, steps of 1..16, no-op dummies).
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from paper_2607_08786_amd import three_layer as tl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "pdd_worked_example.json")


def test_pdd_worked_example():
    g = json.load(open(GOLDEN))
    pts = [tuple(p) for p in g["points_t_r"]]
    code = tl.pdd_encode(pts)
    assert len(code) == 4 + len(pts) - 1          # 16 + 16 bits, then one byte per point
    assert tl.pdd_points(code) == pts
    (ta, ra), (tb, rb) = pts
    assert [tb - ta, rb - ra] == g["steps"][0]
    # Algorithm 1: each point moves W_t[t] to W_r[r] and clears W_t[t].
    wt = np.zeros(16, np.uint16)
    wt_idx = np.zeros(16, np.uint8)
    wt[6], wt[7] = 0x3C00, 0xC000                 # 1.0 and -2.0
    wt_idx[6], wt_idx[7] = 1, 3
    wr = np.zeros(16, np.uint16)
    wr_idx = np.zeros(16, np.uint8)
    tl.pdd_apply(code, wt, wt_idx, wr, wr_idx)
    assert wr[3] == 0x3C00 and wr[11] == 0xC000 and wr_idx[3] == 1 and wr_idx[11] == 3
    assert wt[6] == 0 and wt[7] == 0


def test_pdd_step_range():
    assert tl.pdd_points(tl.pdd_encode([(0, 0), (16, 16)])) == [(0, 0), (16, 16)]   # the largest step
    for bad in ([(0, 0), (17, 1)], [(0, 0), (1, 17)], [(5, 5), (5, 6)], [(5, 5), (6, 5)]):
        with pytest.raises(ValueError):
            tl.pdd_encode(bad)


def _roundtrip(bits, mask):
    enc = tl.encode(bits, mask)
    for t in enc.tiles:
        tl.check_tile(t)
    out = tl.decode(enc)
    assert np.array_equal(out, oracle.masked_bits(bits, mask.astype(np.uint8)))
    return enc


@pytest.mark.parametrize("p", [0.0, 0.1, 0.3, 0.5, 0.6, 0.8, 1.0])
def test_roundtrip_random(p):
    rng = np.random.default_rng(int(p * 100) + 7)
    M, K = 150, 300                                # partial tiles in both directions
    bits = rng.integers(1, 1 << 16, size=(M, K), dtype=np.uint16)
    mask = rng.random((M, K)) < p
    enc = _roundtrip(bits, mask)
    st = tl.layer_stats(enc.tiles, M, K)
    assert st["nnz"] == int(mask.sum())
    total = st["sparse_tc_frac"] + st["slot_filling_frac"] + st["residual_frac"]
    assert st["nnz"] == 0 or abs(total - 1.0) < 1e-12   # every kept entry is in exactly one layer


def test_roundtrip_special_values():
    # Opaque 16-bit words: -0.0, subnormals, Inf, NaN payloads round-trip; a kept
    # +0.0 decodes to the same +0.0 the masked matrix holds.
    rng = np.random.default_rng(3)
    bits = rng.choice(np.array([0x0000, 0x8000, 0x0001, 0x7C00, 0xFC00, 0x7E01, 0x3C00], np.uint16),
                      size=(64, 128))
    mask = rng.random((64, 128)) < 0.6
    _roundtrip(bits, mask)


def test_every_window_pattern():
    # Brute force: every one of the 16 masks of a 4-wide window, in every window
    # position of a tile; counts per layer follow the definitions.
    pat = np.array([[(v >> j) & 1 for j in range(4)] for v in range(16)], bool)
    mask = np.zeros((64, 128), bool)
    win_pat = (np.arange(64 * 32) * 7 + 3) % 16     # all 16 patterns, spread over rows
    mask.reshape(64, 32, 4)[:] = pat[win_pat.reshape(64, 32)]
    bits = (np.arange(64 * 128, dtype=np.int64) % 65535 + 1).astype(np.uint16).reshape(64, 128)
    tile = tl.encode_tile(bits, mask)
    tl.check_tile(tile)
    counts = pat.sum(1)[win_pat]
    assert tile.n_sparse_tc == int(np.minimum(counts, 2).sum())
    assert tile.n_surplus == int(np.maximum(counts - 2, 0).sum())
    assert tile.n_empty == int(np.maximum(2 - counts, 0).sum())
    assert tile.n_placed + len(tile.residual) == tile.n_surplus
    assert np.array_equal(tl.decode_tile(tile), np.where(mask, bits, 0).astype(np.uint16))


def test_structured_2of4_needs_no_other_layer():
    # A mask that is already 2:4 (two kept per window) fills the Sparse-TC layer
    # exactly: no surplus, no empty slot, no code, no residual.
    rng = np.random.default_rng(5)
    mask = np.zeros((64, 128), bool)
    for w in range(64 * 32):
        r, c = divmod(w, 32)
        mask[r, 4 * c + rng.choice(4, 2, replace=False)] = True
    bits = rng.integers(1, 1 << 16, size=(64, 128), dtype=np.uint16)
    tile = tl.encode_tile(bits, mask)
    assert tile.n_surplus == 0 and tile.n_empty == 0 and tile.codes == [] and len(tile.residual) == 0
    assert np.array_equal(tl.decode_tile(tile), np.where(mask, bits, 0).astype(np.uint16))


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_closed_forms_independent_masks(p):
    # Independent keep decisions with probability p: surplus per window
    # 4p^3(1-p) + 2p^4, empty slots per window 2(1-p)^4 + 4p(1-p)^3. 64 tiles =
    # 131072 windows; bounds of 5 standard deviations of the per-window counts.
    rng = np.random.default_rng(11)
    n_tiles = 64
    mask = rng.random((64 * n_tiles, 128)) < p
    bits = np.ones(mask.shape, np.uint16)
    tiles = [tl.encode_tile(bits[i * 64:(i + 1) * 64], mask[i * 64:(i + 1) * 64]) for i in range(n_tiles)]
    windows = n_tiles * 64 * 32
    q = [(1 - p) ** 4, 4 * p * (1 - p) ** 3, 6 * p ** 2 * (1 - p) ** 2, 4 * p ** 3 * (1 - p), p ** 4]
    sur = np.array([0, 0, 0, 1, 2]); emp = np.array([2, 1, 0, 0, 0])
    for got, vals, expect in ((sum(t.n_surplus for t in tiles), sur, tl.expected_surplus_per_window(p)),
                              (sum(t.n_empty for t in tiles), emp, tl.expected_empty_per_window(p))):
        var = float(np.dot(q, vals ** 2) - np.dot(q, vals) ** 2)
        assert abs(got / windows - expect) < 5 * np.sqrt(var / windows), (got / windows, expect)
    assert abs(tl.expected_surplus_fraction(0.5) - 3 / 16) < 1e-15


def test_dummies_are_noops():
    # Sparse surplus (70% sparsity) forces dummy points; with every kept value
    # nonzero, a point whose parked value is 0 is a dummy, and its W_r slot must
    # stay 0 after decoding.
    rng = np.random.default_rng(13)
    mask = rng.random((64, 128)) < 0.3
    bits = rng.integers(1, 1 << 16, size=(64, 128), dtype=np.uint16)
    tile = tl.encode_tile(bits, mask)
    assert tile.n_dummies > 0
    wt, wt_idx = tile.wt_vals.copy(), tile.wt_idx.copy()
    wr, wr_idx = np.zeros(tl.SLOTS, np.uint16), np.zeros(tl.SLOTS, np.uint8)
    dummy_r = [r for code in tile.codes for (t, r) in tl.pdd_points(code) if tile.wt_vals[t] == 0]
    assert len(dummy_r) == tile.n_dummies
    for code in tile.codes:
        tl.pdd_apply(code, wt, wt_idx, wr, wr_idx)
    assert all(wr[r] == 0 for r in dummy_r)
    assert np.array_equal(tl.decode_tile(tile), np.where(mask, bits, 0).astype(np.uint16))


def test_storage_bounds_and_workload_statistics():
    # Bitmap format: 2 bytes per kept value + 1 bit per position, exactly. The
    # three-layer format never costs less than its Sparse-TC layer, 1.125 bytes
    # per position. On the 13B attention masks (per-row top 50%), the layer
    # shares sit near the paper's (17.7% slot filling, under 1% residual;
    # approximate: the paper's masks come from pruned OPT weights).
    cfg = wl.CONFIGS["attn13b"]
    W = wl.draw_weights(cfg["cfg_id"], cfg["M"], cfg["K"], cfg["dist"], cfg["scale"])
    mask = wl.make_mask(cfg, W, 50)
    st = tl.sample_stats(W, mask, [0, 40])
    assert abs(st["bitmap_bytes_per_position"] - (2 * st["density"] + 1 / 8)) < 1e-12
    assert st["bytes_per_position"] >= 1.125
    assert 0.15 < st["slot_filling_frac"] < 0.21
    assert st["residual_frac"] < 0.02


# 2:4 window statistics of the sparse matrix-core operand shape (16 x 64).
def test_sparse_mfma_windows_pins():
    import numpy as np
    from paper_2607_08786_amd import three_layer as tl
    # An exact 2:4 mask: every window keeps its first two entries; one operand covers every block.
    m = np.tile(np.array([1, 1, 0, 0], dtype=np.uint8), (32, 32))
    st = tl.sparse_mfma_windows(m)
    assert st["window_kept_share"] == [0.0, 0.0, 1.0, 0.0, 0.0] and st["blocks_one_operand"] == 1.0
    # One window with 3 kept entries spoils exactly its own block.
    m2 = m.copy()
    m2[17, 64 + 2] = 1
    st2 = tl.sparse_mfma_windows(m2)
    assert st2["blocks"] == 4 and st2["blocks_one_operand"] == 0.75
    # Independent keep decisions: the window histogram is Binomial(4, p), and the closed form of
    # the one-operand share matches a large random mask at a density where it is not ~0.
    rng = np.random.default_rng(5)
    for p in (0.5, 0.05):
        mm = (rng.random((4096, 1024)) < p).astype(np.uint8)
        st3 = tl.sparse_mfma_windows(mm)
        binom = [1 * (1 - p) ** 4, 4 * p * (1 - p) ** 3, 6 * p ** 2 * (1 - p) ** 2, 4 * p ** 3 * (1 - p), p ** 4]
        assert np.allclose(st3["window_kept_share"], binom, atol=3e-3)
        assert abs(st3["blocks_one_operand"] - tl.expected_one_operand_blocks(p)) < 0.02
    assert tl.expected_one_operand_blocks(0.5) < 1e-40
