"""CPU model of the paper's three-layer storage format (Section 3.2, Algorithm 1).

Not on the GPU path: the kernels stream this library's own bitmap format. This
model encodes a pruned matrix the way Section 3.2 describes, decodes it with
the steps of Algorithm 1, and counts what each layer holds and costs, so the
two formats can be compared on the same masks.

Layers, per tile of 64 rows x 128 columns (windows of 4 consecutive columns,
32 per row, 2048 per tile):

* Sparse-TC layer W_t: a 2:4 matrix, two value slots per window with a 2-bit
  in-window index each. Slot t = 2 * (32 * row + window) + k. A window keeps its
  first two kept entries (by column) in slots 0 and 1; a window with fewer than
  two leaves empty slots (value 0).
* Slot-filling layer: the third and fourth kept entries of a window (surplus)
  belong to a second 2:4 matrix W_r, slot r = 2 * (32 * row + window) + (rank - 2).
  The encoder parks each surplus value in an empty slot of W_t, in order (the
  j-th surplus entry goes to the next usable empty slot), and writes its W_r
  in-window index into that slot's otherwise unused index field. The pairs
  (t, r) are delta coded (parallel differential distance, PDD): a code starts
  with t and r in 16 bits each, then one byte per point, the low nibble holding
  t's step minus 1 and the high nibble r's step minus 1 (steps of 1..16).
  Decoding a code moves W_t[t] (value and index field) to W_r[r] and clears
  W_t[t], point by point (Algorithm 1).
* Dummy points: when r would step by more than 16, the encoder spends the next
  empty slot of W_t as a stepping stone: it stays empty (value 0), and the
  point moves that 0 to a W_r slot strictly between two surplus entries, which
  no real point uses, so the move changes nothing.
* Codes: a step in t of more than 16 cannot be bridged (every empty slot
  before the next one used is already filled, none is left as a stepping
  stone), so a new code starts there; codes are independent (one per thread).
* Residual layer: surplus entries left over when a tile runs out of empty
  slots, stored as CSR (row pointers, column indices, values).

Readings where the paper is not specific: steps are stored minus 1; coordinates are compressed slot indices;
the first two entries of a window stay in the Sparse-TC layer; surplus and
empty slots pair in order within a tile; dummy points are the no-op moves
above; codes split where a step cannot be bridged; values are opaque 16-bit
words (a kept +0.0 is indistinguishable from an empty slot, which the product
cannot tell apart either).
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import sys
import time

import numpy as np

TILE_ROWS = 64
TILE_COLS = 128
WIN = 4
WINDOWS = TILE_COLS // WIN            # windows per tile row
SLOTS = 2 * TILE_ROWS * WINDOWS       # W_t (and W_r) slots per tile: 4096
MAX_STEP = 16                         # largest step a 4-bit field codes (stored minus 1)


# ---------------------------------------------------------------------------
# PDD codes (Algorithm 1's bit layout)
# ---------------------------------------------------------------------------

def pdd_encode(points) -> bytes:
    """One code for a run of (t, r) points: t and r of the first in 16 bits
    each (bits 0-15 and 16-31), then per point one byte, bits 0-3 = t step - 1,
    bits 4-7 = r step - 1."""
    points = list(points)
    if not points:
        raise ValueError("a code holds at least one point")
    t0, r0 = points[0]
    if not (0 <= t0 < 1 << 16 and 0 <= r0 < 1 << 16):
        raise ValueError("first point out of the 16-bit range")
    out = bytearray(int(t0 | (r0 << 16)).to_bytes(4, "little"))
    for (ta, ra), (tb, rb) in zip(points, points[1:]):
        dt, dr = tb - ta, rb - ra
        if not (1 <= dt <= MAX_STEP and 1 <= dr <= MAX_STEP):
            raise ValueError(f"step ({dt}, {dr}) outside 1..{MAX_STEP}")
        out.append((dt - 1) | ((dr - 1) << 4))
    return bytes(out)


def pdd_points(code: bytes):
    """The (t, r) points of a code, in order."""
    head = int.from_bytes(code[:4], "little")
    t, r = head & 0xFFFF, head >> 16
    pts = [(t, r)]
    for b in code[4:]:
        t += (b & 0xF) + 1
        r += (b >> 4) + 1
        pts.append((t, r))
    return pts


def pdd_apply(code: bytes, wt_vals, wt_idx, wr_vals, wr_idx) -> None:
    """Algorithm 1 on one code: for every point, W_r[r] <- W_t[t] (value and
    index field) and W_t[t] <- 0."""
    for t, r in pdd_points(code):
        wr_vals[r] = wt_vals[t]
        wr_idx[r] = wt_idx[t]
        wt_vals[t] = 0


# ---------------------------------------------------------------------------
# One tile
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Tile:
    wt_vals: np.ndarray            # uint16 [SLOTS]: Sparse-TC values, surplus parked in empty slots
    wt_idx: np.ndarray             # uint8 [SLOTS]: 2-bit in-window indices
    codes: list                    # PDD codes (bytes), one per independent run
    residual: np.ndarray           # int64 [n, 3]: (row, column, value bits), tile-local
    n_sparse_tc: int = 0           # kept entries that are a window's first or second
    n_surplus: int = 0             # third and fourth entries
    n_placed: int = 0              # surplus entries parked in W_t (real points)
    n_dummies: int = 0
    n_empty: int = 0               # empty W_t slots before filling
    n_gap_dummies: int = 0         # dummies if every step over 16 were bridged (ceil(step / 16) - 1 each)


def _window_ranks(mask):
    """Rank (0..3) of each kept entry within its window, -1 where not kept."""
    m = mask.reshape(mask.shape[0], -1, WIN).astype(np.int8)
    rank = np.cumsum(m, axis=-1) - 1
    return np.where(m > 0, rank, -1).reshape(mask.shape)


def encode_tile(bits: np.ndarray, mask: np.ndarray) -> Tile:
    """Encodes one 64 x 128 tile (uint16 value bits, bool mask)."""
    assert bits.shape == (TILE_ROWS, TILE_COLS) and mask.shape == bits.shape
    rank = _window_ranks(mask)
    rows, cols = np.nonzero(mask)                 # row-major: ascending window, then column
    rk = rank[rows, cols]
    win = rows * WINDOWS + cols // WIN
    wt_vals = np.zeros(SLOTS, np.uint16)
    wt_idx = np.zeros(SLOTS, np.uint8)
    tc = rk < 2
    t_slots = 2 * win[tc] + rk[tc]
    wt_vals[t_slots] = bits[rows[tc], cols[tc]]
    wt_idx[t_slots] = cols[tc] % WIN
    # Empty slots: k >= count of the window. Their index fields take the
    # window's unused positions, so W_t stays a valid 2:4 pattern.
    count = mask.reshape(TILE_ROWS, WINDOWS, WIN).sum(-1).reshape(-1)
    occupied = np.zeros(SLOTS, bool)
    occupied[t_slots] = True
    empty = np.nonzero(~occupied)[0]
    for w in np.nonzero(count < 2)[0]:
        used = set(wt_idx[2 * w + k] for k in range(count[w]))
        free = [p for p in range(WIN) if p not in used]
        for k in range(count[w], 2):
            wt_idx[2 * w + k] = free[k - count[w]]
    sp = ~tc
    s_r = 2 * win[sp] + (rk[sp] - 2)              # ascending
    s_val = bits[rows[sp], cols[sp]]
    s_idx = (cols[sp] % WIN).astype(np.uint8)
    s_row, s_col = rows[sp], cols[sp]

    codes, run = [], []
    n_placed = n_dummies = 0
    residual = []
    i = 0                                          # next empty slot
    t_prev = r_prev = None
    for j in range(len(s_r)):
        r = int(s_r[j])
        while True:
            if i >= len(empty):                    # no empty slot left in the tile
                residual.append((int(s_row[j]), int(s_col[j]), int(s_val[j])))
                break
            e = int(empty[i])
            if run and e - t_prev > MAX_STEP:      # cannot be bridged: a new code
                codes.append(pdd_encode(run))
                run = []
            if not run:
                run.append((e, r))
            elif r - r_prev <= MAX_STEP:
                run.append((e, r))
            else:                                  # dummy: e stays empty, its 0 lands between surplus slots
                run.append((e, r_prev + MAX_STEP))
                n_dummies += 1
                t_prev, r_prev = e, r_prev + MAX_STEP
                i += 1
                continue
            wt_vals[e] = s_val[j]
            wt_idx[e] = s_idx[j]
            n_placed += 1
            t_prev, r_prev = e, r
            i += 1
            break
    if run:
        codes.append(pdd_encode(run))
    res = np.array(residual, np.int64).reshape(-1, 3)
    # The statistic the paper quotes: splitting every long step of the real
    # points (in pairing order, within the tile) into steps of at most 16.
    real = [(t, r) for code in codes for (t, r) in pdd_points(code) if wt_vals[t] != 0]
    gaps = sum(max(0, -(-max(tb - ta, rb - ra) // MAX_STEP) - 1) for (ta, ra), (tb, rb) in zip(real, real[1:]))
    return Tile(wt_vals, wt_idx, codes, res, n_sparse_tc=int(tc.sum()), n_surplus=int(sp.sum()),
                n_placed=n_placed, n_dummies=n_dummies, n_empty=len(empty), n_gap_dummies=int(gaps))


def decode_tile(tile: Tile):
    """Dense 64 x 128 value bits from a tile: Algorithm 1 on every code, then
    W_t, W_r and the residual scattered to their positions."""
    wt_vals = tile.wt_vals.copy()
    wt_idx = tile.wt_idx.copy()
    wr_vals = np.zeros(SLOTS, np.uint16)
    wr_idx = np.zeros(SLOTS, np.uint8)
    for code in tile.codes:
        pdd_apply(code, wt_vals, wt_idx, wr_vals, wr_idx)
    out = np.zeros((TILE_ROWS, TILE_COLS), np.uint16)
    slot = np.arange(SLOTS)
    row, win = slot // (2 * WINDOWS), (slot // 2) % WINDOWS
    for vals, idx in ((wt_vals, wt_idx), (wr_vals, wr_idx)):
        nz = vals != 0
        out[row[nz], WIN * win[nz] + idx[nz]] = vals[nz]
    if len(tile.residual):
        out[tile.residual[:, 0], tile.residual[:, 1]] = tile.residual[:, 2].astype(np.uint16)
    return out


def check_tile(tile: Tile) -> None:
    """Structural invariants: both layers 2:4 (distinct indices per window where
    slots hold values), every step within 1..16, dummies are no-ops."""
    wt_vals = tile.wt_vals.copy()
    wt_idx = tile.wt_idx.copy()
    wr_vals = np.zeros(SLOTS, np.uint16)
    wr_idx = np.zeros(SLOTS, np.uint8)
    targets = set()
    for code in tile.codes:
        pts = pdd_points(code)
        for (ta, ra), (tb, rb) in zip(pts, pts[1:]):
            assert 1 <= tb - ta <= MAX_STEP and 1 <= rb - ra <= MAX_STEP
        for t, r in pts:
            assert r not in targets, "two points land on one W_r slot"
            targets.add(r)
        pdd_apply(code, wt_vals, wt_idx, wr_vals, wr_idx)
    for vals, idx in ((wt_vals, wt_idx), (wr_vals, wr_idx)):
        v = vals.reshape(-1, 2)
        i = idx.reshape(-1, 2)
        both = (v[:, 0] != 0) & (v[:, 1] != 0)
        assert np.all(i[both, 0] != i[both, 1]), "two values of a window share a position"


# ---------------------------------------------------------------------------
# Whole matrices
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Encoded:
    M: int
    K: int
    tiles: list                    # row-major over (M / 64) x (K / 128) tiles (padded)


def _tiles(bits, mask, rows=None):
    M, K = bits.shape
    Mp, Kp = -(-M // TILE_ROWS) * TILE_ROWS, -(-K // TILE_COLS) * TILE_COLS
    b = np.zeros((Mp, Kp), np.uint16)
    m = np.zeros((Mp, Kp), bool)
    b[:M, :K] = bits
    m[:M, :K] = mask.astype(bool)
    for ti in (range(Mp // TILE_ROWS) if rows is None else rows):
        for tj in range(Kp // TILE_COLS):
            sl = np.s_[ti * TILE_ROWS:(ti + 1) * TILE_ROWS, tj * TILE_COLS:(tj + 1) * TILE_COLS]
            yield ti, tj, b[sl], m[sl]


def encode(bits: np.ndarray, mask: np.ndarray) -> Encoded:
    """Encodes an M x K matrix (uint16 value bits, mask: nonzero = kept)."""
    bits = np.ascontiguousarray(bits, np.uint16)
    return Encoded(bits.shape[0], bits.shape[1], [encode_tile(b, m) for _, _, b, m in _tiles(bits, mask)])


def decode(enc: Encoded) -> np.ndarray:
    """Dense M x K value bits (pruned positions 0)."""
    nt = -(-enc.K // TILE_COLS)
    Mp = -(-enc.M // TILE_ROWS) * TILE_ROWS
    out = np.zeros((Mp, nt * TILE_COLS), np.uint16)
    for n, tile in enumerate(enc.tiles):
        ti, tj = divmod(n, nt)
        out[ti * TILE_ROWS:(ti + 1) * TILE_ROWS, tj * TILE_COLS:(tj + 1) * TILE_COLS] = decode_tile(tile)
    return out[:enc.M, :enc.K]


def layer_stats(tiles, M: int, K: int) -> dict:
    """Counts per layer and bytes per weight position (M: rows the tiles cover).

    Bytes: W_t values 2 B and index fields 2 bits per slot; a code 4 B plus 1 B
    per point after the first, and 4 B in a table of code starts; the residual
    in CSR with 2 B values, 4 B column indices and 4 B row pointers (M + 1)."""
    nnz = sum(t.n_sparse_tc + t.n_surplus for t in tiles)
    n = len(tiles)
    codes = sum(len(t.codes) for t in tiles)
    points = sum(t.n_placed + t.n_dummies for t in tiles)
    resid = sum(len(t.residual) for t in tiles)
    positions = n * TILE_ROWS * TILE_COLS
    b_tc = n * SLOTS * 2 + n * SLOTS // 4
    b_pdd = codes * 4 + (points - codes) + codes * 4
    b_res = resid * 6 + 4 * (M + 1) if resid else 0
    frac = lambda x: x / nnz if nnz else 0.0
    return {
        "tiles": n, "nnz": nnz, "density": nnz / positions,
        "sparse_tc_frac": frac(sum(t.n_sparse_tc for t in tiles)),
        "slot_filling_frac": frac(sum(t.n_placed for t in tiles)),
        "surplus_frac": frac(sum(t.n_surplus for t in tiles)),
        "dummy_frac": frac(sum(t.n_dummies for t in tiles)),
        "gap_dummy_frac": frac(sum(t.n_gap_dummies for t in tiles)),
        "residual_frac": frac(resid),
        "codes_per_tile": codes / n if n else 0.0,
        "bytes_per_position": (b_tc + b_pdd + b_res) / positions,
        "bitmap_bytes_per_position": (2 * nnz + positions / 8) / positions,
        "csr_bytes_per_position": (6 * nnz) / positions,
    }


def sample_stats(bits, mask, row_tiles) -> dict:
    """layer_stats over the tiles of the given tile rows (64-row bands)."""
    tiles = [encode_tile(b, m) for _, _, b, m in _tiles(np.asarray(bits, np.uint16), mask, rows=row_tiles)]
    return layer_stats(tiles, len(row_tiles) * TILE_ROWS, bits.shape[1])


# ---------------------------------------------------------------------------
# Closed forms for independent keep decisions (probability p per entry)
# ---------------------------------------------------------------------------

def expected_surplus_per_window(p: float) -> float:
    """A window with 3 kept entries has 1 surplus, with 4 kept 2."""
    return 4 * p ** 3 * (1 - p) + 2 * p ** 4


def expected_empty_per_window(p: float) -> float:
    """A window with no kept entry leaves 2 empty slots, with 1 kept 1."""
    return 2 * (1 - p) ** 4 + 4 * p * (1 - p) ** 3


def expected_surplus_fraction(p: float) -> float:
    return expected_surplus_per_window(p) / (4 * p)


def sparse_mfma_windows(mask: np.ndarray, rows: int = 16, k: int = 64) -> dict:
    """How a mask maps onto 2:4 sparse matrix-core operands (Sections 3.2, 4.3).

    A sparse MFMA of the 16 x 64 operand shape takes at most 2 kept entries in
    every 4 consecutive k of every row. Returns the share of 4-wide windows by
    kept count (0..4) and the share of rows x k blocks whose windows all hold at
    most 2, i.e. blocks one sparse operand covers; every other block needs a
    second operand for its windows' 3rd and 4th entries.
    """
    m = np.asarray(mask, dtype=np.uint8)
    R = m.shape[0] - m.shape[0] % rows
    C = m.shape[1] - m.shape[1] % k
    win = m[:R, :C].reshape(R, C // 4, 4).sum(axis=2)
    dist = np.bincount(win.ravel(), minlength=5)[:5] / win.size
    worst = win.reshape(R // rows, rows, C // k, k // 4).max(axis=(1, 3))
    return {"window_kept_share": [float(x) for x in dist], "share_over_2": float(dist[3] + dist[4]),
            "blocks_one_operand": float((worst <= 2).mean()), "blocks": int(worst.size)}


def expected_one_operand_blocks(p: float, rows: int = 16, k: int = 64) -> float:
    """Independent keep decisions with probability p: a block of rows x k/4
    windows fits one 2:4 operand when no window keeps 3 or 4 entries."""
    return (1 - 4 * p ** 3 * (1 - p) - p ** 4) ** (rows * k // 4)


# ---------------------------------------------------------------------------
# Report over the workload set (run as a module)
# ---------------------------------------------------------------------------

def _report(argv=None) -> int:
    ap = argparse.ArgumentParser(description="Three-layer format statistics on the synthetic workload masks")
    ap.add_argument("--bands", type=int, default=4, help="64-row bands sampled per matrix")
    ap.add_argument("--sparse-mfma", action="store_true",
                    help="2:4 window statistics (sparse_mfma_windows) on the first 4096 rows instead")
    args = ap.parse_args(argv)
    import workloads as wl
    rng = np.random.default_rng(0)
    for name, cfg in wl.CONFIGS.items():
        W = wl.draw_weights(cfg["cfg_id"], cfg["M"], cfg["K"], cfg["dist"], cfg["scale"])
        bands = sorted(rng.choice(-(-cfg["M"] // TILE_ROWS), size=min(args.bands, cfg["M"] // TILE_ROWS),
                                  replace=False).tolist())
        for s in cfg["sparsity"]:
            mask = wl.make_mask(cfg, W, s)
            t0 = time.perf_counter()
            if args.sparse_mfma:
                st = sparse_mfma_windows(mask[:4096])
            else:
                st = sample_stats(W, mask, bands)
                st.update(bands=bands)
            st.update(workload=name, sparsity_pct=s, seconds=time.perf_counter() - t0)
            print(json.dumps(st), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(_report())
