"""Seeded generators for the SpMM workloads.

Shapes follow the decode-phase setting of Section 5.1: the sparse weight W is
M x K, the dense activation X is K x N with N the batch of tokens, and the
product Y is M x N. Storage conventions used throughout this repository:

* W: row-major M x K fp16 (``nn.Linear.weight`` layout), returned as uint16
  bit patterns.
* mask: row-major M x K uint8, nonzero = the weight is kept.
* X: token-major, i.e. an N x K array whose row n is column n of the logical
  K x N matrix (the ``[B, H]`` activation of Section 2.1), fp16 bit patterns.

Every draw comes from ``numpy.random.default_rng(SeedSequence([2607, cfg_id,
stream, n_or_0, chunk]))`` with stream 0 = W values, 1 = mask / column scales,
2 = X, and ``chunk`` the index of a block of ``ROW_CHUNK`` rows (0 for draws
that are not chunked). Chunks are independent streams, so they are drawn in
parallel threads. W samples are drawn in float32 and cast to fp16 with
round-to-nearest-even; X in float64.

Pruning is magnitude based (Section 5.3 prunes with Wanda; real weights are not
available here, so magnitudes of synthetic weights stand in):

* per row: keep the ``keep_count(K, s)`` largest |w| of each row, ranking by the
  fp16 magnitude bits, ties to the lower column index;
* global: the same over the whole matrix, ties to the lower row-major index;
* per row with column scale (the 13B FFN pair): rank by |w| * s_k where s_k is a
  log-normal scale of input feature k, so the density of W's columns varies.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import hashlib
import os

import numpy as np

ROW_CHUNK = 1024
BASE_SEED = 2607
_WORKERS = max(1, min(16, os.cpu_count() or 1))


def seed_for(cfg_id: int, stream: int, n_or_0: int = 0, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([BASE_SEED, cfg_id, stream, n_or_0, chunk]))


def _parallel_chunks(M: int, fn) -> None:
    """Calls fn(chunk_index, r0, r1) for every ROW_CHUNK block of rows, in threads."""
    blocks = [(c, r0, min(M, r0 + ROW_CHUNK)) for c, r0 in enumerate(range(0, M, ROW_CHUNK))]
    if len(blocks) == 1 or _WORKERS == 1:
        for b in blocks:
            fn(*b)
        return
    with concurrent.futures.ThreadPoolExecutor(_WORKERS) as ex:
        for f in [ex.submit(fn, *b) for b in blocks]:
            f.result()


def keep_count(K: int, sparsity_pct: int) -> int:
    """Kept entries out of K at ``sparsity_pct`` percent sparsity: round((100-s)K/100), halves up."""
    return ((100 - sparsity_pct) * K * 2 + 100) // 200


def _f16_bits(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a.astype(np.float16)).view(np.uint16)


def draw_weights(cfg_id: int, M: int, K: int, dist: str, scale: float) -> np.ndarray:
    """M x K fp16 bit patterns; chunk c of ROW_CHUNK rows uses its own seed.

    normal: scale * Z; student_t4: scale * Z / sqrt(G / 2) with G ~ Gamma(2, 1),
    i.e. Z over the root of a chi-square(4) variable divided by its 4 degrees
    of freedom (Student's t with 4 degrees of freedom).
    """
    if dist not in ("normal", "student_t4"):
        raise ValueError(dist)
    out = np.empty((M, K), dtype=np.uint16)

    def fill(c, r0, r1):
        rng = seed_for(cfg_id, 0, 0, c)
        z = rng.standard_normal((r1 - r0, K), dtype=np.float32)
        if dist == "student_t4":
            g = rng.standard_gamma(2.0, size=(r1 - r0, K), dtype=np.float32)
            z /= np.sqrt(g * np.float32(0.5))
        z *= np.float32(scale)
        out[r0:r1] = z.astype(np.float16).view(np.uint16)

    _parallel_chunks(M, fill)
    return out


def make_x(cfg_id: int, K: int, N: int) -> np.ndarray:
    """N x K (token-major) fp16 bit patterns with entries N(0, 1)."""
    rng = seed_for(cfg_id, 2, N)
    return _f16_bits(rng.normal(0.0, 1.0, size=(N, K)))


def _magnitude_bits(W: np.ndarray) -> np.ndarray:
    return W & np.uint16(0x7FFF)


def prune_per_row(score: np.ndarray, keep: int) -> np.ndarray:
    """Keep the ``keep`` largest scores of each row (ties: lower column index)."""
    M, K = score.shape
    mask = np.zeros((M, K), dtype=np.uint8)
    if keep <= 0:
        return mask
    if keep >= K:
        mask[:] = 1
        return mask

    def fill(c, r0, r1):
        s = score[r0:r1]
        t = np.partition(s, K - keep, axis=1)[:, K - keep][:, None]  # keep-th largest
        gt = s > t
        eq = s == t
        need = keep - gt.sum(axis=1, keepdims=True)
        take_eq = eq & (np.cumsum(eq, axis=1) <= need)
        mask[r0:r1] = gt | take_eq

    _parallel_chunks(M, fill)
    return mask


def prune_global(W: np.ndarray, keep: int) -> np.ndarray:
    """Keep the ``keep`` largest |w| of the whole matrix (ties: lower row-major index)."""
    M, K = W.shape
    mask = np.zeros((M, K), dtype=np.uint8)
    if keep <= 0:
        return mask
    hists = [None] * ((M + ROW_CHUNK - 1) // ROW_CHUNK)

    def hist(c, r0, r1):
        hists[c] = np.bincount(_magnitude_bits(W[r0:r1]).ravel(), minlength=1 << 15)

    _parallel_chunks(M, hist)
    h = np.sum(hists, axis=0).astype(np.int64)
    ge = np.cumsum(h[::-1])[::-1]  # ge[t] = count(|w| bits >= t)
    t = int(np.nonzero(ge >= keep)[0].max())
    n_gt = int(ge[t + 1]) if t + 1 < len(ge) else 0
    need = keep - n_gt  # entries with magnitude bits == t to keep, lowest index first
    eq_counts = [0] * len(hists)

    def above(c, r0, r1):
        m = _magnitude_bits(W[r0:r1])
        mask[r0:r1] = m > t
        eq_counts[c] = int(np.count_nonzero(m == t))

    _parallel_chunks(M, above)
    for c, r0 in enumerate(range(0, M, ROW_CHUNK)):
        if need <= 0:
            break
        if eq_counts[c] == 0:
            continue
        r1 = min(M, r0 + ROW_CHUNK)
        idx = np.flatnonzero(_magnitude_bits(W[r0:r1]) == t)[:need]
        mask[r0:r1].reshape(-1)[idx] = 1
        need -= idx.size
    return mask


@dataclasses.dataclass
class Instance:
    name: str
    cfg_id: int
    M: int
    K: int
    N: int
    sparsity_pct: int
    prune: str
    W: np.ndarray  # uint16 M x K
    mask: np.ndarray  # uint8 M x K
    X: np.ndarray  # uint16 N x K

    def digests(self) -> dict:
        return {k: hashlib.sha256(np.ascontiguousarray(getattr(self, k)).tobytes()).hexdigest()
                for k in ("W", "mask", "X")}

    @property
    def nnz(self) -> int:
        return int(np.count_nonzero(self.mask))


# Layer shapes of the workloads. cfg_id keys the seeds.
CONFIGS = {
    "tiny": dict(cfg_id=1, M=1024, K=1024, dist="normal", scale=0.02, prune="bernoulli",
                 sparsity=(50,), Ns=(16,)),
    "attn13b": dict(cfg_id=2, M=5120, K=5120, dist="normal", scale=0.02, prune="row",
                    sparsity=(50,), Ns=(8, 16, 32)),
    "ffn13b_up": dict(cfg_id=31, M=13824, K=5120, dist="normal", scale=0.02, prune="row_colscale",
                      sparsity=(50,), Ns=(16, 64)),
    "ffn13b_down": dict(cfg_id=32, M=5120, K=13824, dist="normal", scale=0.02, prune="row_colscale",
                        sparsity=(50,), Ns=(16, 64)),
    "ffn66b": dict(cfg_id=4, M=36864, K=9216, dist="normal", scale=0.02, prune="global",
                   sparsity=(60, 50), Ns=(16, 64, 128)),
    "ffn70b": dict(cfg_id=5, M=28672, K=8192, dist="student_t4", scale=0.02, prune="row",
                   sparsity=(40, 50, 60, 70), Ns=(8, 16, 32, 64, 128, 256)),
}


# One GPU's share of a layer under row sharding (not part of the workload set
# above): the first M rows drawn with the layer's generator and seeds. Per-row
# pruning makes each row's mask independent of the others; rows of a partly
# drawn seed chunk are drawn from the same distribution as the full layer's.
SHARDS = {
    "ffn70b_shard8": dict(base="ffn70b", M=28672 // 8, sparsity=(50,)),  # 70B FFN over 8 GPUs: 3584 x 8192
}


def layer_config(name: str) -> dict:
    """The shape and generator settings of a workload or of a shard."""
    if name in SHARDS:
        sh = SHARDS[name]
        return dict(CONFIGS[sh["base"]], M=sh["M"], sparsity=sh["sparsity"])
    return CONFIGS[name]


def make_mask(cfg: dict, W: np.ndarray, sparsity_pct: int) -> np.ndarray:
    M, K = W.shape
    kind = cfg["prune"]
    if kind == "bernoulli":
        rng = seed_for(cfg["cfg_id"], 1)
        mask = np.empty((M, K), dtype=np.uint8)
        for r0 in range(0, M, ROW_CHUNK):
            r1 = min(M, r0 + ROW_CHUNK)
            mask[r0:r1] = rng.random((r1 - r0, K)) < (100 - sparsity_pct) / 100.0
        return mask
    if kind == "row":
        return prune_per_row(_magnitude_bits(W), keep_count(K, sparsity_pct))
    if kind == "row_colscale":
        rng = seed_for(cfg["cfg_id"], 1)
        s = rng.lognormal(0.0, 0.5, size=K)
        absw = np.abs(W.view(np.float16).astype(np.float64))
        return prune_per_row(absw * s[None, :], keep_count(K, sparsity_pct))
    if kind == "global":
        return prune_global(W, keep_count(M * K, sparsity_pct))
    raise ValueError(kind)


def make_instance(name: str, N: int, sparsity_pct: int | None = None) -> Instance:
    cfg = layer_config(name)
    s = cfg["sparsity"][0] if sparsity_pct is None else sparsity_pct
    W = draw_weights(cfg["cfg_id"], cfg["M"], cfg["K"], cfg["dist"], cfg["scale"])
    mask = make_mask(cfg, W, s)
    X = make_x(cfg["cfg_id"], cfg["K"], N)
    return Instance(name=name, cfg_id=cfg["cfg_id"], M=cfg["M"], K=cfg["K"], N=N,
                    sparsity_pct=s, prune=cfg["prune"], W=W, mask=mask, X=X)


def instance_list():
    """(name, N, sparsity) for every instance of the workload set."""
    out = []
    for name, cfg in CONFIGS.items():
        for s in cfg["sparsity"]:
            for N in cfg["Ns"]:
                out.append((name, N, s))
    return out


def make_random(M: int, K: int, N: int, density: float, seed: int, scale: float = 0.02,
                x_scale: float = 1.0):
    """Small ad-hoc case: W ~ N(0, scale), Bernoulli(density) mask, X ~ N(0, x_scale)."""
    rng = np.random.default_rng(np.random.SeedSequence([BASE_SEED, 999, seed, M, K, N]))
    W = _f16_bits(rng.normal(0.0, scale, size=(M, K)))
    mask = (rng.random((M, K)) < density).astype(np.uint8)
    X = _f16_bits(rng.normal(0.0, x_scale, size=(N, K)))
    return W, mask, X


def make_small_int(M: int, K: int, N: int, density: float, seed: int, lo: int = -3, hi: int = 3):
    """Small-integer W and X (exactly representable in fp16), Bernoulli(density) mask."""
    rng = np.random.default_rng(np.random.SeedSequence([BASE_SEED, 998, seed, M, K, N]))
    W = _f16_bits(rng.integers(lo, hi + 1, size=(M, K)).astype(np.float64))
    mask = (rng.random((M, K)) < density).astype(np.uint8)
    X = _f16_bits(rng.integers(lo, hi + 1, size=(N, K)).astype(np.float64))
    return W, mask, X


# Decoder blocks of the synthetic decode-step benchmark: one block's linear
# layers in execution order, (name, out, in, epilogue), with 13B shapes (hidden
# 5120, FFN 13824) and 70B-like shapes (hidden 8192, grouped K/V projections of
# 1024, FFN 28672); the FFN's first layer carries the activation, the output
# projection and the FFN's last layer a residual add. Weights as the workload
# set draws them, pruned per row to the given sparsity by magnitude.
BLOCKS = {
    "block13b": dict(cfg_id=70, hidden=5120, dist="normal", scale=0.02,
                     layers=[("q", 5120, 5120, "bias"), ("k", 5120, 5120, "bias"), ("v", 5120, 5120, "bias"),
                             ("o", 5120, 5120, "bias+residual"), ("up", 13824, 5120, "bias+relu"),
                             ("down", 5120, 13824, "bias+residual")]),
    "block70b": dict(cfg_id=80, hidden=8192, dist="student_t4", scale=0.02,
                     layers=[("q", 8192, 8192, "bias"), ("k", 1024, 8192, "bias"), ("v", 1024, 8192, "bias"),
                             ("o", 8192, 8192, "bias+residual"), ("up", 28672, 8192, "bias+relu"),
                             ("down", 8192, 28672, "bias+residual")]),
}


@dataclasses.dataclass
class BlockLayer:
    name: str
    M: int
    K: int
    W: np.ndarray       # fp16 bits M x K
    mask: np.ndarray    # uint8 M x K
    bias: np.ndarray    # fp16 bits [M]
    epilogue: str


def make_block(name: str, sparsity_pct: int = 50) -> list:
    cfg = BLOCKS[name]
    out = []
    for i, (lname, M, K, epi) in enumerate(cfg["layers"]):
        cid = cfg["cfg_id"] + i
        W = draw_weights(cid, M, K, cfg["dist"], cfg["scale"])
        mask = prune_per_row(_magnitude_bits(W), keep_count(K, sparsity_pct))
        bias = _f16_bits(seed_for(cid, 3).normal(0.0, cfg["scale"], size=M))
        out.append(BlockLayer(lname, M, K, W, mask, bias, epi))
    return out
