"""Seeded workload generators: determinism, kept counts, tie rules (CPU only)."""
import numpy as np

import workloads as wl


def test_keep_count_rounding():
    assert wl.keep_count(8192, 40) == 4915  # 4915.2
    assert wl.keep_count(8192, 50) == 4096
    assert wl.keep_count(10, 45) == 6  # 5.5 rounds up
    assert wl.keep_count(5120, 50) == 2560


def test_tiny_is_deterministic_and_bernoulli():
    a = wl.make_instance("tiny", 16)
    b = wl.make_instance("tiny", 16)
    assert a.digests() == b.digests()
    d = a.nnz / a.W.size
    assert abs(d - 0.5) < 0.005
    assert a.W.shape == (1024, 1024) and a.X.shape == (16, 1024)
    w = a.W.view(np.float16).astype(np.float64)
    assert abs(w.std() - 0.02) < 0.001
    x = a.X.view(np.float16).astype(np.float64)
    assert abs(x.std() - 1.0) < 0.05


def test_per_row_topk_exact_counts_and_ties():
    score = np.array([[3, 1, 3, 2, 3, 0],
                      [5, 5, 5, 5, 5, 5]], dtype=np.uint16)
    m = wl.prune_per_row(score, 2)
    assert m.tolist() == [[1, 0, 1, 0, 0, 0], [1, 1, 0, 0, 0, 0]]
    m3 = wl.prune_per_row(score, 4)
    assert m3.tolist() == [[1, 0, 1, 1, 1, 0], [1, 1, 1, 1, 0, 0]]


def test_global_topk_exact_count_and_ties():
    W = np.array([[1, 4, 2], [4, 4, 0]], dtype=np.uint16)
    m = wl.prune_global(W, 3)
    assert m.tolist() == [[0, 1, 0], [1, 1, 0]]
    m2 = wl.prune_global(W, 2)  # ties at magnitude 4: lowest row-major index first
    assert m2.tolist() == [[0, 1, 0], [1, 0, 0]]
    rng = np.random.default_rng(0)
    W = rng.integers(0, 50, size=(40, 37)).astype(np.uint16)
    for keep in (0, 1, 100, 740, 1480):
        assert int(wl.prune_global(W, keep).sum()) == keep


def test_global_sign_ignored():
    W = np.array([[0x8005, 0x0004, 0x0003]], dtype=np.uint16)  # -5*ulp, 4*ulp, 3*ulp
    assert wl.prune_global(W, 1).tolist() == [[1, 0, 0]]


def test_attn13b_row_counts():
    inst = wl.make_instance("attn13b", 8)
    assert np.all(inst.mask.sum(axis=1) == 2560)
    # kept entries dominate dropped entries in magnitude, row by row
    mag = inst.W & 0x7FFF
    r = 17
    assert mag[r][inst.mask[r] == 1].min() >= mag[r][inst.mask[r] == 0].max()


def test_colscale_makes_column_density_nonuniform():
    # same rule as the 13B FFN pair, on a smaller shape
    rng = wl.seed_for(31, 1)
    K = 512
    s = rng.lognormal(0.0, 0.5, size=K)
    W = wl.gen._f16_bits(np.random.default_rng(1).normal(0, 0.02, size=(256, K)))
    absw = np.abs(W.view(np.float16).astype(np.float64))
    mask = wl.prune_per_row(absw * s[None, :], wl.keep_count(K, 50))
    assert np.all(mask.sum(axis=1) == 256)
    col = mask.mean(axis=0)
    assert col.std() > 0.1  # uniform pruning would give about 0.03


def test_instance_list_size():
    assert len(wl.instance_list()) == 38


# A shard is the first M/8 rows of its layer: whole seed chunks reproduce the
# layer's rows exactly, and per-row pruning keeps each row's mask its own.
def test_shard_rows_match_layer():
    sh = wl.make_instance("ffn70b_shard8", 1)
    assert (sh.M, sh.K, sh.sparsity_pct) == (3584, 8192, 50)
    full_rows = wl.draw_weights(5, 2048, 8192, "student_t4", 0.02)
    assert np.array_equal(full_rows, sh.W[:2048])
    assert np.array_equal(wl.make_x(5, 8192, 1), sh.X)
    kept = sh.mask.sum(axis=1)
    assert np.all(kept == wl.keep_count(8192, 50))
    assert len(wl.instance_list()) == 38
