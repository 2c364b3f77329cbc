"""The bench's algorithmic-work formulas against sums written out by hand for
small cases (the roofline numbers of the bench line rest on them)."""
import numpy as np

import bench
import synth


def test_path_work_single_image_by_hand():
    shape = synth.small_shape(n_layers=2, d_model=64, n_heads=1, mlp_hidden=128, vocab=256,
                              n_classes=3, grid=4)          # T = 16
    d, f, V, L = 64, 128, 256, 2
    k = np.array([13], dtype=np.int32)
    counts = np.array([[2], [1], [0]], dtype=np.int32)    # 13 -> 15 -> 16
    W, esz = 4, 2
    wb = (L * (4 * d * d + 3 * d * f) + d * V) * esz
    kvr = L * 2 * d * esz
    # prefill: rows 0..13, one logits row
    b = wb + 2 * 14 * kvr + V * 8 + V * 4
    fl = 2.0 * 14 * L * (4 * d * d + 3 * d * f) + 2.0 * d * V + 4.0 * d * L * sum(range(1, 15))
    for n in (13, 15):                                     # two rounds of W + 1 = 5 rows
        b += wb + n * kvr + 5 * kvr + 5 * V * 8 + V * 4
        fl += 2.0 * 5 * (L * (4 * d * d + 3 * d * f) + d * V)
        fl += 4.0 * d * L * sum(n + i + 1 for i in range(5))
    got = bench.path_work(shape, k, counts, W, 1, esz)
    assert got == (b, fl)


def test_path_work_counts_only_active_images_and_cfg_branches():
    shape = synth.small_shape(n_layers=1, d_model=64, n_heads=1, mlp_hidden=64, vocab=128,
                              n_classes=3, grid=4)
    k = np.array([16, 10], dtype=np.int32)                 # image 0 is complete
    counts = np.array([[0, 6], [0, 0]], dtype=np.int32)
    one = bench.path_work(shape, k[1:], counts[:, 1:], 6, 1)
    both = bench.path_work(shape, k, counts, 6, 1)
    assert one == both
    b1, f1 = bench.path_work(shape, k[1:], counts[:, 1:], 6, 1)
    b2, f2 = bench.path_work(shape, k[1:], counts[:, 1:], 6, 2)
    assert b2 > b1 and f2 > f1


def test_rollout_work_gemm_launches_by_hand():
    shape = synth.WORKLOADS["llamagen_b"].model
    k = np.array([100, 255], dtype=np.int32)
    counts = np.array([[5, 1], [4, 0], [0, 0]], dtype=np.int32)
    d, L = 768, 12
    b, fl = bench.rollout_work("qkv", shape, k, counts, 16, 1)
    per = lambda rows: (3 * d * d * 2 + rows * d * 2 + rows * 3 * d * 2, 2.0 * rows * 3 * d * d)
    # prefill, then rounds with 2, 1 and 1 active images (image 0 is still
    # short of T after the last listed round)
    rows = [101 + 256, 2 * 17, 1 * 17, 1 * 17]
    assert b == sum(L * per(r)[0] for r in rows)
    assert fl == sum(L * per(r)[1] for r in rows)
