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
    alg, act, fl, n = bench.rollout_work("qkv", shape, k, counts, 16, 1)
    # algorithmic: the weights and the K, V rows appended to the cache;
    # activations: the normed input rows and the q rows
    per = lambda rows: (3 * d * d * 2 + rows * 2 * d * 2, rows * d * 2 + rows * d * 2,
                        2.0 * rows * 3 * d * d)
    # prefill, then rounds with 2, 1 and 1 active images (image 0 is still
    # short of T after the last listed round)
    rows = [101 + 256, 2 * 17, 1 * 17, 1 * 17]
    assert alg == sum(L * per(r)[0] for r in rows)
    assert act == sum(L * per(r)[1] for r in rows)
    assert fl == sum(L * per(r)[2] for r in rows)
    assert n == 4 * L


def test_rollout_work_attention_and_lm_head_by_hand():
    """Attention reads each sequence's committed K and V once per layer (the
    whole prefix in the prefill) and attends (W + 1)(n + 1) + W(W + 1)/2 keys
    per round and sequence; the lm_head reads its weights and writes one fp32
    logits row per row, on the last prefill row of each sequence only. Two
    guidance branches double every row."""
    shape = synth.small_shape(n_layers=2, d_model=64, n_heads=1, mlp_hidden=128, vocab=256,
                              n_classes=3, grid=4)          # T = 16
    d, V, L, W = 64, 256, 2, 4
    k = np.array([5, 16], dtype=np.int32)                  # image 1 is complete
    counts = np.array([[3, 0], [0, 0]], dtype=np.int32)    # 5 -> 8 -> 8
    for cfg in (1, 2):
        alg, act, fl, n = bench.rollout_work("attn", shape, k, counts, W, cfg)
        keys_pf = sum(range(1, 7))                          # rows 0..5 attend 1..6 keys
        keys_r = [5 * (c + 1) + W * (W + 1) // 2 for c in (5, 8)]
        assert fl == 4.0 * d * L * cfg * (keys_pf + sum(keys_r))
        assert alg == L * cfg * 2 * d * 2 * (6 + 5 + 8)
        assert act == L * cfg * 2 * d * 2 * (6 + 5 + 5)
        assert n == 3 * L
        alg, act, fl, n = bench.rollout_work("lmhead", shape, k, counts, W, cfg)
        rows = cfg * (1 + 5 + 5)
        assert alg == 3 * d * V * 2 + rows * V * 4
        assert act == rows * d * 2
        assert fl == 2.0 * rows * d * V and n == 3


# ------------------------------------------------------------------ rocprofv3 summaries

_WIDE = "void hbsjd::k_gemm_wide<hbsjd::EpiSwiGLU<unsigned short> >(unsigned short const*, int)"
_SMALL = ("void hbsjd::k_gemm_f16<128, 128, 2, 2, 3, false, hbsjd::EpiSwiGLU<unsigned short> >"
          "(unsigned short const*, int)")
_W2 = "void hbsjd::k_gemm_f16<64, 64, 2, 2, 3, true, hbsjd::EpiNone<1> >(unsigned short const*)"
_ATTN = "void hbsjd::k_attn_f16<2>(unsigned short const*, unsigned short*, int)"


def test_kernel_class_names():
    assert bench.kernel_class(_WIDE) == ("w13", True)
    assert bench.kernel_class(_SMALL) == ("w13", False)
    assert bench.kernel_class(_W2) == ("w2", False)
    assert bench.kernel_class(_W2.replace("EpiNone<1>", "EpiResidual<1>")) == ("w2", False)
    assert bench.kernel_class(_WIDE.replace("EpiSwiGLU<unsigned short>", "EpiResidual<0>")) == (
        "oproj", True)
    assert bench.kernel_class(_ATTN) == ("attn", False)
    assert bench.kernel_class("void hbsjd::k_attn_f16_seq<3>(unsigned short const*, int)") == (
        "attn", False)
    assert bench.kernel_class("hbsjd::k_attn_f16_qs(unsigned short const*, unsigned short*)") == (
        "attn", False)
    assert bench.kernel_class("hbsjd::k_transform(hbsjd::TransformArgs)") == ("transform", False)
    assert bench.kernel_class("hbsjd::k_transform_rows_setup(int)")[0] is None
    assert bench.kernel_class("__amd_rocclr_copyBuffer")[0] is None


def test_logical_launches_pair_wide_and_small_tile_dispatches():
    """A wide dispatch followed at once by the smaller-tile kernel of the same
    class is one launch; a small-tile dispatch alone (rows known on the host)
    or after another class is a launch of its own."""
    seq = [(1, _WIDE), (2, _SMALL), (3, _W2), (4, _SMALL), (5, _WIDE), (6, _ATTN),
           (7, _SMALL), (8, _WIDE), (9, "__amd_rocclr_copyBuffer"), (10, _SMALL)]
    groups = bench.logical_launches([{"id": i, "name": n} for i, n in reversed(seq)])
    got = [(c, [d["id"] for d in ds]) for c, ds in groups]
    assert got == [("w13", [1, 2]), ("w2", [3]), ("w13", [4]), ("w13", [5]), ("attn", [6]),
                   ("w13", [7]), ("w13", [8]), ("w13", [10])]


def _write_counters(path, rows):
    import csv
    import os
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_traffic_summary_scales_by_the_copy_and_sums_paired_dispatches(tmp_path):
    """Counters in KiB summed over instances and over the two dispatches of a
    paired launch, averaged over launches, divided by the copy's reading per
    byte: FETCH_SIZE reads half of a 1 GiB copy (factor 0.5), WRITE_SIZE all."""
    import json
    gib_kib = (1 << 30) / 1024
    _write_counters(tmp_path / "copy_FETCH_SIZE", [(7, "copy", "FETCH_SIZE", gib_kib / 4)] * 2)
    _write_counters(tmp_path / "copy_WRITE_SIZE", [(7, "copy", "WRITE_SIZE", gib_kib / 2)] * 2)
    # two w13 launches: (wide 100 + small 4) and (small 96) KiB fetched;
    # instance rows of one dispatch add up
    _write_counters(tmp_path / "bench_FETCH_SIZE",
                    [(1, _WIDE, "FETCH_SIZE", 60), (1, _WIDE, "FETCH_SIZE", 40),
                     (2, _SMALL, "FETCH_SIZE", 4), (3, _ATTN, "FETCH_SIZE", 10),
                     (4, _SMALL, "FETCH_SIZE", 96)])
    _write_counters(tmp_path / "bench_WRITE_SIZE",
                    [(1, _WIDE, "WRITE_SIZE", 30), (2, _SMALL, "WRITE_SIZE", 2),
                     (3, _ATTN, "WRITE_SIZE", 5), (4, _SMALL, "WRITE_SIZE", 32)])
    out = tmp_path / "traffic.json"
    out.write_text(json.dumps({"other": {"x": 1}}))
    assert bench.traffic_summary(str(tmp_path), "wl", str(out)) == 0
    rec = json.loads(out.read_text())
    assert rec["other"] == {"x": 1}
    w13 = rec["wl"]["w13"]
    assert w13["launches"] == 2 and w13["copy_fetch_factor"] == 0.5
    assert w13["fetch_kib_per_launch"] == 100.0 and w13["write_kib_per_launch"] == 32.0
    assert w13["hbm_bytes_per_launch"] == int(100 * 1024 / 0.5 + 32 * 1024)
    assert rec["wl"]["attn"]["hbm_bytes_per_launch"] == int(10 * 1024 / 0.5 + 5 * 1024)


def test_mfma_summary_normalises_grbm_by_the_xcds(tmp_path, capsys):
    """MfmaUtil divides the summed busy cycles by GRBM_GUI_ACTIVE / 8 (the
    cycles of the 8 XCDs summed) times the SIMDs: a kernel whose MFMA
    instructions kept every SIMD busy for a third of its cycles reads 1/3,
    the same as its flop rate against the peak at 2.4 GHz."""
    import csv
    cus, clk = 256, 2.4e9
    secs = 1e-3
    grbm = 8 * secs * clk                      # all XCDs' cycles
    busy = secs * clk * 4 * cus / 3            # a third of every SIMD's cycles
    mops = busy * 2                            # 16 busy cycles per 8192-MOP MFMA
    (tmp_path / "p").mkdir()
    (tmp_path / "t").mkdir()
    name = "hbsjd::k_mfma_probe(int, float*)"
    with open(tmp_path / "p" / "run_counter_collection.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for c, v in [("SQ_INSTS_VALU_MFMA_MOPS_F16", mops), ("SQ_VALU_MFMA_BUSY_CYCLES", busy),
                     ("GRBM_GUI_ACTIVE", grbm)]:
            w.writerow([1, name, c, v])
    with open(tmp_path / "t" / "run_kernel_trace.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writerow([name, 0, int(secs * 1e9)])
    assert bench.mfma_summary(str(tmp_path / "p"), str(tmp_path / "t"), cus=cus) == 0
    row = [ln for ln in capsys.readouterr().out.splitlines() if ln.startswith("mfma_probe")][0]
    frac, util = float(row.split()[-2]), float(row.split()[-1])
    assert abs(util - 1 / 3) < 1e-4
    assert abs(frac - (mops * 512 / secs) / 2.5e15) < 1e-4
