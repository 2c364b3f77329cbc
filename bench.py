"""Benchmark of the batched SJD rollout on one MI355X.

A step is one whole rollout (prefill, first window, then verification rounds
until every image holds T tokens). The headline workload is the LlamaGen-XL
shape with classifier-free guidance: 36 layers, d 1280, 20 heads, MLP 3456,
vocab 16384, 16x16 grid, batch 128 images run as 256 rows (conditional and
null class, logits combined at scale 2.0), prefixes uniform 0-128, W = 32,
H = 24, temperature 1.0, top-k 1000, bf16 weights. The LlamaGen-B shape
(12 layers, d 768, 12 heads, MLP 2048, batch 32, W = 16, top-k 2000, no
guidance), whose rounds are memory-bound, is measured in the same run under
"extra_workloads". Weights are seeded random-init and prefixes synthetic;
inputs are resident on the GPU before timing starts. Prints one JSON line.

Other modes:
  --peaks                 achievable copy and matmul rates (one JSON line)
  --copy-probe            one 1 GiB device-to-device copy, the calibration run
                          of the HBM byte counters
  --mfma-probe            the library's MFMA calibration kernel: sustained
                          rate, and the run the MFMA counters are read against
  --trace-summary DIR     per-class launch durations from the kernel trace CSV
                          that rocprofv3 --kernel-trace wrote under DIR
  --mfma-summary P T      MFMA counters per kernel class and tile (rocprofv3
                          --pmc CSVs under P) against the durations traced
                          under T by the same command
  --traffic-summary DIR   HBM bytes per launch and class from FETCH_SIZE and
                          WRITE_SIZE counter runs under DIR (copy_FETCH_SIZE,
                          copy_WRITE_SIZE, bench_FETCH_SIZE, bench_WRITE_SIZE),
                          merged into profiles/hbm_traffic.json
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import statistics
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "committed tokens/s per MI355X for batched SJD rollout; mean accepted tokens/round"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0     # dense fp16 / bf16 MFMA, the operand types of the matrix products
# classes launched once per layer are timed one launch in 4 (see the timed
# region below); once-per-forward classes every launch
PER_LAYER = ("qkv", "attn", "oproj", "w13", "w2", "norm")
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CSRC = os.path.join("paper_2608_18183_amd", "csrc")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------- algorithmic work

GEMMS = {  # class: (N, K, output bytes per output element)
    "qkv": lambda d, f, V, e: (3 * d, d, e),        # q, K, V in the operand type
    "oproj": lambda d, f, V, e: (d, d, 4),          # fp32 partial sums
    "w13": lambda d, f, V, e: (2 * f, d, e / 2),    # SwiGLU writes f of the 2f columns
    "w2": lambda d, f, V, e: (d, f, 4),
    "lmhead": lambda d, f, V, e: (V, d, 4),         # fp32 logits
}


def launch_work(cls, shape, rows, keys=0, ctx_keys=0, images=0, cfg=1, esz=2):
    """Work of ONE launch of a kernel class over `rows` rows (both guidance
    branches counted): (algorithmic bytes, activation bytes, flops).

    Algorithmic bytes are the launch's share of the rollout's memory roofline
    terms: the weights read once, the K and V rows appended to the cache (the
    QKV product) or read from it (attention: ctx_keys = keys of the cache read,
    summed over sequences), the logits written once (lm_head) and read once
    with one proposal row kept per image (the transform). Activation bytes are
    the rows handed between kernels (the inputs of a product, its other
    outputs, the residual stream through the norms), which a fused forward
    would not move; they are reported apart and not counted in the roofline.
    Flops: 2 per weight per row, attention 4 d per (row, key attended) with
    keys = keys attended summed over rows."""
    d, f, V = shape.d_model, shape.mlp_hidden, shape.vocab
    if cls in GEMMS:
        N, K, ob = GEMMS[cls](d, f, V, esz)
        alg = N * K * esz
        act = rows * K * esz + rows * N * ob
        if cls == "qkv":
            alg += rows * 2 * d * esz
            act -= rows * 2 * d * esz
        elif cls == "lmhead":
            alg += rows * N * ob
            act -= rows * N * ob
        return float(alg), float(act), 2.0 * rows * N * K
    if cls == "attn":
        return float(ctx_keys * 2 * d * esz), float(rows * 2 * d * esz), 4.0 * d * keys
    if cls == "transform":   # logits rows read; p rows of every position written
        return float(rows * V * 4 + images * V * 4), float(rows // cfg * V * 4), 0.0
    if cls == "norm":        # partial sums read, residual read and written, normed row written
        return 0.0, float(rows * d * (4.0 + 8.0 + esz)), 0.0
    return 0.0, 0.0, 0.0


def rollout_work(cls, shape, prefix_len, counts, W, cfg, esz=2):
    """(algorithmic bytes, activation bytes, flops, launches) of every launch of
    `cls` in one rollout, from the per-round commit counts (host array
    [rounds, B]); only active images count, so rows a Full round carries for
    finished images are not credited."""
    T, L = shape.T, shape.n_layers
    k = prefix_len.astype(np.int64)
    act = k < T
    ka = k[act]
    tot = [0.0, 0.0, 0.0, 0]

    def add(n_launch, rows, keys=0, ctx_keys=0, images=0):
        w = launch_work(cls, shape, rows, keys, ctx_keys, images, cfg, esz)
        for i in range(3):
            tot[i] += n_launch * w[i]
        tot[3] += n_launch

    # prefill: positions 0..k_b of each active image; each sequence's K and V
    # read once per layer; the lm_head on each sequence's last row
    pf_rows = int(np.sum(ka + 1)) * cfg
    n_seq = int(act.sum()) * cfg
    pf_keys = int(np.sum((ka + 1) * (ka + 2) // 2)) * cfg
    if cls in ("qkv", "oproj", "w13", "w2"):
        add(L, pf_rows)
    elif cls == "attn":
        add(L, pf_rows, pf_keys, pf_rows)
    elif cls == "norm":
        add(2 * L - 1, pf_rows)
        add(1, n_seq)
    elif cls == "lmhead":
        add(1, n_seq)
    elif cls == "transform":
        add(1, n_seq, images=int(act.sum()))
    cur = k.copy()
    for r in range(counts.shape[0]):
        a = cur < T
        A = int(a.sum())
        if A == 0:
            break
        rows = A * cfg * (W + 1)
        n = cur[a]
        keys = int(np.sum((W + 1) * (n + 1) + W * (W + 1) // 2)) * cfg
        ctx_keys = int(np.sum(n)) * cfg      # the committed cache of each sequence
        if cls in ("qkv", "oproj", "w13", "w2"):
            add(L, rows)
        elif cls == "attn":
            add(L, rows, keys, ctx_keys)
        elif cls == "norm":
            add(2 * L, rows)
        elif cls == "lmhead":
            add(1, rows)
        elif cls == "transform":
            add(1, rows, images=A)
        cur = cur + counts[r]
    return tuple(tot)


def path_work(shape, prefix_len, counts, W, cfg, esz=2):
    """Algorithmic (bytes, flops) of one whole rollout (prefill and every
    round), from the per-round commit counts (host array [rounds, B]); active
    images only. Per forward: the weights once; each sequence's committed K
    and V read once per layer and the new rows' K and V written; the logits
    written and read once and one probability row per image kept as the next
    round's proposal. Flops: 2 per weight per row (the lm_head on its rows
    only) plus 4 d per layer, row and key attended."""
    d, f, V, L, T = shape.d_model, shape.mlp_hidden, shape.vocab, shape.n_layers, shape.T
    layer_params = L * (4 * d * d + 3 * d * f)
    wbytes = (layer_params + d * V) * esz
    kv_row = L * 2 * d * esz            # K and V of one position, all layers
    k = prefix_len.astype(np.int64)
    act = k < T
    ka = k[act]
    n_img = int(act.sum())
    rows = int(np.sum(ka + 1)) * cfg
    keys = int(np.sum((ka + 1) * (ka + 2) // 2)) * cfg
    out_rows = n_img * cfg
    tot_b = wbytes + 2 * rows * kv_row + out_rows * V * 8 + n_img * V * 4
    tot_f = 2.0 * rows * layer_params + 2.0 * out_rows * d * V + 4.0 * d * L * keys
    cur = k.copy()
    for r in range(counts.shape[0]):
        a = cur < T
        A = int(a.sum())
        if A == 0:
            break
        n = cur[a]
        rows = A * cfg * (W + 1)
        keys = int(np.sum((W + 1) * (n + 1) + W * (W + 1) // 2)) * cfg
        tot_b += (wbytes + int(np.sum(n)) * cfg * kv_row + rows * kv_row + rows * V * 8
                  + A * V * 4)
        tot_f += 2.0 * rows * (layer_params + d * V) + 4.0 * d * L * keys
        cur = cur + counts[r]
    return tot_b, tot_f


# ---------------------------------------------------------------- rocprofv3 summaries

# kernel class of a dispatch: the GEMM classes by their epilogue type
_GEMM_EPI = (("EpiQkv", "qkv"), ("EpiSwiGLU", "w13"), ("EpiNone<0>", "oproj"),
             ("EpiNone<1>", "w2"), ("EpiResidual<0>", "oproj"), ("EpiResidual<1>", "w2"),
             ("EpiLogits", "lmhead"))
_KERNEL_CLASS = {"k_attn_f16": "attn", "k_attn_f16_seq": "attn", "k_attn_f16_qs": "attn",
                 "k_attn_f32": "attn",
                 "k_reduce_norm": "norm",
                 "k_rmsnorm": "norm", "k_embed_norm": "embed", "k_round_setup": "setup",
                 "k_transform": "transform", "k_verify": "verify", "k_bikl": "bikl",
                 "k_bikl_mean": "bikl"}
CLASS_SOURCE = {"qkv": "gemm.hip", "w13": "gemm.hip", "oproj": "gemm.hip", "w2": "gemm.hip",
                "lmhead": "gemm.hip", "attn": "attention.hip", "norm": "rowops.hip",
                "embed": "rowops.hip", "setup": "rowops.hip", "transform": "sampler.hip",
                "verify": "sampler.hip", "bikl": "sampler.hip"}


def kernel_class(name: str):
    """(class, is_wide_gemm) of a kernel name as rocprofv3 prints it."""
    m = re.search(r"\b(k_[A-Za-z0-9_]+)", name)
    if not m:
        return None, False
    fn = m.group(1)
    if fn.startswith("k_gemm_"):
        compact = name.replace(" ", "")
        for tag, cls in _GEMM_EPI:
            if tag in compact:
                return cls, fn == "k_gemm_wide"
        return None, False
    return _KERNEL_CLASS.get(fn), False


def logical_launches(dispatches):
    """Group dispatches (dicts with 'id', 'name' and a payload) in dispatch
    order into the library's launches: a matrix product whose rows are known
    only on the device goes out as the wide-tile kernel followed at once by the
    smaller-tile kernel of the same class, of which one does the work; the two
    count as one launch. Returns [(class, [dispatch, ...]), ...]."""
    out = []
    pending = None
    for d in sorted(dispatches, key=lambda x: x["id"]):
        cls, wide = kernel_class(d["name"])
        if cls is None:
            pending = None
            continue
        if (pending is not None and pending[0] == cls and not wide
                and d["id"] == pending[1][-1]["id"] + 1):
            pending[1].append(d)
            pending = None
            continue
        out.append((cls, [d]))
        pending = out[-1] if wide else None
    return out


def _find(dirpath, suffix):
    hits = sorted(glob.glob(os.path.join(dirpath, "**", "*" + suffix), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {dirpath}")
    return hits[0]


def trace_summary(dirpath, last=None):
    """Per-class launches and kernel time from a rocprofv3 kernel trace.
    last = {class: n}: also average that class over its last n launches (the
    timed rollouts, when nothing of that class launches after them)."""
    path = _find(dirpath, "kernel_trace.csv")
    disp = []
    for r in csv.DictReader(open(path)):
        disp.append({"id": int(r["Dispatch_Id"]), "name": r["Kernel_Name"],
                     "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
    groups = logical_launches(disp)
    per = {}
    for cls, ds in groups:
        per.setdefault(cls, []).append(sum(d["ns"] for d in ds))
    total = sum(sum(v) for v in per.values())
    print(f"kernel trace: {path}")
    print(f"{'class':10s} {'launches':>9s} {'total ms':>10s} {'share':>7s} {'avg us':>9s}")
    for cls, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        print(f"{cls:10s} {len(v):9d} {sum(v) / 1e6:10.3f} {sum(v) / total:7.3f} "
              f"{sum(v) / len(v) / 1e3:9.3f}")
    for cls, n in (last or {}).items():
        v = per.get(cls, [])[-n:]
        if v:
            print(f"last {len(v)} launches of {cls}: avg {sum(v) / len(v) / 1e3:.3f} us "
                  f"(sum of the kernel durations of each launch)")
    return 0


def _counter_per_dispatch(path):
    vals, names = {}, {}
    for r in csv.DictReader(open(path)):
        i = int(r["Dispatch_Id"])
        vals[i] = vals.get(i, 0.0) + float(r["Counter_Value"])
        names[i] = r["Kernel_Name"]
    return vals, names


def _source_hash(cls):
    files = [os.path.join(CSRC, CLASS_SOURCE[cls]), os.path.join(CSRC, "common.h"),
             os.path.join(CSRC, "launch.h")]
    return hashlib.sha256(b"".join(open(os.path.join(ROOT, f), "rb").read()
                                   for f in files)).hexdigest()


def traffic_summary(dirpath, workload, out_path=TRAFFIC_JSON):
    """HBM bytes per launch and class: each counter (KiB, summed over its
    instances) per dispatch, summed over a launch's dispatches, averaged over
    the class's launches and divided by what it reads per byte moved by the
    1 GiB copy (bytes read for FETCH_SIZE, written for WRITE_SIZE)."""
    fac = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        vals, _ = _counter_per_dispatch(_find(os.path.join(dirpath, f"copy_{c}"),
                                              "counter_collection.csv"))
        fac[c] = statistics.median(vals.values()) * 1024.0 / float(1 << 30)
    per = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        vals, names = _counter_per_dispatch(_find(os.path.join(dirpath, f"bench_{c}"),
                                                  "counter_collection.csv"))
        groups = logical_launches([{"id": i, "name": names[i], "v": v} for i, v in vals.items()])
        for cls, ds in groups:
            per.setdefault(cls, {}).setdefault(c, []).append(sum(d["v"] for d in ds))
    rec = {}
    print(f"copy factors: FETCH_SIZE {fac['FETCH_SIZE']:.5f}  WRITE_SIZE {fac['WRITE_SIZE']:.5f}")
    print(f"{'class':10s} {'launches':>9s} {'fetch KiB':>11s} {'write KiB':>11s} "
          f"{'HBM MB/launch':>14s}")
    for cls, v in sorted(per.items()):
        if "FETCH_SIZE" not in v or "WRITE_SIZE" not in v:
            continue
        f, w = statistics.mean(v["FETCH_SIZE"]), statistics.mean(v["WRITE_SIZE"])
        b = f * 1024 / fac["FETCH_SIZE"] + w * 1024 / fac["WRITE_SIZE"]
        rec[cls] = {"source": os.path.join(CSRC, CLASS_SOURCE[cls]),
                    "source_sha256": _source_hash(cls),
                    "launches": len(v["FETCH_SIZE"]), "fetch_kib_per_launch": round(f, 1),
                    "write_kib_per_launch": round(w, 1),
                    "copy_fetch_factor": round(fac["FETCH_SIZE"], 5),
                    "copy_write_factor": round(fac["WRITE_SIZE"], 5),
                    "hbm_bytes_per_launch": int(b)}
        print(f"{cls:10s} {len(v['FETCH_SIZE']):9d} {f:11.1f} {w:11.1f} {b / 1e6:14.3f}")
    try:
        allrec = json.load(open(out_path))
    except (OSError, ValueError):
        allrec = {}
    allrec[workload] = rec
    with open(out_path, "w") as fh:
        json.dump(allrec, fh, indent=1)
        fh.write("\n")
    print(f"wrote {out_path} [{workload}]")
    return 0


def _variant(name: str) -> str:
    if "k_gemm_wide" in name:
        return "wide"   # 256, 192 or 128 rows by 256 columns, chosen per launch
    m = re.search(r"k_gemm_f16<(\d+), (\d+)", name)
    return f"{m.group(1)}x{m.group(2)}" if m else "-"


def mfma_summary(pmc_dir, trace_dir, cus=256, xcds=8):
    """MFMA counters per kernel class and tile, against traced durations of
    the same command. Executed MFMA flops = SQ_INSTS_VALU_MFMA_MOPS_F16 x 512;
    MfmaUtil = sum of SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / xcds x
    4 x cus SIMDs), since GRBM_GUI_ACTIVE reads the cycles of all XCDs summed
    (what the calibration kernel, busy on every SIMD for its whole run, shows)."""
    vals, names = {}, {}
    for r in csv.DictReader(open(_find(pmc_dir, "counter_collection.csv"))):
        i = int(r["Dispatch_Id"])
        vals.setdefault(i, {}).setdefault(r["Counter_Name"], 0.0)
        vals[i][r["Counter_Name"]] += float(r["Counter_Value"])
        names[i] = r["Kernel_Name"]
    dur = {}
    for r in csv.DictReader(open(_find(trace_dir, "kernel_trace.csv"))):
        key = (r["Kernel_Name"], )
        dur.setdefault(key, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    rows = {}
    for i, v in vals.items():
        cls, _ = kernel_class(names[i])
        if cls is None:
            cls = "mfma_probe" if "k_mfma_probe" in names[i] else "other"
        key = (cls, _variant(names[i]), names[i])
        agg = rows.setdefault(key, {"n": 0})
        agg["n"] += 1
        for c, x in v.items():
            agg[c] = agg.get(c, 0.0) + x
    print(f"MFMA counters ({pmc_dir}) against traced durations ({trace_dir}); "
          f"MfmaUtil = busy / (GRBM_GUI_ACTIVE / {xcds} x {4 * cus} SIMDs)")
    print(f"{'class':11s} {'tile':8s} {'dispatches':>10s} {'avg us':>9s} {'GFLOP/disp':>11s} "
          f"{'TFLOP/s':>8s} {'of peak':>8s} {'MfmaUtil':>9s}")
    for (cls, var, name), a in sorted(rows.items()):
        ds = dur.get((name, ), [])
        if not ds or "SQ_INSTS_VALU_MFMA_MOPS_F16" not in a:
            continue
        n = a["n"]
        fl = a["SQ_INSTS_VALU_MFMA_MOPS_F16"] * 512.0 / n
        us = sum(ds) / len(ds) / 1e3
        util = a["SQ_VALU_MFMA_BUSY_CYCLES"] / (a["GRBM_GUI_ACTIVE"] / xcds * 4 * cus)
        tf = fl / us / 1e6
        print(f"{cls:11s} {var:8s} {n:10d} {us:9.2f} {fl / 1e9:11.3f} {tf:8.1f} "
              f"{tf / MFMA_PEAK_TFLOPS:8.4f} {util:9.4f}")
    return 0


def measured_traffic(workload, cls):
    """HBM bytes per launch of a kernel class on a workload from
    profiles/hbm_traffic.json, or None when there is none or the kernel's
    source (its file and the two shared headers) changed since the counters
    were taken."""
    try:
        rec = json.load(open(TRAFFIC_JSON))[workload][cls]
        if _source_hash(cls) != rec["source_sha256"]:
            return None
    except (OSError, KeyError, ValueError, TypeError):
        return None
    return rec["hbm_bytes_per_launch"]


# ---------------------------------------------------------------- host baseline

def host_info():
    """nproc (the CPUs this process may run on), os.cpu_count() and the CPU
    model that lscpu names."""
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    model = "unknown"
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    return nproc, os.cpu_count() or 1, model


def cpu_baseline(shape, blob_rounded, batch, wl, n_img, rounds, seed):
    """The oracle on the host: the first n_img images of the same batch (both
    guidance branches of each), prefill plus `rounds` verification rounds;
    committed tokens per second."""
    import oracle
    import synth
    om = oracle.Model(shape, blob_rounded)
    sub = synth.Batch(batch.prefix_tokens[:n_img].copy(), batch.prefix_len[:n_img].copy(),
                      batch.labels[:n_img].copy(), batch.temperature[:n_img].copy())
    t0 = time.perf_counter()
    r = om.rollout(sub, W=wl.window, H=wl.history, top_k=wl.top_k, cfg_scale=wl.cfg_scale,
                   seed=seed, exec_mode=1, max_rounds=rounds, allow_partial=True)
    dt = time.perf_counter() - t0
    committed = int(r["counts"].sum())
    return committed / dt, committed, dt


# ---------------------------------------------------------------- achievable peaks

def achievable_peaks() -> int:
    """What this GPU reaches outside the library, next to the datasheet peaks the
    roofline uses: a 1 GiB device-to-device copy (bytes read + written per
    second) and large bf16 matmuls through torch (hipBLASLt)."""
    import torch
    torch.cuda.set_device(0)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, reps):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / 1e3 / reps

    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    t_copy = timed(lambda: b.copy_(a), 20)
    copy_gbs = 2 * a.numel() * 4 / t_copy / 1e9
    del a, b
    n = 8192
    x = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    y = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    t_mm = timed(lambda: torch.matmul(x, y), 20)
    tflops = 2.0 * n ** 3 / t_mm / 1e12
    del x, y
    # the XL round's W1|W3 product (8448 rows, K 1280, N 6912), W stored [N][K]
    m, k, nn = 8448, 1280, 6912
    xa = torch.randn(m, k, device="cuda").to(torch.bfloat16)
    wt = torch.randn(nn, k, device="cuda").to(torch.bfloat16).t()
    t_xl = timed(lambda: torch.matmul(xa, wt), 20)
    xl_tflops = 2.0 * m * k * nn / t_xl / 1e12
    print(json.dumps({"achievable_peaks": {
        "xl_w13_matmul_tflops": round(xl_tflops, 1), "xl_w13_matmul_us": round(t_xl * 1e6, 1),
        "xl_w13_shape_mkn": [m, k, nn],
        "copy_gbs": round(copy_gbs, 1), "copy_frac_of_peak": round(copy_gbs / HBM_PEAK_GBS, 4),
        "copy_bytes": 2 * (1 << 30),
        "bf16_matmul_tflops": round(tflops, 1),
        "bf16_matmul_frac_of_peak": round(tflops / MFMA_PEAK_TFLOPS, 4),
        "matmul_shape": [n, n, n], "matmul": "torch.matmul (hipBLASLt)"}}))
    return 0


def mfma_probe(launches: int = 10) -> int:
    """The library's MFMA calibration kernel (one 256-thread workgroup per CU,
    back-to-back independent 16x16x32 fp16 MFMAs, no memory traffic): its
    sustained rate and the clock that rate implies at 4096 flops per CU per
    cycle (the dense fp16 peak of 2.5 PFLOP/s at 256 CUs and 2.4 GHz)."""
    import torch

    import paper_2608_18183_amd as P
    torch.cuda.set_device(0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    iters = 32768
    sink = torch.zeros(256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    flops = cus * 4 * iters * 8 * 16384.0
    P.hbsjd_mfma_probe(cus, iters, sink, stream)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(launches):
        P.hbsjd_mfma_probe(cus, iters, sink, stream)
    ev[1].record(stream)
    torch.cuda.synchronize()
    us = ev[0].elapsed_time(ev[1]) * 1e3 / launches
    tf = flops / us / 1e6
    print(json.dumps({"mfma_probe": {
        "workgroups": cus, "wavefronts": 4 * cus, "iters": iters, "launches": launches,
        "flops_per_launch": flops, "avg_launch_us": round(us, 2),
        "tflops": round(tf, 1), "frac_of_peak": round(tf / MFMA_PEAK_TFLOPS, 4),
        "implied_clock_ghz": round(tf * 1e12 / (cus * 4096.0) / 1e9, 3)}}), flush=True)
    return 0


def copy_probe() -> int:
    """One 1 GiB device-to-device copy after a fill: the run whose FETCH_SIZE
    and WRITE_SIZE readings give the counters' bytes per byte moved."""
    import torch
    torch.cuda.set_device(0)
    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print("copied 1 GiB three times", flush=True)
    return 0


# ---------------------------------------------------------------- one workload

def measure(P, torch, name, args, ar_steps, abl_steps, score_steps):
    """Time `args.steps` rollouts of a workload (after `args.warmup` untimed
    ones) and the optional baselines beside it. Returns (record, state) where
    state holds what the host baseline needs."""
    import synth
    wl = synth.WORKLOADS[name]
    shape = wl.model
    T = shape.T
    t0 = time.perf_counter()
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    batch = synth.make_batch(wl, 1)
    B = wl.batch
    cfg = 2 if wl.cfg_scale else 1
    esz = 2 if wl.dtype == "bf16" else 4
    desc = P.ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.mlp_hidden,
                       shape.vocab, shape.n_classes, shape.grid,
                       P.DTYPE_BF16 if wl.dtype == "bf16" else P.DTYPE_F32,
                       bool(shape.has_lm_bias), shape.rms_eps, shape.rope_base)
    ctx = P.Context(desc)
    ctx.hbsjd_load_weights(blob)
    log(f"{name}: weights generated and loaded ({time.perf_counter() - t0:.1f} s)")
    prefix = torch.from_numpy(batch.prefix_tokens).cuda()
    max_rounds = int(T - batch.prefix_len.min())
    out_tokens = torch.empty((B, T), dtype=torch.int32, device="cuda")
    out_counts = torch.empty((max_rounds, B), dtype=torch.int32, device="cuda")
    mode = {"auto": P.EXEC_AUTO, "full": P.EXEC_FULL, "compact": P.EXEC_COMPACT}[args.exec_mode]
    # the Full/Compact threshold from the library's latency test (Sec. 4.3),
    # unless one is given; rollouts below pass gamma = -1 to use the context's
    gamma = args.gamma if args.gamma >= 0 else ctx.hbsjd_calibrate_gamma(B, wl.window)

    def step(seed, counts=out_counts):
        return ctx.hbsjd_rollout(prefix, batch.prefix_len, batch.labels, batch.temperature,
                                 wl.window, history=wl.history, top_k=wl.top_k,
                                 cfg_scale=wl.cfg_scale, seed=seed, exec_mode=mode,
                                 gamma=args.gamma, max_rounds=max_rounds, out_tokens=out_tokens,
                                 out_counts=counts)

    # warm-up; the first warm-up rollout also times every kernel class to find
    # the dominant one
    dominant = None
    for i in range(max(args.warmup, 1)):
        if i == 0:
            ctx.hbsjd_profile_start(P.KERNELS)
        step(999 - i)
        if i == 0:
            prof = ctx.hbsjd_profile_read()
            ctx.hbsjd_profile_start(())
            dominant = max(prof, key=lambda k: prof[k][0])
    torch.cuda.synchronize()
    log(f"{name}: gamma {gamma}, warm-up done, dominant kernel class {dominant}")
    # timed region: only the dominant class is bracketed by events. Each timed
    # rollout writes its own commit counts (allocated here, outside the timed
    # region): the roofline's algorithmic work is computed from them after the
    # baseline and ablation runs have reused the shared buffers.
    timed_counts = [torch.empty_like(out_counts) for _ in range(args.steps)]
    # A per-layer class has one launch in 4 bracketed: each bracketed launch
    # costs a few microseconds of queue time outside the kernel, which
    # bracketing all of them would add to the throughput being measured.
    timed_every = 4 if dominant in PER_LAYER else 1
    ctx.hbsjd_profile_sample(timed_every)
    ctx.hbsjd_profile_start([dominant])
    results = []
    step_s = []   # each rollout call is blocking, so the host clock brackets it
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ts = time.perf_counter()
        results.append(step(1000 + i, timed_counts[i]))
        step_s.append(time.perf_counter() - ts)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_ms, dom_n = ctx.hbsjd_profile_read()[dominant]
    ctx.hbsjd_profile_start(())
    ctx.hbsjd_profile_sample(1)
    committed_per_step = int(np.sum(T - batch.prefix_len))
    value = committed_per_step * args.steps / elapsed
    log(f"{name}: {args.steps} timed rollouts, {1000 * elapsed / args.steps:.1f} ms each")

    # the cached-AR baseline on the same batch (one row per image per round),
    # timed after the SJD region with the same clock
    ar = None
    if ar_steps > 0:
        def ar_step(seed):
            return ctx.hbsjd_rollout(prefix, batch.prefix_len, batch.labels, batch.temperature,
                                     1, top_k=wl.top_k, cfg_scale=wl.cfg_scale, seed=seed,
                                     verify_mode=P.VERIFY_AR, max_rounds=max_rounds,
                                     out_tokens=out_tokens, out_counts=out_counts)
        ar_step(998)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for i in range(ar_steps):
            ar_step(1000 + i)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t1) / ar_steps
        ar = {"ms_per_step": round(1000.0 * dt, 3), "steps": ar_steps,
              "value": round(committed_per_step / dt, 1), "unit": "tokens/s",
              "speedup_of_sjd": round(value * dt / committed_per_step, 3)}
        log(f"{name}: cached AR {1000 * dt:.1f} ms per rollout")

    # execution ablations on the same batch (Sec. 5: Table 2 compares cached
    # AR, Batch-Synchronous SJD and independent progress with Full execution;
    # Tables 3 and 8 and Fig. 2c compare Full, Compact and the hybrid switch
    # over gamma). Each is timed after one untimed rollout of its own setting.
    ablations = None
    if abl_steps > 0:
        def abl(exec_mode, g, progress):
            def run(seed):
                return ctx.hbsjd_rollout(prefix, batch.prefix_len, batch.labels,
                                         batch.temperature, wl.window, history=wl.history,
                                         top_k=wl.top_k, cfg_scale=wl.cfg_scale, seed=seed,
                                         exec_mode=exec_mode, gamma=g, max_rounds=max_rounds,
                                         out_tokens=out_tokens, out_counts=out_counts,
                                         progress=progress)
            run(997)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            rs = [run(1000 + i) for i in range(abl_steps)]
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t2) / abl_steps
            ir = sum(r["image_rounds"] for r in rs)
            full_rounds = sum(int(np.sum(r["mode"] == 0)) for r in rs)
            return {"ms_per_step": round(1000.0 * dt, 3),
                    "value": round(committed_per_step / dt, 1),
                    "rounds": [r["rounds"] for r in rs],
                    "full_rounds": full_rounds,
                    "mean_accepted_tokens_per_round":
                        round(sum(r["verified"] for r in rs) / max(ir, 1), 4)}
        ind = P.PROGRESS_INDEPENDENT
        ablations = {
            "independent_full": abl(P.EXEC_FULL, 0, ind),
            "independent_compact": abl(P.EXEC_COMPACT, 0, ind),
            "batch_synchronous_full": abl(P.EXEC_FULL, 0, P.PROGRESS_SYNC),
            "batch_synchronous_compact": abl(P.EXEC_COMPACT, 0, P.PROGRESS_SYNC),
            "gamma_sweep": {str(g): abl(P.EXEC_AUTO, g, ind)
                            for g in sorted({0, B // 8, B // 4, B // 2, B})},
        }
        if ar is not None:
            for k in ("independent_full", "independent_compact", "batch_synchronous_full",
                      "batch_synchronous_compact"):
                ablations[k]["speedup_vs_cached_ar"] = round(
                    ar["ms_per_step"] / ablations[k]["ms_per_step"], 3)
        log(f"{name}: ablations done")

    # teacher scoring of the completed sequences (Sec. 3.1, Eq. 3): student and
    # an L-architecture teacher forward, then the per-position biKL kernel,
    # whose launches are timed with HIP events on the library's stream
    scoring = None
    if score_steps > 0:
        tshape = synth.teacher_shape(shape)
        teacher = P.Context(P.ModelDesc(tshape.n_layers, tshape.d_model, tshape.n_heads,
                                        tshape.mlp_hidden, tshape.vocab, tshape.n_classes,
                                        tshape.grid, desc.dtype, False, tshape.rms_eps,
                                        tshape.rope_base))
        teacher.hbsjd_load_weights(synth.make_weights(tshape, 5))
        seqs = out_tokens.clone()
        ctx.hbsjd_score_bikl(teacher, seqs, batch.prefix_len, batch.labels)
        torch.cuda.synchronize()
        ctx.hbsjd_profile_start(["bikl"])
        t3 = time.perf_counter()
        for _ in range(score_steps):
            _, loss = ctx.hbsjd_score_bikl(teacher, seqs, batch.prefix_len, batch.labels)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t3) / score_steps
        bms, bn = ctx.hbsjd_profile_read()["bikl"]
        ctx.hbsjd_profile_start(())
        avg_s = bms / 1e3 / max(bn, 1)
        # algorithmic bytes per launch: both fp32 logits rows read once and
        # one fp32 written per scored position
        kb = committed_per_step * (2 * shape.vocab * 4 + 4)
        scoring = {
            "teacher": f"{tshape.n_layers}L d{tshape.d_model} h{tshape.n_heads} "
                       f"f{tshape.mlp_hidden} (LlamaGen-L architecture) on the same grid, "
                       f"random-init",
            "ms_per_batch": round(1000.0 * dt, 3),
            "scored_positions": committed_per_step,
            "value": round(committed_per_step / dt, 1),
            "unit": "scored positions/s",
            "mean_loss": round(float(loss.mean()), 6),
            "bikl_roofline": {"bound": "hbm", "achieved": round(kb / avg_s / 1e9, 2),
                              "peak": HBM_PEAK_GBS, "unit": "GB/s",
                              "frac": round(kb / avg_s / 1e9 / HBM_PEAK_GBS, 5),
                              "avg_launch_us": round(avg_s * 1e6, 3), "launches": bn,
                              "bytes_per_launch": kb},
        }
        del teacher
        log(f"{name}: teacher scoring done")

    counts_total = sum(int(r["verified"]) for r in results)    # committed tokens = sum of counts
    image_rounds = sum(r["image_rounds"] for r in results)
    mean_accepted = counts_total / max(image_rounds, 1)
    reject_rate = sum(r["rejected"] for r in results) / max(counts_total, 1)

    # roofline of the dominant kernel class over the timed region: the
    # algorithmic work of all its launches over their summed duration, which
    # the bracketed launches (one in timed_every) sample
    alg = actb = fl = 0.0
    launches = 0
    for r in results:
        w = rollout_work(dominant, shape, batch.prefix_len, r["counts"].cpu().numpy(),
                         wl.window, cfg, esz=esz)
        alg, actb, fl, launches = alg + w[0], actb + w[1], fl + w[2], launches + w[3]
    avg_s = dom_ms / 1e3 / max(dom_n, 1)     # mean duration of a bracketed launch
    t_s = avg_s * launches
    if fl / (MFMA_PEAK_TFLOPS * 1e12) > alg / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(fl / t_s / 1e12, 3), "peak": MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(alg / t_s / 1e9, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 5)
    traffic = measured_traffic(name, dominant)
    roof["traffic"] = traffic
    roof["kernel"] = dominant
    roof["launches"] = launches
    roof["timed_launches"] = dom_n
    roof["timed_every"] = timed_every
    roof["avg_launch_us"] = round(1e6 * avg_s, 3)
    roof["flops_per_launch"] = round(fl / max(launches, 1))
    roof["bytes_per_launch"] = round(alg / max(launches, 1))
    roof["activation_bytes_per_launch"] = round(actb / max(launches, 1))
    roof["activation_gbs"] = round(actb / t_s / 1e9, 2)
    roof["time_share"] = round(t_s / elapsed, 4)
    # the whole path over the timed rollouts (prefill and rounds)
    pb = pf = 0.0
    for r in results:
        b, f_ = path_work(shape, batch.prefix_len, r["counts"].cpu().numpy(), wl.window, cfg,
                          esz=esz)
        pb += b
        pf += f_
    path = {"bytes_per_step": round(pb / len(results)), "flops_per_step": round(pf / len(results)),
            "achieved_gbs": round(pb / elapsed / 1e9, 2),
            "frac_hbm": round(pb / elapsed / 1e9 / HBM_PEAK_GBS, 5),
            "achieved_tflops": round(pf / elapsed / 1e12, 3),
            "frac_mfma": round(pf / elapsed / 1e12 / MFMA_PEAK_TFLOPS, 5),
            "bound": "hbm" if pb / (HBM_PEAK_GBS * 1e9) >= pf / (MFMA_PEAK_TFLOPS * 1e12)
            else "mfma"}

    rec = {
        "workload": f"{name}: {shape.n_layers}L d{shape.d_model} h{shape.n_heads} "
                    f"f{shape.mlp_hidden} V{shape.vocab} {shape.grid}x{shape.grid}, batch {B}"
                    f"{f' ({B * cfg} rows with guidance)' if cfg == 2 else ''}, W {wl.window}, "
                    f"H {wl.history}, top-k {wl.top_k}, cfg {wl.cfg_scale}",
        "value": round(value, 1),
        "unit": "tokens/s",
        "ms_per_step": round(1000.0 * elapsed / args.steps, 3),
        "batch": B, "window": wl.window, "history": wl.history,
        "gamma": gamma, "gamma_source": "given" if args.gamma >= 0 else "calibrated",
        "mean_accepted_tokens_per_round": round(mean_accepted, 4),
        "rounds_per_step": [r["rounds"] for r in results],
        "step_ms": {"per_seed": [round(1000.0 * x, 3) for x in step_s],
                    "mean": round(1000.0 * float(np.mean(step_s)), 3),
                    "median": round(1000.0 * float(np.median(step_s)), 3),
                    "p95": round(1000.0 * float(np.percentile(step_s, 95)), 3)},
        "active_per_round": [int(x) for x in results[0]["active"]],
        "mode_per_round": "".join("F" if int(x) == 0 else "C" for x in results[0]["mode"]),
        "reject_rate": round(reject_rate, 4),
        "committed_tokens_per_step": committed_per_step,
        "roofline": roof,
        "path_roofline": path,
        "cached_ar": ar,
        "ablations": ablations,
        "teacher_scoring": scoring,
    }
    del ctx
    torch.cuda.empty_cache()
    state = {"wl": wl, "shape": shape, "blob": blob, "batch": batch}
    return rec, state


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llamagen_xl_cfg")
    ap.add_argument("--extra-workload", default="llamagen_b",
                    help="a second workload measured in the same run ('none' = skip)")
    ap.add_argument("--exec-mode", default="auto", choices=["auto", "full", "compact"])
    ap.add_argument("--gamma", type=int, default=-1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=0,
                    help="images in the host sample (0 = one sequence per OpenMP thread)")
    ap.add_argument("--cpu-rounds", type=int, default=3,
                    help="verification rounds after the prefill in the host sample")
    ap.add_argument("--ar-steps", type=int, default=1,
                    help="timed cached-AR rollouts of the headline workload (0 = skip)")
    ap.add_argument("--ablation-steps", type=int, default=0,
                    help="timed rollouts per execution ablation of the headline workload: "
                         "Full, Compact, a gamma sweep and Batch-Synchronous SJD (0 = skip)")
    ap.add_argument("--score-steps", type=int, default=0,
                    help="timed teacher-scoring calls (Eq. 3) on the headline workload")
    ap.add_argument("--extra-ar-steps", type=int, default=2)
    ap.add_argument("--extra-ablation-steps", type=int, default=1)
    ap.add_argument("--extra-score-steps", type=int, default=2)
    ap.add_argument("--peaks", action="store_true",
                    help="measure achievable peaks instead (a 1 GiB device copy and "
                         "bf16 torch.matmul) and print them as one JSON line")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--mfma-probe", action="store_true",
                    help="time the MFMA calibration kernel and print its rate as one JSON line")
    ap.add_argument("--trace-summary", metavar="DIR")
    ap.add_argument("--last", action="append", default=[], metavar="CLASS=N",
                    help="with --trace-summary: average CLASS over its last N launches")
    ap.add_argument("--traffic-summary", metavar="DIR")
    ap.add_argument("--mfma-summary", nargs=2, metavar=("PMC_DIR", "TRACE_DIR"),
                    help="MFMA counters (SQ_INSTS_VALU_MFMA_MOPS_F16, SQ_VALU_MFMA_BUSY_CYCLES, "
                         "GRBM_GUI_ACTIVE) per class and tile against traced durations")
    args = ap.parse_args()
    if args.trace_summary:
        return trace_summary(args.trace_summary,
                             {c: int(n) for c, n in (x.split("=") for x in args.last)})
    if args.traffic_summary:
        return traffic_summary(args.traffic_summary, args.workload)
    if args.mfma_summary:
        return mfma_summary(*args.mfma_summary)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the rollout "
              f"shards by image with no cross-GPU exchange, so each GPU would run its own "
              f"images as an independent single-GPU rollout", file=sys.stderr)
        return 2
    if args.peaks:
        return achievable_peaks()
    if args.copy_probe:
        return copy_probe()
    if args.mfma_probe:
        return mfma_probe()

    import torch

    import paper_2608_18183_amd as P
    import synth

    torch.cuda.set_device(0)
    head, st = measure(P, torch, args.workload, args, args.ar_steps, args.ablation_steps,
                       args.score_steps)
    extra = {}
    if args.extra_workload != "none" and args.extra_workload != args.workload:
        rec, _ = measure(P, torch, args.extra_workload, args, args.extra_ar_steps,
                         args.extra_ablation_steps, args.extra_score_steps)
        extra[args.extra_workload] = rec

    cpu = None
    if not args.no_cpu_baseline:
        wl, shape = st["wl"], st["shape"]
        cfg = 2 if wl.cfg_scale else 1
        threads = int(os.environ.get("OMP_NUM_THREADS") or 0) or (os.cpu_count() or 1)
        n_img = args.cpu_images or min(wl.batch, max(1, math.ceil(threads / cfg)))
        nproc, ncpu, model = host_info()
        rb = synth.bf16_rounded_blob(shape, st["blob"]) if wl.dtype == "bf16" else st["blob"]
        st["blob"] = None
        log(f"host baseline: oracle on {n_img} images, prefill + {args.cpu_rounds} rounds, "
            f"{threads} threads")
        v, committed, dt = cpu_baseline(shape, rb, st["batch"], wl, n_img, args.cpu_rounds,
                                        seed=1000)
        cpu = {"value": round(v, 4), "unit": "tokens/s", "cores": min(threads, n_img * cfg),
               "kind": "oracle",
               "sample": f"{args.workload}: the first {n_img} images of the same batch "
                         f"({n_img * cfg} sequences with guidance), prefill + "
                         f"{args.cpu_rounds} rounds, seed 1000: {committed} committed tokens "
                         f"in {dt:.1f} s; fp32 oracle on the bf16-rounded weights, one "
                         f"sequence per OpenMP thread",
               "omp_threads": threads, "nproc": nproc, "os_cpu_count": ncpu,
               "cpu_model": model}
        log(f"host baseline: {committed} tokens in {dt:.1f} s")

    wl = st["wl"]
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights, uniform random prefixes)",
        "config": {"workload": head["workload"],
                   "batch": head["batch"], "window": head["window"], "history": head["history"],
                   "exec_mode": args.exec_mode, "gamma": head["gamma"],
                   "gamma_source": head["gamma_source"],
                   "weights": "bf16-rounded N(0, 0.02), held as fp16 x 2^e per matrix; "
                              "fp16 MFMA operands, fp32 accumulation, residual stream and "
                              "sampling" if wl.dtype == "bf16" else "fp32",
                   "parallelism": "single GPU"},
    }
    for k in ("mean_accepted_tokens_per_round", "rounds_per_step", "step_ms", "active_per_round",
              "mode_per_round", "reject_rate", "committed_tokens_per_step", "roofline",
              "path_roofline", "cached_ar", "ablations", "teacher_scoring"):
        line[k] = head[k]
    line["cpu_baseline"] = cpu
    line["extra_workloads"] = extra
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
