"""Benchmark of the batched SJD rollout on one MI355X.

A step is one whole rollout (prefill, first window, then verification rounds
until every image holds T tokens) of the LlamaGen-B-shaped workload: 12 layers,
d 768, 12 heads, MLP 2048, vocab 16384, 16x16 grid, batch 32 with prefixes of
uniform length 0-128, W = 16, H = 24, temperature 1.0, top-k 2000, bf16,
seeded random-init weights and synthetic prefixes. Inputs are resident on the
GPU before timing starts. Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "committed tokens/s per MI355X for batched SJD rollout; mean accepted tokens/round"
HBM_PEAK_GBS = 8000.0
# classes launched once per layer are timed one launch in 4 (see the timed
# region below); once-per-forward classes every launch
PER_LAYER = ("qkv", "attn", "oproj", "w13", "w2", "norm")
BF16_PEAK_TFLOPS = 2500.0


GEMMS = {  # class: (N, K, output bytes per output column and row)
    "qkv": lambda d, f, V, e: (3 * d, d, e),        # q, K, V written in the compute dtype
    "oproj": lambda d, f, V, e: (d, d, 4),          # fp32 partial sums written
    "w13": lambda d, f, V, e: (2 * f, d, e / 2),    # SwiGLU writes f of the 2f columns
    "w2": lambda d, f, V, e: (d, f, 4),
    "lmhead": lambda d, f, V, e: (V, d, 4),         # fp32 logits
}


def launch_work(cls, shape, rows, keys=0, seq_keys=0, esz=2):
    """Algorithmic (bytes, flops) of ONE launch of a kernel class over `rows`
    rows of active images. GEMMs read the weights once and the activations once;
    attention reads each sequence's K and V once (seq_keys = sum over sequences
    of keys read) and does 4 d flops per (row, key) pair (keys = sum over rows of
    keys attended); the transform reads a logits row and writes a probability row."""
    d, f, V = shape.d_model, shape.mlp_hidden, shape.vocab
    if cls in GEMMS:
        N, K, ob = GEMMS[cls](d, f, V, esz)
        return N * K * esz + rows * K * esz + rows * N * ob, 2.0 * rows * N * K
    if cls == "attn":
        return seq_keys * 2 * d * esz + rows * 2 * d * esz, 4.0 * d * keys
    if cls == "transform":
        return rows * V * 8.0, 0.0
    if cls == "norm":     # partial sums read, residual read and written, normed row written
        return rows * d * (4.0 + 8.0 + esz), 0.0
    return 0.0, 0.0


def rollout_work(cls, shape, prefix_len, counts, W, cfg, esz=2):
    """Algorithmic (bytes, flops) of every launch of `cls` in one rollout, from the
    per-round commit counts (host array [rounds, B]); only active images count."""
    T, L = shape.T, shape.n_layers
    k = prefix_len.astype(np.int64)
    act = k < T
    ka = k[act]
    tot_b = tot_f = 0.0

    def add(n_launch, rows, keys=0, seq_keys=0):
        nonlocal tot_b, tot_f
        b, fl = launch_work(cls, shape, rows, keys, seq_keys, esz)
        tot_b += n_launch * b
        tot_f += n_launch * fl

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
        add(1, int(act.sum()))
    cur = k.copy()
    for r in range(counts.shape[0]):
        a = cur < T
        A = int(a.sum())
        if A == 0:
            break
        rows = A * cfg * (W + 1)
        n = cur[a]
        keys = int(np.sum((W + 1) * (n + 1) + W * (W + 1) // 2)) * cfg
        seq_keys = int(np.sum(n + W + 1)) * cfg
        if cls in ("qkv", "oproj", "w13", "w2"):
            add(L, rows)
        elif cls == "attn":
            add(L, rows, keys, seq_keys)
        elif cls == "norm":
            add(2 * L, rows)
        elif cls == "lmhead":
            add(1, rows)
        elif cls == "transform":
            add(1, A * (W + 1))
        cur = cur + counts[r]
    return tot_b, tot_f


def path_work(shape, prefix_len, counts, W, cfg, esz=2):
    """Algorithmic (bytes, flops) of one whole rollout (prefill and every
    round), from the per-round commit counts (host array [rounds, B]); active
    images only. Per forward: the weights once; each sequence's KV read once
    per layer and the new rows' KV written; the logits written and read once
    and one probability row per image kept as the next round's proposal.
    Flops: 2 per weight per row (the lm_head on its rows only) plus 4 d per
    layer, row and key attended."""
    d, f, V, L, T = shape.d_model, shape.mlp_hidden, shape.vocab, shape.n_layers, shape.T
    layer_params = L * (4 * d * d + 3 * d * f)
    wbytes = (layer_params + d * V) * esz
    kv_row = L * 2 * d * esz            # K and V of one position, all layers
    k = prefix_len.astype(np.int64)
    act = k < T
    ka = k[act]
    n_img = int(act.sum())
    # prefill: positions 0..k_b of each active image (both CFG branches); the
    # lm_head runs on each sequence's last row
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


def measured_traffic(cls):
    """HBM bytes per launch of a kernel class from the committed counter
    summary (profiles/hbm_traffic.json: FETCH_SIZE and WRITE_SIZE passes scaled
    by a copy of known size), or None when there is none or the kernel's
    source (its file and the two shared headers) changed since the counters
    were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    csrc = os.path.join(ROOT, "paper_2608_18183_amd", "csrc")
    try:
        rec = json.load(open(path))[cls]
        src = b"".join(open(f, "rb").read() for f in
                       [os.path.join(ROOT, rec["source"]), os.path.join(csrc, "common.h"),
                        os.path.join(csrc, "launch.h")])
    except (OSError, KeyError, ValueError):
        return None
    if hashlib.sha256(src).hexdigest() != rec["source_sha256"]:
        return None
    return rec["hbm_bytes_per_launch"]


def cpu_baseline(shape, blob_rounded, batch, wl, n_img, rounds):
    """The oracle on the host: the first n_img images of the same batch, prefill
    plus `rounds` verification rounds; committed tokens per second."""
    import oracle
    import synth
    om = oracle.Model(shape, blob_rounded)
    sub = synth.Batch(batch.prefix_tokens[:n_img].copy(), batch.prefix_len[:n_img].copy(),
                      batch.labels[:n_img].copy(), batch.temperature[:n_img].copy())
    t0 = time.perf_counter()
    r = om.rollout(sub, W=wl.window, H=wl.history, top_k=wl.top_k, cfg_scale=wl.cfg_scale,
                   seed=1000, exec_mode=1, max_rounds=rounds, allow_partial=True)
    dt = time.perf_counter() - t0
    committed = int(r["counts"].sum())
    return committed / dt, committed, dt


def achievable_peaks() -> int:
    """What this GPU reaches outside the library, next to the datasheet peaks the
    roofline uses: a 1 GiB device-to-device copy (bytes read + written per
    second) and a large bf16 matmul through torch (hipBLASLt)."""
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
        "bf16_matmul_frac_of_peak": round(tflops / BF16_PEAK_TFLOPS, 4),
        "matmul_shape": [n, n, n], "matmul": "torch.matmul (hipBLASLt)"}}))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llamagen_b")
    ap.add_argument("--exec-mode", default="auto", choices=["auto", "full", "compact"])
    ap.add_argument("--gamma", type=int, default=-1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=0, help="images in the CPU sample (0 = auto)")
    ap.add_argument("--ar-steps", type=int, default=2,
                    help="timed rollouts of the cached-AR baseline after the SJD ones (0 = skip)")
    ap.add_argument("--score-steps", type=int, default=2,
                    help="timed teacher-scoring calls (Eq. 3) on the completed rollout (0 = skip)")
    ap.add_argument("--ablation-steps", type=int, default=1,
                    help="timed rollouts per execution ablation: Full, Compact, a gamma sweep "
                         "and Batch-Synchronous SJD (0 = skip)")
    ap.add_argument("--peaks", action="store_true",
                    help="measure achievable peaks instead (a 1 GiB device copy and a "
                         "8192^3 bf16 torch.matmul) and print them as one JSON line")
    args = ap.parse_args()
    if args.peaks:
        return achievable_peaks()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the rollout "
              f"shards by image with no cross-GPU exchange, so each GPU would run its own "
              f"images as an independent single-GPU rollout", file=sys.stderr)
        return 2

    import torch

    import paper_2608_18183_amd as P
    import synth

    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.workload]
    shape = wl.model
    T = shape.T
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    batch = synth.make_batch(wl, 1)
    B = wl.batch
    cfg = 2 if wl.cfg_scale else 1
    desc = P.ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.mlp_hidden,
                       shape.vocab, shape.n_classes, shape.grid,
                       P.DTYPE_BF16 if wl.dtype == "bf16" else P.DTYPE_F32,
                       bool(shape.has_lm_bias), shape.rms_eps, shape.rope_base)
    ctx = P.Context(desc)
    ctx.hbsjd_load_weights(blob)
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
    # timed region: only the dominant class is bracketed by events. Each timed
    # rollout writes its own commit counts (allocated here, outside the timed
    # region): the roofline's algorithmic work is computed from them after the
    # baseline and ablation runs have reused the shared buffers.
    timed_counts = [torch.empty_like(out_counts) for _ in range(args.steps)]
    # A per-layer class has one launch in 4 bracketed (layers 0, 4 and 8 of
    # each 12-layer forward): each bracketed launch costs a few microseconds
    # of queue time outside the kernel, which bracketing all of them would add
    # to the throughput being measured.
    timed_every = 4 if dominant in PER_LAYER else 1
    ctx.hbsjd_profile_sample(timed_every)
    ctx.hbsjd_profile_start([dominant])
    results = []
    step_s = []   # each rollout call is blocking, so the host clock brackets it
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

    # the cached-AR baseline on the same batch (one row per image per round),
    # timed after the SJD region with the same clock
    ar = None
    if args.ar_steps > 0:
        def ar_step(seed):
            return ctx.hbsjd_rollout(prefix, batch.prefix_len, batch.labels, batch.temperature,
                                     1, top_k=wl.top_k, cfg_scale=wl.cfg_scale, seed=seed,
                                     verify_mode=P.VERIFY_AR, max_rounds=max_rounds,
                                     out_tokens=out_tokens, out_counts=out_counts)
        ar_step(998)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for i in range(args.ar_steps):
            ar_step(1000 + i)
        torch.cuda.synchronize()
        ar_elapsed = time.perf_counter() - t1
        ar = {"ms_per_step": round(1000.0 * ar_elapsed / args.ar_steps, 3),
              "steps": args.ar_steps}

    committed_per_step = int(np.sum(T - batch.prefix_len))

    # execution ablations on the same batch (Sec. 5: Table 2 compares cached
    # AR, Batch-Synchronous SJD and independent progress with Full execution;
    # Tables 3 and 8 and Fig. 2c compare Full, Compact and the hybrid switch
    # over gamma). Each is timed after one untimed rollout of its own setting.
    ablations = None
    if args.ablation_steps > 0:
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
            rs = [run(1000 + i) for i in range(args.ablation_steps)]
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t2) / args.ablation_steps
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

    # teacher scoring of the completed sequences (Sec. 3.1, Eq. 3): student and
    # an L-architecture teacher forward, then the per-position biKL kernel,
    # whose launches are timed with HIP events on the library's stream
    scoring = None
    if args.score_steps > 0:
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
        for _ in range(args.score_steps):
            _, loss = ctx.hbsjd_score_bikl(teacher, seqs, batch.prefix_len, batch.labels)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t3) / args.score_steps
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

    value = committed_per_step * args.steps / elapsed
    counts_total = sum(int(r["verified"]) for r in results)    # committed tokens = sum of counts
    image_rounds = sum(r["image_rounds"] for r in results)
    rounds = [r["rounds"] for r in results]
    mean_accepted = counts_total / max(image_rounds, 1)
    reject_rate = sum(r["rejected"] for r in results) / max(counts_total, 1)

    # roofline of the dominant kernel class over the timed region: the work of
    # all its launches over their summed duration, which the bracketed launches
    # (one in timed_every) sample
    tb = tf = 0.0
    for r in results:
        b, fl = rollout_work(dominant, shape, batch.prefix_len, r["counts"].cpu().numpy(),
                             wl.window, cfg, esz=2 if wl.dtype == "bf16" else 4)
        tb += b
        tf += fl
    t_s = dom_ms / 1e3 * timed_every
    hbm_t, mfma_t = tb / (HBM_PEAK_GBS * 1e9), tf / (BF16_PEAK_TFLOPS * 1e12)
    if mfma_t > hbm_t:
        roof = {"bound": "mfma", "achieved": round(tf / t_s / 1e12, 3), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(tb / t_s / 1e9, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 5)
    # the whole path over the timed rollouts (prefill and rounds)
    pb = pf = 0.0
    for r in results:
        b, fl = path_work(shape, batch.prefix_len, r["counts"].cpu().numpy(), wl.window, cfg,
                          esz=2 if wl.dtype == "bf16" else 4)
        pb += b
        pf += fl
    path = {"bytes_per_step": round(pb / len(results)), "flops_per_step": round(pf / len(results)),
            "achieved_gbs": round(pb / elapsed / 1e9, 2),
            "frac_hbm": round(pb / elapsed / 1e9 / HBM_PEAK_GBS, 5),
            "achieved_tflops": round(pf / elapsed / 1e12, 3),
            "frac_mfma": round(pf / elapsed / 1e12 / BF16_PEAK_TFLOPS, 5),
            "bound": "hbm" if pb / (HBM_PEAK_GBS * 1e9) >= pf / (BF16_PEAK_TFLOPS * 1e12)
            else "mfma"}
    roof["traffic"] = measured_traffic(dominant)
    roof["kernel"] = dominant
    roof["launches"] = dom_n * timed_every
    roof["timed_launches"] = dom_n
    roof["timed_every"] = timed_every
    roof["avg_launch_us"] = round(1000.0 * dom_ms / max(dom_n, 1), 3)
    roof["time_share"] = round(t_s / elapsed, 4)

    if ar is not None:
        ar["value"] = round(committed_per_step * ar["steps"] * 1000.0 / (ar["ms_per_step"] * ar["steps"]), 1)
        ar["unit"] = "tokens/s"
        ar["speedup_of_sjd"] = round(value / ar["value"], 3)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        cores = min(16, os.cpu_count() or 1)
        n_img = args.cpu_images or min(cores, B)
        rb = synth.bf16_rounded_blob(shape, blob) if wl.dtype == "bf16" else blob
        v, committed, dt = cpu_baseline(shape, rb, batch, wl, n_img, rounds=6)
        cpu = {"value": round(v, 2), "unit": "tokens/s", "cores": min(cores, n_img),
               "kind": "oracle",
               "sample": f"first {n_img} images of the same batch, prefill + 6 rounds "
                         f"({committed} committed tokens in {dt:.1f} s), fp32 oracle on the "
                         f"bf16-rounded weights"}

    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1000.0 * elapsed / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights, uniform random prefixes)",
        "config": {"workload": f"{args.workload}: {shape.n_layers}L d{shape.d_model} "
                               f"h{shape.n_heads} f{shape.mlp_hidden} V{shape.vocab} "
                               f"{shape.grid}x{shape.grid}, batch {B}, W {wl.window}, "
                               f"top-k {wl.top_k}, cfg {wl.cfg_scale}",
                   "batch": B, "window": wl.window, "history": wl.history,
                   "exec_mode": args.exec_mode, "gamma": gamma,
                   "gamma_source": "given" if args.gamma >= 0 else "calibrated",
                   "parallelism": "single GPU"},
        "mean_accepted_tokens_per_round": round(mean_accepted, 4),
        "rounds_per_step": rounds,
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
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
