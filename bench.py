#!/usr/bin/env python3
"""Benchmark of the SLiM compressed linear layer on one MI355X.

Default: the decode-shaped layer (X bf16 [16 x 4096], W 4096 x 4096 packed 2:4 + int4 group-128,
rank-384 fp16 adapter), the weight-stream GB/s half of the metric, followed in the same JSON line by
the prefill layer (X bf16 [2048 x 4096], W 11008 x 4096, rank 384), the dense-equivalent TFLOP/s
half ("prefill" object), and by the SLoPe training step after the input gradient on the 70B MLP
projection ("train" object: masked weight gradient, sparse add, pack update, transposed repack).
One step = one slim_linear call per layer on inputs resident in HBM; the weight copies rotate over
more than 3x the 256 MB MALL, one running copy counter across the warm-up, timed and per-kernel
passes, so the weight stream comes from HBM. Per-kernel figures (average and median) come from at
least 200 dispatches (40 for the training step), timed by their own dispatches in short bursts
right after replays of the timed steps; the roofline uses the average. Prints one JSON line.

  python bench.py [--steps K] [--warmup W]
                  [--workload decode|prefill|block13b|mlp70b|mlp70b_bwd|tiny|train70b|slimquant|slimlora]
                  [--m M] [--no-cpu-baseline] [--no-prefill] [--no-train] [--qadapter] [--dispatches D]
  python bench.py --copy-probe MB     # plain device copy of MB megabytes (counter calibration)
  python bench.py --vendor-probe      # torch.mm (the vendor dense GEMM) on the same shapes, as context

The roofline's "traffic" field comes from the hardware-counter summary committed under profiles/
for the same kernel and workload; it is null when no summary matches, or when the kernel sources
have changed since the counters were taken (the summary records their hash).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

METRIC = "dense-equiv TFLOP/s (M≥2048) and weight-stream HBM GB/s (M≤16), 2:4+int4+LoRA"
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
MFMA_F16_PEAK_TFS = 2516.6       # MI355X dense fp16/bf16 MFMA
PACK_BYTES_PER_WEIGHT = 0.390625  # 4-bit code x 1/2 + 2-bit index x 1/2 + fp16 scale / 128
WARM_MS = 200.0                   # sustained work before the measured replay (clock ramp-up)
KBURST = 4                        # event-recorded steps per burst of the per-kernel pass
TRAIN_STEPS, TRAIN_DISPATCHES = 10, 40   # the training step runs milliseconds


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="decode", choices=WORKLOADS)
    ap.add_argument("--m", type=int, default=None, help="rows of X (tokens); default per workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true",
                    help="decode workload only: skip the second (prefill, M = 2048) measurement")
    ap.add_argument("--qadapter", action="store_true",
                    help="forward with 4-bit group-128 adapters (slim_pack_adapter_q / slim_linear_qa)")
    ap.add_argument("--no-train", action="store_true", help="skip the training-step object of the default line")
    ap.add_argument("--dispatches", type=int, default=200,
                    help="steps of the per-kernel pass (average and median per kernel; at least --steps)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU budget of the oracle baseline (about 10-30 s)")
    ap.add_argument("--vendor-probe", action="store_true",
                    help="time torch.mm, the vendor's dense GEMM, on the shapes of the workloads (context only)")
    ap.add_argument("--copy-probe", type=float, default=None, metavar="MB",
                    help="only run a plain device-to-device copy of MB megabytes (HBM counter calibration)")
    return ap.parse_args()


ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("include/slim.h", "paper_2608_24070_amd/csrc/api.cpp", "paper_2608_24070_amd/csrc/slim_host.h",
                  "paper_2608_24070_amd/csrc/slim_device.h", "paper_2608_24070_amd/csrc/sparse_gemm.hip",
                  "paper_2608_24070_amd/csrc/adapter_gemm.hip", "paper_2608_24070_amd/csrc/pack.hip",
                  "paper_2608_24070_amd/csrc/train.hip", "paper_2608_24070_amd/csrc/quant.hip",
                  "paper_2608_24070_amd/csrc/lora.hip", "paper_2608_24070_amd/csrc/hybrid.hip")


def kernel_source_hash():
    """sha256 over the sources that decide what the measured kernels do (first 16 hex digits)."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(rel.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def counter_traffic(kernel, workload_key):
    """HBM bytes per launch of `kernel` on `workload_key` from the committed counter summary.

    profiles/hbm_traffic.txt holds lines
        traffic <kernel> <workload> <fetch_bytes> <write_bytes> <source_hash>
    with FETCH_SIZE and WRITE_SIZE already scaled by the copy-kernel calibration. Returns None if
    no line matches or the sources have changed since.
    """
    path = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    cur = kernel_source_hash()
    with open(path) as f:
        for line in f:
            t = line.split()
            if len(t) == 6 and t[0] == "traffic" and t[1] == kernel and t[2] == workload_key and t[5] == cur:
                return float(t[3]) + float(t[4])
    return None


def copy_probe(mb):
    """A plain device copy of `mb` MB, 10 times: the known-size kernel the HBM counters are scaled by."""
    import torch
    n = int(mb * 1e6) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b.copy_(a)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    print(json.dumps({"copy_probe_bytes_each_way": n * 4, "launches": 11, "avg_ms": round(ms, 4),
                      "read_plus_write_GBps": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}))


def vendor_probe():
    """torch.mm (rocBLAS / hipBLASLt) on dense operands of the shapes measured here: the weight
    gradient's [N x M] . [M x K] in bf16, and the forward products in fp16 with the dense weight
    (prefill, 70B at M 8192, decode at M 16); a point of comparison for the library's kernels, not
    part of the path. Back-to-back calls on one weight, so small ones may be served from cache."""
    import torch
    g = torch.Generator(device="cuda:0")
    g.manual_seed(0)

    def timeit(fn, reps):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    out = {}
    for name, (m, k, n, dt, reps) in {
            "grad_w 70B: [28672 x 8192] . [8192 x 8192] bf16": (28672, 8192, 8192, torch.bfloat16, 10),
            "prefill: [2048 x 4096] . [4096 x 11008] fp16": (2048, 4096, 11008, torch.float16, 50),
            "70B MLP M 8192: [8192 x 8192] . [8192 x 28672] fp16": (8192, 8192, 28672, torch.float16, 10),
            "decode: [16 x 4096] . [4096 x 4096] fp16": (16, 4096, 4096, torch.float16, 200),
            "70B MLP M 16: [16 x 8192] . [8192 x 28672] fp16": (16, 8192, 28672, torch.float16, 100)}.items():
        a = torch.randn(m, k, device="cuda:0", dtype=dt, generator=g)
        b = torch.randn(k, n, device="cuda:0", dtype=dt, generator=g)
        us = timeit(lambda: torch.mm(a, b), reps)
        out[name] = {"us": round(us, 2), "TFLOP/s": round(2 * m * k * n / us / 1e6, 1),
                     "GB/s (weight)": round(2 * k * n / us / 1e3, 1)}
        del a, b
    print(json.dumps({"vendor_probe": out}))


def layer_bytes(M, N, K, r, qadapter=False):
    """Algorithmic bytes of one forward layer call: packed weight + adapter + bf16 X + fp32 Y."""
    return N * K * PACK_BYTES_PER_WEIGHT + adapter_bytes(K, N, r, qadapter) + 2 * M * K + 4 * M * N


def kernel_bytes(kernel, M, N, K, r, bwd, has_finish=True, qadapter=False):
    """Algorithmic HBM bytes of one launch of a library kernel on one layer: the operands it must
    read and the results it must produce, once each (split partials and re-reads not counted).
    Forward: rows = N, reduction = K; backward: rows = K, reduction = N."""
    rows, red = (K, N) if bwd else (N, K)
    weight = N * K * PACK_BYTES_PER_WEIGHT
    first = (r * red // 2 + 2 * r * ((red + 127) // 128)) if qadapter else 2 * r * red
    second = (rows * r // 2 + 2 * rows * ((r + 127) // 128)) if qadapter else 2 * r * rows
    if kernel.startswith("decode"):      # packed weight + adapter first factor + activations -> T (fp16)
        return weight + first + 2 * M * red + 2 * M * r + (0 if has_finish else 4 * M * rows)
    if kernel.startswith("finish"):      # adapter second factor + T -> Y
        return second + 2 * M * r + 4 * M * rows
    if kernel.startswith("tile"):        # packed weight + fp16 activations + second factor + T -> Y
        return weight + 2 * M * red + 2 * r * rows + 2 * M * r + 4 * M * rows
    if kernel.startswith("adapter_gemm"):  # fp16 activations + first factor -> T
        return 2 * M * red + 2 * r * red + 2 * M * r
    if kernel.startswith("rowprep"):     # activations -> their row-scaled fp16 copy
        return 4 * M * red + 4 * M
    return 0


def layer_flops(M, N, K, r):
    """Dense-equivalent FLOPs: the 2:4 product counted as dense, plus both adapter products."""
    return 2 * M * N * K + 2 * M * r * (K + N)


WORKLOADS = ["decode", "prefill", "block13b", "mlp70b", "mlp70b_bwd", "tiny", "train70b", "slimquant", "slimlora",
             "patch7b"]
FP64_PEAK_TFS = 78.6        # MI355X fp64 vector peak


def workload_layers(wk, m):
    from paper_2608_24070_amd import configs
    if wk == "decode":
        return configs.DECODE.layers, m or 16
    if wk == "prefill":
        return configs.PREFILL.layers, m or 2048
    if wk == "block13b":
        return configs.BLOCK13B.layers, m or 4096
    if wk in ("mlp70b", "mlp70b_bwd"):
        return configs.MLP70B.layers, m or 8192
    return configs.TINY.layers, m or 16


def adapter_bytes(K, N, r, qadapter):
    """Bytes of the adapter factors: fp16, or 4-bit codes plus an fp16 scale per 128 elements."""
    if not qadapter:
        return 2 * r * (K + N)
    return r * K // 2 + 2 * r * ((K + 127) // 128) + N * r // 2 + 2 * N * ((r + 127) // 128)


def measure(wk, m, steps, warmup, dispatches, qadapter=False):
    """Set up one workload (synthetic inputs resident in HBM, packed once, > 3x the MALL of distinct
    weight copies) and time it: K timed steps back to back, then `dispatches` steps with per-kernel
    events. Every pass takes the next copy from one running counter, so a copy is read again only
    after every other copy has been."""
    import torch
    from paper_2608_24070_amd import slim, synth

    dev = torch.device("cuda:0")
    layers, M = workload_layers(wk, m)
    bwd = wk == "mlp70b_bwd"

    def dev_bits(bits, dtype):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(dtype)

    t0 = time.time()
    per_layer = []
    pack_ms = 0.0
    for ly in layers:
        W = torch.from_numpy(synth.weights(ly.n, ly.k, seed=0, name=f"{wk}/{ly.name}/W")).to(dev)
        Lb, Rb, _, _ = synth.adapter(ly.k, ly.n, ly.r, seed=0, name=f"{wk}/{ly.name}/")
        torch.cuda.synchronize()
        tp = time.perf_counter()
        p = slim.pack(W)
        if bwd:
            p = slim.pack_bwd(p)
        torch.cuda.synchronize()
        pack_ms += (time.perf_counter() - tp) * 1e3
        del W
        ad = slim.pack_adapter(dev_bits(Lb, torch.float16), dev_bits(Rb, torch.float16))
        pl = {"layer": ly, "pack": p, "L": ad["L"], "R": ad["R"], "Lt": ad["Lt"], "Rt": ad["Rt"]}
        if qadapter:
            pl["qa"] = slim.pack_adapter_q(ad["L"], ad["R"])
        per_layer.append(pl)
    # activations: q/k/v/gate/up of the block share X; o and down get their own
    acts = {}
    for ly in layers:
        a_len = ly.n if bwd else ly.k
        key = (ly.name if ly.name in ("o", "down") else "shared", a_len)
        if key not in acts:
            bits, _ = synth.activations(M, a_len, seed=0, name=f"{wk}/{key[0]}/X")
            acts[key] = dev_bits(bits, torch.bfloat16)
    for pl in per_layer:
        ly = pl["layer"]
        a_len = ly.n if bwd else ly.k
        pl["x"] = acts[(ly.name if ly.name in ("o", "down") else "shared", a_len)]
        pl["out"] = torch.empty((M, ly.k if bwd else ly.n), dtype=torch.float32, device=dev)

    # distinct copies of the weight side over > 3x the 256 MB MALL (capped at 2 GB)
    copy_bytes = sum(pl["pack"]["codes" if not bwd else "codesT"].numel() * 1.5625 + pl["L"].numel() * 4
                     for pl in per_layer)
    n_copies = int(min(64, max(1, math.ceil(3 * 256e6 / copy_bytes)), max(1, 2e9 // copy_bytes)))
    copies = []
    for c in range(n_copies):
        cp = []
        for pl in per_layer:
            if qadapter:
                ad = {k: v for k, v in pl["qa"].items()}
            else:
                ad = {"L": pl["L"], "R": pl["R"]} if bwd else {"Lt": pl["Lt"], "Rt": pl["Rt"]}
            if c == 0:
                cp.append({"pack": pl["pack"], "ad": ad})
            else:
                cp.append({"pack": {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in pl["pack"].items()},
                           "ad": {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in ad.items()}})
        copies.append(cp)
    wsq = slim.slim_bwd_dx_workspace if bwd else (slim.slim_linear_qa_workspace if qadapter else slim.slim_linear_workspace)
    ws_need = max(wsq(
        M, pl["layer"].n, pl["layer"].k, pl["layer"].r) for pl in per_layer)
    ws = torch.zeros(ws_need + 256, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    counter = [0]

    def step():
        cp = copies[counter[0] % n_copies]
        counter[0] += 1
        for pl, c in zip(per_layer, cp):
            if bwd:
                slim.bwd_dx(pl["x"], c["pack"], c["ad"]["L"], c["ad"]["R"], out=pl["out"], ws=ws)
            elif qadapter:
                slim.linear_qa(pl["x"], c["pack"], c["ad"], out=pl["out"], ws=ws)
            else:
                slim.linear(pl["x"], c["pack"], c["ad"], out=pl["out"], ws=ws)

    # Timed region: the K steps are captured once into a HIP graph (the library records only kernel
    # launches, so a replay runs exactly the eager steps back to back, with no host launch gaps), and a
    # second graph holds the steps over the other weight copies, so that in the cycle (filler, timed)
    # every copy is read once. Both are replayed for at least WARM_MS before the measured replay so the
    # GPU runs at the clock of sustained work; two events bracket exactly the K timed steps.
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(5):
        step()
    host_ms = (time.perf_counter() - t) / 5 * 1e3       # host enqueue cost of one eager step
    torch.cuda.synchronize()
    n_fill = max(0, n_copies - steps)
    g_fill, g_timed = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    if n_fill:
        with torch.cuda.graph(g_fill):
            for _ in range(n_fill):
                step()
    with torch.cuda.graph(g_timed):
        for _ in range(steps):
            step()
    torch.cuda.synchronize()
    tw = time.perf_counter()
    warm_cycles = 0
    while (time.perf_counter() - tw) * 1e3 < WARM_MS and warm_cycles < 200:
        if n_fill:
            g_fill.replay()
        g_timed.replay()
        warm_cycles += 1
        torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if n_fill:
        g_fill.replay()
    ev0.record(stream)
    g_timed.replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / steps
    print(f"[bench] {wk} M={M}: {ms_per_step * 1e3:.2f} us/step over {steps} steps "
          f"({n_copies} weight copies, host enqueue {host_ms * 1e3:.0f} us/step, {warm_cycles} warm-up cycles, "
          f"setup {setup_s:.1f}s)", file=sys.stderr, flush=True)

    # Per-kernel durations: each library launch records a start and a stop event as part of its own
    # dispatch (slim_timing_*, hipExtLaunchKernel), so they carry the kernel's begin and end times.
    # Event-recorded launches leave the GPU idle for microseconds between kernels, and a long run of
    # them lets the GPU fall out of the state of sustained work (kernel times up to 1.5x the ones in
    # the timed replay); so the pass runs in bursts of KBURST event-recorded steps, each right after a
    # replay of the timed graphs. The per-kernel times then add up to no more than the measured step.
    slim.slim_timing_reset()
    done = 0
    while done < dispatches:
        if n_fill:
            g_fill.replay()
        g_timed.replay()
        slim.slim_timing_enable(True)
        for _ in range(min(KBURST, dispatches - done)):
            step()
        slim.slim_timing_enable(False)
        done += KBURST
    torch.cuda.synchronize()
    kt = slim.slim_timing_read()
    del g_fill, g_timed
    kernels = {k: {"launches": n, "avg_us": round(1e3 * ms / max(n, 1), 3), "median_us": round(1e3 * med, 3)}
               for k, (n, ms, med) in kt.items()}
    dominant = max(kt.items(), key=lambda kv: kv[1][1])[0]
    launches_per_step = kt[dominant][0] / dispatches
    # average launch duration: the per-launch figure below is a mean over the step's layers, which differ
    # in shape in the 13B block, so it pairs with the mean duration (total time over launches)
    avg_s = kt[dominant][1] / kt[dominant][0] * 1e-3

    tot_bytes = sum(layer_bytes(M, pl["layer"].n, pl["layer"].k, pl["layer"].r, qadapter) for pl in per_layer)
    tot_flops = sum(layer_flops(M, pl["layer"].n, pl["layer"].k, pl["layer"].r) for pl in per_layer)
    has_finish = any(k.startswith("finish") for k in kt)
    wkey = f"{wk}_m{M}"
    if M <= 32:
        unit = "GB/s"
        value = tot_bytes / (ms_per_step * 1e-3) / 1e9
        dk_bytes = sum(kernel_bytes(dominant, M, pl["layer"].n, pl["layer"].k, pl["layer"].r, bwd, has_finish, qadapter)
                       for pl in per_layer) / launches_per_step
        achieved = dk_bytes / avg_s / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_launch": int(dk_bytes)}
    else:
        unit = "TFLOP/s"
        value = tot_flops / (ms_per_step * 1e-3) / 1e12
        # dominant kernel (the sparse contraction): dense-equivalent 2MNK plus the adapter's second product
        dk_flops = sum(2 * M * pl["layer"].n * pl["layer"].k + 2 * M * pl["layer"].r *
                       (pl["layer"].k if bwd else pl["layer"].n) for pl in per_layer) / launches_per_step
        achieved = dk_flops / avg_s / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_F16_PEAK_TFS, "unit": "TFLOP/s",
                    "frac": round(achieved / MFMA_F16_PEAK_TFS, 4), "dense_equiv_flops_per_launch": int(dk_flops)}
    traffic = counter_traffic(dominant, wkey)
    roofline["traffic"] = None if traffic is None else round(traffic / 1e6, 3)
    roofline["traffic_unit"] = "MB per launch (HBM fetch + write, copy-calibrated counters)"
    roofline["kernel"] = dominant
    roofline["timing"] = (f"average of {kt[dominant][0]} dispatches; hip events recorded by each kernel dispatch "
                          f"(hipExtLaunchKernel), in bursts of {KBURST} steps each right after a replay of the "
                          "timed graphs")

    shape = ", ".join(f"{ly.name} {ly.n}x{ly.k} r{ly.r}" for ly in layers)
    ly0 = layers[0]
    res = {
        "value": round(value, 2), "unit": unit, "ms_per_step": round(ms_per_step, 6),
        "config": {
            "workload": f"{wk}: M={M}, {shape}, bf16 {'dY' if bwd else 'X'}, "
                        f"{'dX' if bwd else 'Y'} fp32, 2:4 + int4 group-128 weights"
                        + (", int4 group-128 adapters" if qadapter else ", fp16 adapters"),
            "M": M, "layers": len(layers), "N": ly0.n, "K": ly0.k, "r": ly0.r,
            "bytes_per_step": int(tot_bytes), "dense_equiv_flops_per_step": int(tot_flops),
            "weight_copies_rotated": n_copies, "pack_ms_one_time": round(pack_ms, 2),
        },
        "kernels": kernels,
        "roofline": roofline,
    }
    del copies, per_layer, acts, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res, layers, M, bwd


def measure_train(steps, warmup, dispatches, m=8192, n=28672, k=8192):
    """The training-step calls after the input gradient (SLoPe) on the 70B MLP projection: one step =
    slim_grad_w (dY [m, n], X [m, k] bf16 -> masked, compressed fp32 gradient) + slim_sparse_add
    (loss scale and weight decay) + slim_update_pack16 + slim_pack16_t (transposed repack). Timed as
    one replay of a captured K-step graph after WARM_MS of replays; per-kernel times as measure()."""
    import torch
    from paper_2608_24070_amd import slim
    dev = torch.device("cuda:0")
    t0 = time.time()
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    W = torch.randn((n, k), device=dev, generator=gen) * 0.02
    p = slim.pack16(W)
    del W
    pt = slim.pack16_t(p)
    dY = (torch.randn((m, n), device=dev, generator=gen) * 0.01).to(torch.bfloat16)
    X = torch.randn((m, k), device=dev, generator=gen).to(torch.bfloat16)
    g = torch.empty((n, k // 2), dtype=torch.float32, device=dev)
    upd = torch.empty_like(g)
    wnew = p["vals"].view(torch.float16).float()        # the optimizer's output stands in fixed
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    def step():
        slim.grad_w(dY, X, p, out=g)
        slim.sparse_add(g, p["vals"], 1.0 / 1024.0, 0.01, out=upd)
        slim.update_pack16(wnew, p)
        slim.pack16_t(p, out=pt)

    # a step takes milliseconds: at most TRAIN_STEPS timed steps and TRAIN_DISPATCHES per-kernel steps
    steps = min(steps, TRAIN_STEPS)
    dispatches = min(dispatches, TRAIN_DISPATCHES)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    gt, g1 = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gt):
        for _ in range(steps):
            step()
    with torch.cuda.graph(g1):
        step()
    torch.cuda.synchronize()
    tw = time.perf_counter()
    warm = 0
    while (time.perf_counter() - tw) * 1e3 < WARM_MS and warm < 200:
        gt.replay()
        warm += 1
        torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    gt.replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    print(f"[bench] train step M={m}: {ms * 1e3:.2f} us/step over {steps} steps ({warm} warm-up cycles, "
          f"setup {setup_s:.1f}s)", file=sys.stderr, flush=True)
    slim.slim_timing_reset()
    done = 0
    while done < dispatches:
        g1.replay()
        slim.slim_timing_enable(True)
        for _ in range(min(KBURST, dispatches - done)):
            step()
        slim.slim_timing_enable(False)
        done += KBURST
    torch.cuda.synchronize()
    kt = slim.slim_timing_read()
    del gt, g1
    kernels = {kn: {"launches": c, "avg_us": round(1e3 * tot / max(c, 1), 3), "median_us": round(1e3 * med, 3)}
               for kn, (c, tot, med) in kt.items()}
    flops = 2.0 * m * n * k                                  # issued by the gradient kernel (dense tile)
    avg_s = kt["grad_w"][1] / kt["grad_w"][0] * 1e-3
    achieved = flops / avg_s / 1e12
    traffic = counter_traffic("grad_w", f"train70b_m{m}")
    res = {
        "metric": "dense-equiv TFLOP/s of the weight-gradient step",
        "value": round(flops / (ms * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "ms_per_step": round(ms, 6),
        "config": {"workload": f"train step after dX: 70B MLP projection {n}x{k}, M={m}, bf16 dY and X, "
                               "fp16 value packs, fp32 gradient", "M": m, "N": n, "K": k,
                   "dense_equiv_flops_per_step": flops},
        "kernels": kernels,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_F16_PEAK_TFS, "unit": "TFLOP/s",
                     "frac": round(achieved / MFMA_F16_PEAK_TFS, 4), "dense_equiv_flops_per_launch": flops,
                     "traffic": None if traffic is None else round(traffic / 1e6, 3),
                     "traffic_unit": "MB per launch (HBM fetch + write, copy-calibrated counters)",
                     "kernel": "grad_w",
                     "timing": f"average of {kt['grad_w'][0]} dispatches; hip events recorded by each kernel "
                               f"dispatch, in bursts of {KBURST} steps each right after a replayed step",
                     "note": "the kernel computes the dense tile and keeps the half M^R selects"},
    }
    del p, pt, dY, X, g, upd, wnew
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def _host_fields():
    model, usable, nproc = host_cpu()
    return {"cpu_model": model, "nproc": nproc, "usable_cpus": usable}


def _sync_call_times(call, steps, dispatches):
    """Wall time per call of a synchronous library call (it reads back a status word, so it cannot be
    captured in a graph), and per-kernel times from `dispatches` further calls with the timing hooks on."""
    import torch
    from paper_2608_24070_amd import slim
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    slim.slim_timing_reset()
    slim.slim_timing_enable(True)
    for _ in range(dispatches):
        call()
    slim.slim_timing_enable(False)
    torch.cuda.synchronize()
    kt = slim.slim_timing_read()
    kernels = {kn: {"launches": c, "avg_us": round(1e3 * tot / max(c, 1), 3), "median_us": round(1e3 * med, 3)}
               for kn, (c, tot, med) in kt.items()}
    return ms, kt, kernels


def measure_slimquant(steps, warmup, dispatches, cpu, n=28672, k=8192):
    """SLiM-Quant's scale search (slim_quant_search) on the 70B MLP projection's fp32 weight: one step
    = one search (maximum pass, histogram pass into 20000 bins, float64 grid search)."""
    import numpy as np
    import torch
    from paper_2608_24070_amd import slim
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    W = torch.randn((n, k), device=dev, generator=gen) * 0.02
    for _ in range(max(warmup, 1)):
        slim.quant_search(W)
    steps = min(steps, 50)
    ms, kt, kernels = _sync_call_times(lambda: slim.quant_search(W), steps, min(dispatches, 50))
    nbytes = 4.0 * n * k
    avg_s = kt["quant_hist"][1] / kt["quant_hist"][0] * 1e-3
    achieved = nbytes / avg_s / 1e9
    print(f"[bench] slim-quant search {n}x{k}: {ms * 1e3:.1f} us/search", file=sys.stderr, flush=True)
    base = None
    if cpu:
        from oracle import slim_quant as Q
        rows = 2048
        Wh = W[:rows].cpu().numpy()
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 10.0 or reps < 1:
            Q.search(Wh, bins=Q.bin_count(n, k))
            reps += 1
        sec = (time.perf_counter() - t0) / reps
        base = {"value": round(rows * k * 4 / sec / 1e9, 4), "unit": "GB/s", "cores": torch.get_num_threads(),
                "kind": "oracle", "sample": f"search over the first {rows} of {n} rows ({reps} calls, "
                                            f"{sec * 1e3:.0f} ms each)", **_host_fields()}
    return {
        "metric": "SLiM-Quant scale search, weight GB/s (fp32 bytes of W per search time)",
        "value": round(nbytes / (ms * 1e-3) / 1e9, 2), "unit": "GB/s", "ms_per_step": round(ms, 6),
        "config": {"workload": f"slim-quant search: 70B MLP projection {n}x{k} fp32 W, 4-bit, 20000 bins",
                   "N": n, "K": k, "bins": slim.slim_quant_bins(n, k)},
        "kernels": kernels,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_launch": int(nbytes),
                     "traffic": None, "kernel": "quant_hist",
                     "timing": f"average of {kt['quant_hist'][0]} dispatches; hip events recorded by each kernel "
                               "dispatch"},
        "cpu_baseline": base,
    }


def measure_slimlora(steps, warmup, cpu, n=4096, k=4096, r=384, b=2048):
    """SLiM-LoRA (slim_lora) on the decode layer 4096 x 4096 at rank 384 with 2048 bf16 calibration
    rows (1% outlier channels x20): one step = one adapter fit."""
    import numpy as np
    import torch
    from paper_2608_24070_amd import slim, synth
    dev = torch.device("cuda:0")
    W = torch.from_numpy(synth.weights(n, k, seed=0, name="bench/lora/W")).to(dev)
    xbits, _ = synth.activations(b, k, seed=0, name="bench/lora/X", dtype="bf16", outliers=True)
    X = torch.from_numpy(xbits.view(np.int16)).to(dev).view(torch.bfloat16)
    p = slim.pack(W)
    for _ in range(max(min(warmup, 1), 1)):
        out = slim.lora(W, p, X, r)
    steps = min(steps, 3)
    ms, kt, kernels = _sync_call_times(lambda: slim.lora(W, p, X, r), steps, 1)
    sweeps = out["sweeps"]
    dp = (min(n, k) + 63) // 64 * 64                       # the Gram side, padded to the 64-wide pairs
    npair = dp // 64
    # FLOPs per launch of the two kernels that can dominate a fit: the tile update of G, J_a^T (G J_c)
    # on the tiles a <= c, and the pair solves, 63 steps of 32 rotations per pair, each rotating two
    # rows (6 FLOPs per element) and two columns of the pair's G block and of its J (12)
    flops_of = {"lora_apply_g": 4.0 * 64 ** 3 * npair * (npair + 1) / 2,
                "lora_pair_solve": float(npair * 63 * 32 * 64 * 18)}
    # the roofline prices the dominant kernel by total time (raises if it is neither of those)
    dom = max(kt.items(), key=lambda kv: kv[1][1])[0]
    if dom not in flops_of:
        raise RuntimeError(f"slim-lora: dominant kernel is {dom}, which has no FLOP model here")
    flops = flops_of[dom]
    avg_s = kt[dom][1] / kt[dom][0] * 1e-3
    achieved = flops / avg_s / 1e12
    print(f"[bench] slim-lora {n}x{k} r={r}: {ms:.1f} ms/fit, {sweeps} sweeps", file=sys.stderr, flush=True)
    base = None
    if cpu:
        from oracle import slim_lora as LR
        from oracle import slim_oracle as O
        rows = 1024                                          # the oracle's SVD on a 1024-row slice of W
        Wh = W[:rows].cpu().numpy()
        ref = O.pack(Wh)
        Wc = O.unpack(ref["codes"], ref["meta"], ref["scales"], rows, k)
        Xh = X.float().cpu().numpy()
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 10.0 or reps < 1:
            LR.lora(Wh, Wc, Xh, r)
            reps += 1
        sec = (time.perf_counter() - t0) / reps
        base = {"value": round(1.0 / sec, 4), "unit": "fits/s", "cores": torch.get_num_threads(), "kind": "oracle",
                "sample": f"adapter fit of a {rows} x {k} slice of W (rank {r}, {b} calibration rows; the SVD cost "
                          f"grows with the slice), {reps} calls of {sec * 1e3:.0f} ms", **_host_fields()}
    return {
        "metric": "SLiM-LoRA adapter fit, fits/s",
        "value": round(1e3 / ms, 4), "unit": "fits/s", "ms_per_step": round(ms, 3),
        "config": {"workload": f"slim-lora: decode layer {n}x{k}, rank {r}, {b} bf16 calibration rows "
                               "(1% outlier channels x20), float64 block-Jacobi", "N": n, "K": k, "r": r, "B": b,
                   "jacobi_sweeps": sweeps},
        "kernels": kernels,
        "roofline": {"bound": "alu", "achieved": round(achieved, 2), "peak": FP64_PEAK_TFS, "unit": "TFLOP/s",
                     "frac": round(achieved / FP64_PEAK_TFS, 4), "flops_per_launch": int(flops), "traffic": None,
                     "kernel": dom,
                     "timing": f"average of {kt[dom][0]} dispatches of one fit; hip events recorded by "
                               "each kernel dispatch"},
        "cpu_baseline": base,
    }


def measure_hybrid(steps, warmup, dispatches, m, frac, n=11008, k=4096, seed=0):
    """PATCH's hybrid dense / 2:4 tile layer (slim_linear_hybrid) on the LLaMA-2-7B gate projection
    11008 x 4096 with a synthetic tile map (fraction `frac` of the 128 x 128 tiles 2:4, the rest
    dense; sparsity frac / 2), fp16 X [m, 4096]. Timed like measure(): a captured graph of `steps`
    calls over weight copies rotating past the MALL, after WARM_MS of replays."""
    import numpy as np
    import torch
    from paper_2608_24070_amd import slim
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    W = torch.randn((n, k), device=dev, generator=gen) * 0.02
    kinds = (np.random.default_rng(seed).random((n // 128, k // 128)) < frac).astype(np.uint8)
    p0 = slim.pack_hybrid(W, kinds)
    wbytes = int(p0["payload"].numel())
    n_copies = max(1, min(64, -(-3 * 256 * 2 ** 20 // wbytes))) if m <= 32 else 1
    copies = [p0] + [{"tile_info": p0["tile_info"], "payload": p0["payload"].clone(), "N": n, "K": k}
                     for _ in range(n_copies - 1)]
    del W
    X = (torch.randn((m, k), device=dev, generator=gen)).to(torch.float16)
    Y = torch.empty((m, n), dtype=torch.float32, device=dev)
    ctr = [0]

    def step():
        slim.linear_hybrid(X, copies[ctr[0] % n_copies], out=Y)
        ctr[0] += 1

    for _ in range(max(warmup, 2)):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    graphs = []
    for _ in range(n_copies if m <= 32 else 1):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(steps):
                step()
        graphs.append(g)
    torch.cuda.synchronize()
    tw = time.perf_counter()
    while (time.perf_counter() - tw) * 1e3 < WARM_MS:
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    graphs[0].replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    slim.slim_timing_reset()
    done = 0
    while done < dispatches:
        graphs[0].replay()
        slim.slim_timing_enable(True)
        for _ in range(min(KBURST, dispatches - done)):
            step()
        slim.slim_timing_enable(False)
        done += KBURST
    torch.cuda.synchronize()
    kt = slim.slim_timing_read()
    del graphs, copies
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    kernels = {kn: {"launches": c, "avg_us": round(1e3 * tot / max(c, 1), 3), "median_us": round(1e3 * med, 3)}
               for kn, (c, tot, med) in kt.items()}
    avg_s = kt["hybrid_gemm"][1] / kt["hybrid_gemm"][0] * 1e-3
    flops = 2.0 * m * n * k
    algo_bytes = wbytes + 2 * m * k + 4 * m * n
    if m <= 32:
        achieved = algo_bytes / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_launch": int(algo_bytes)}
        value, unit = algo_bytes / (ms * 1e-3) / 1e9, "GB/s"
    else:
        achieved = flops / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_F16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_F16_PEAK_TFS, 4), "dense_equiv_flops_per_launch": int(flops)}
        value, unit = flops / (ms * 1e-3) / 1e12, "TFLOP/s"
    roof.update({"traffic": None, "kernel": "hybrid_gemm",
                 "timing": f"average of {kt['hybrid_gemm'][0]} dispatches; hip events recorded by each kernel "
                           f"dispatch, in bursts of {KBURST} steps each right after a replay of the timed graph"})
    print(f"[bench] patch hybrid {n}x{k} M={m} sparse tiles {kinds.mean():.3f}: {ms * 1e3:.2f} us/step "
          f"({n_copies} weight copies)", file=sys.stderr, flush=True)
    return {"value": round(value, 2), "unit": unit, "ms_per_step": round(ms, 6),
            "config": {"workload": f"patch hybrid tiles: LLaMA-2-7B gate projection {n}x{k}, M={m}, fp16 X and "
                                   f"weights, {100 * kinds.mean():.1f}% of 128x128 tiles 2:4 (sparsity "
                                   f"{50 * kinds.mean():.1f}%)", "M": m, "N": n, "K": k,
                       "sparse_tile_fraction": round(float(kinds.mean()), 4), "payload_bytes": wbytes,
                       "weight_copies_rotated": n_copies},
            "kernels": kernels, "roofline": roof}


def measure_patch(steps, warmup, dispatches, frac=0.7):
    """Decode (M = 16) and prefill (M = 2048, batch 16 x 128 tokens) of the hybrid layer, each with the
    same kernel on an all-dense tile map for the speedup PATCH is after."""
    out = {}
    for m in (16, 2048):
        hyb = measure_hybrid(steps, warmup, dispatches, m, frac)
        dense = measure_hybrid(steps, warmup, dispatches, m, 0.0)
        hyb["speedup_vs_dense_tiles"] = round(dense["ms_per_step"] / hyb["ms_per_step"], 4)
        hyb["dense_tiles_ms_per_step"] = dense["ms_per_step"]
        out[m] = hyb
    main = out[16]
    main["metric"] = "PATCH hybrid-tile layer, weight-stream HBM GB/s (M=16)"
    main["prefill"] = {"metric": "PATCH hybrid-tile layer, dense-equiv TFLOP/s (M=2048)", **out[2048]}
    return main


def _single_line(obj, args, dtype, extra=None):
    print(json.dumps({"metric": obj["metric"], "value": obj["value"], "unit": obj["unit"], "n_gpus": 1,
                      "steps": args.steps, "warmup": args.warmup, "ms_per_step": obj["ms_per_step"],
                      "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
                      "data": "synthetic", "config": {**obj["config"], "kernel_source_hash": kernel_source_hash()},
                      "kernels": obj["kernels"], "roofline": obj["roofline"],
                      "cpu_baseline": obj.get("cpu_baseline"), **(extra or {})}))


def main():
    args = parse()
    if args.copy_probe is not None:
        copy_probe(args.copy_probe)
        return
    if args.vendor_probe:
        vendor_probe()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer would shard along N across GPUs; no multi-GPU path is implemented).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    dispatches = max(args.dispatches, args.steps)
    if args.qadapter and args.workload == "mlp70b_bwd":
        print("--qadapter applies to the forward only", file=sys.stderr)
        sys.exit(2)
    if args.workload == "patch7b":
        obj = measure_patch(args.steps, args.warmup, dispatches)
        _single_line(obj, args, "f16", {"speedup_vs_dense_tiles": obj["speedup_vs_dense_tiles"],
                                        "dense_tiles_ms_per_step": obj["dense_tiles_ms_per_step"],
                                        "prefill": obj["prefill"]})
        return
    if args.workload == "slimquant":
        _single_line(measure_slimquant(args.steps, args.warmup, dispatches, not args.no_cpu_baseline), args, "f64")
        return
    if args.workload == "slimlora":
        _single_line(measure_slimlora(args.steps, args.warmup, not args.no_cpu_baseline), args, "f64")
        return
    if args.workload == "train70b":
        # the training-step calls alone (the object the default line carries as "train")
        tr = measure_train(args.steps, args.warmup, dispatches, m=args.m or 8192)
        print(json.dumps({"metric": tr["metric"], "value": tr["value"], "unit": tr["unit"], "n_gpus": 1,
                          "steps": min(args.steps, TRAIN_STEPS), "warmup": args.warmup,
                          "ms_per_step": tr["ms_per_step"], "higher_is_better": True, "scaling": "weak",
                          "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                          "config": {**tr["config"], "kernel_source_hash": kernel_source_hash()},
                          "kernels": tr["kernels"], "roofline": tr["roofline"], "cpu_baseline": None}))
        return
    res, layers, M, bwd = measure(args.workload, args.m, args.steps, args.warmup, dispatches, args.qadapter)
    second = None
    if args.workload == "decode" and not args.no_prefill:
        # the M >= 2048 half of the metric: the prefill layer (11008 x 4096, rank 384) at M = 2048
        s_res, _, _, _ = measure("prefill", None, args.steps, args.warmup, dispatches, args.qadapter)
        second = {"metric": "dense-equiv TFLOP/s (M≥2048)", **s_res}
    train = None
    if args.workload == "decode" and not args.no_train:
        train = measure_train(args.steps, args.warmup, dispatches)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.workload, layers, M, bwd, M <= 32, args.cpu_seconds)

    props = torch.cuda.get_device_properties(0)
    out = {
        "metric": METRIC,
        "value": res["value"],
        "unit": res["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {**res["config"], "kernel_source_hash": kernel_source_hash()},
        "kernels": res["kernels"],
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "gpu": {"name": props.name, "compute_units": props.multi_processor_count,
                "gcn_arch": getattr(props, "gcnArchName", "")},
    }
    if second is not None:
        out["prefill"] = second
    if train is not None:
        out["train"] = train
    print(json.dumps(out))


def host_cpu():
    """CPU model name (as lscpu reports it) and the logical CPUs this process may use."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return model, usable, os.cpu_count() or 1


def cpu_baseline(wk, layers, M, bwd, decode_like, budget_s):
    """Time the CPU oracle (unchanged) on a bounded sample of the same workload, on this host."""
    from oracle import slim_oracle as O
    from paper_2608_24070_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    model, usable, nproc = host_cpu()
    ly = layers[0]
    n_rows = min(ly.n, 512)
    rows = np.arange(n_rows)
    m_rows = min(M, 64)
    W = synth.weights(ly.n, ly.k, seed=0, name=f"{wk}/{ly.name}/W")[:n_rows] if not bwd else None
    _, _, L, R = synth.adapter(ly.k, ly.n, ly.r, seed=0, name=f"{wk}/{ly.name}/")
    if bwd:
        # one 128-column group of the backward: all N rows, 128 input features
        Wblk = synth.weights(ly.n, ly.k, seed=0, name=f"{wk}/{ly.name}/W")[:, :128]
        pb = O.pack_bwd(O.pack(Wblk), ly.n, 128)
        _, dY = synth.activations(m_rows, ly.n, seed=0, name="cpu/dY")
        run = lambda: O.bwd_dx(dY, pb, L[:128], R, ly.n, 128)
        flops = 2 * m_rows * ly.n * 128 + 2 * m_rows * ly.r * (ly.n + 128)
        nbytes = ly.n * 128 * PACK_BYTES_PER_WEIGHT + 2 * ly.r * (ly.n + 128) + 2 * m_rows * ly.n + 4 * m_rows * 128
        sample = f"bwd dX for {m_rows} rows x one 128-wide K group (all {ly.n} N), oracle pack excluded"
    else:
        p = O.pack(W)
        _, X = synth.activations(m_rows, ly.k, seed=0, name="cpu/X")
        run = lambda: O.linear(X, p, L, R[:, rows], n_rows, ly.k)
        flops = layer_flops(m_rows, n_rows, ly.k, ly.r)
        nbytes = layer_bytes(m_rows, n_rows, ly.k, ly.r)
        sample = f"forward for {m_rows} rows of X x {n_rows} of {ly.n} output features, oracle pack excluded"
    times = []
    t_end = time.perf_counter() + budget_s
    while time.perf_counter() < t_end or not times:
        t = time.perf_counter()
        run()
        times.append(time.perf_counter() - t)
        if len(times) >= 2000:
            break
    med = float(np.median(times))
    host = {"cpu_model": model, "nproc": nproc, "usable_cpus": usable,
            "threads_note": "cores = the BLAS thread count the oracle's float64 products ran on"}
    if decode_like:
        return {"value": round(nbytes / med / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
                "sample": sample + f"; median of {len(times)} calls ({med * 1e3:.1f} ms each)", **host}
    return {"value": round(flops / med / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": sample + f"; median of {len(times)} calls ({med * 1e3:.1f} ms each)", **host}


if __name__ == "__main__":
    main()
