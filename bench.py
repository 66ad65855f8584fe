"""Throughput of the pre-decoder hot path on one MI355X.

A step is one predecoder_run over one batch: unpack -> 8 conv3d layers
(bias + GELU fused) -> 1x1x1 head + threshold -> residual + bit repack, for
the d=13, T=13, batch-4096 workload (8 hidden layers of 128 channels, bf16
operands with fp32 accumulation, phenomenological noise p=q=0.003).  Inputs
are resident in HBM before the timed region.

Prints one JSON line: rounds/s (= batch * T / step time), us/round, the
roofline of the dominant kernel (a hidden 128->128 conv layer, MFMA-bound,
algorithmic FLOPs / its mean HIP-event duration) and the CPU oracle timed on a
bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0   # MI355X dense fp8 MFMA
PEAK_HBM_GBS = 8000.0


# The translation unit of the dominant kernel (the hidden conv layer): its
# source and every header it includes.
KERNEL_SOURCES = ("paper_2604_12841_amd/csrc/conv_hidden.hip", "paper_2604_12841_amd/csrc/tiles.h",
                  "paper_2604_12841_amd/csrc/activation.h", "paper_2604_12841_amd/csrc/internal.h",
                  "include/predecoder.h")


def kernel_source_hash():
    """sha256 over the code of the dominant kernel's translation unit
    (KERNEL_SOURCES with comments and whitespace runs removed, so that an
    edit of prose alone keeps a counter summary valid)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        text = open(os.path.join(ROOT, f)).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(f.encode())
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def counted_traffic(profile):
    """HBM bytes per launch of the dominant kernel from a committed counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated), or None when the summary is
    missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_sources_sha256:\s*([0-9a-f]{64})", text)
    m_bytes = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_source_hash():
        return None
    return int(m_bytes.group(1))


def measure_peaks(torch, pdx, stream, iters=20000, copy_mib=1024, reps=5):
    """The ceilings measured on this device (predecoder_peak_mfma /
    predecoder_peak_copy, HIP events on `stream`): back-to-back bf16 and fp8
    matrix instructions on all-zero and on random operands (four workgroups of
    four waves per compute unit), and a plain 1 GiB device copy."""
    n_wg = 4 * torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    g = torch.Generator().manual_seed(7)
    rand = {
        "bf16": torch.randn(2048, generator=g).to(torch.bfloat16).view(torch.uint8),
        "fp8": torch.randn(4096, generator=g).to(torch.float8_e4m3fn).view(torch.uint8),
    }
    res = {}

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    for dt in ("bf16", "fp8"):
        for kind in ("zero", "random"):
            ops = torch.zeros(4096, dtype=torch.uint8) if kind == "zero" else rand[dt]
            ops = ops.cuda()
            flops = []
            t = timed(lambda: flops.append(pdx.peak_mfma(dt, ops, iters, n_wg, out, stream=stream)))
            res["mfma_%s_%s_tflops" % (dt, kind)] = flops[0] / t / 1e12
    n = copy_mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    t = timed(lambda: pdx.peak_copy(src, dst, n, stream=stream))
    res["hbm_copy_gbs"] = 2 * n / t / 1e9
    res["how"] = ("predecoder_peak_mfma: %d workgroups x 4 waves, %d x 4 back-to-back v_mfma_f32_32x32x16_bf16 / "
                  "32x32x64 fp8 per wave, mean of %d launches; predecoder_peak_copy: %d MiB read + written"
                  % (n_wg, iters, reps, copy_mib))
    del src, dst
    return res


def graph_replays(torch, pre, ddet, flips, res, stream, n, warmup):
    """Median / p10 / p90 of `n` recorded-run replays (each timed with its own
    HIP events on `stream`) after `warmup` untimed ones."""
    g = pre.graph(ddet, flips, res)
    for _ in range(warmup):
        g.launch(stream=stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record(stream)
    for k in range(n):
        g.launch(stream=stream)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    g.close()
    ms = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(n)])
    return {"replays": n, "warmup": warmup, "median_ms": float(np.median(ms)),
            "p10_ms": float(np.percentile(ms, 10)), "p90_ms": float(np.percentile(ms, 90)),
            "min_ms": float(ms.min()), "max_ms": float(ms.max())}


def flops_per_sample(layers, H, T):
    """Conv FLOPs per sample on a T x H x H grid (H = d + 1, or d in the paper's layout)."""
    V = T * H ** 2
    return sum(2 * ci * co * k ** 3 for (ci, co, k, _a) in layers) * V


def bench_model6(args, torch, pdx, workload):
    """Model 6 (Sec. VI, Fig. Model8Representation: four residual blocks, 512
    channels, BatchNorm folded at create) in the paper's layout at d = T =
    --d, batch --batch, bf16 (or --dtype fp8: E4M3) with fp32 accumulation."""
    d = T = args.d or 13
    B = args.batch or 1
    dtype = args.dtype or "bf16"
    fp8 = dtype == "fp8"
    peak = PEAK_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS
    blocks = workload.MODEL6_BLOCKS
    weights = workload.resnet_weights(blocks, 4006)
    det, _ = workload.make_inputs(d, T, B, 0.003, 0.003, 5000 + d)
    torch.cuda.set_device(0)
    pre = pdx.Predecoder(weights, d, T, None, dtype, max_batch=B, layout="paper", first="Z", last="Z",
                         blocks=blocks)
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    flips = torch.empty((B, pre.flip_words), dtype=torch.int64, device="cuda")
    res = torch.empty((B, pre.det_words), dtype=torch.int64, device="cuda")
    cur = torch.cuda.current_stream()
    for _ in range(args.warmup):
        pre.run(ddet, flips, res, stream=cur)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(cur)
    for _ in range(args.steps):
        pre.run(ddet, flips, res, stream=cur)
    e1.record(cur)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    stages = pre.stage_times(ddet, flips, res, args.stage_iters, stream=cur)
    pre.close()
    V = T * d * d

    def block_flops(b):
        ci, cm, co, _ = b
        return 2.0 * V * (27 * ci * cm + 27 * cm * co + (ci * co if ci != co else 0))
    total = sum(block_flops(b) for b in blocks) * B
    mid = block_flops(blocks[1]) * B  # block 2: two 512 -> 512 convolutions
    achieved = mid / (stages[2] * 1e-3) / 1e12
    out = {
        "metric": "us/round (pre-decode+residual), Model 6 (residual network) in the paper's layout at d=T=%d" % d,
        "value": ms * 1e3 / (B * T), "unit": "us/round", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "rounds_per_s": B * T / (ms * 1e-3), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8-e4m3" if fp8 else "bf16",
        "data": "synthetic (seeded phenomenological noise p=q=0.003, He-normal convs, random BatchNorm statistics)",
        "config": {"workload": "Model 6 of Sec. VI (blocks %s, BatchNorm folded), paper layout, d=T=%d, batch %d; "
                               "%s / fp32 accumulate" % (blocks, d, B, "E4M3" if fp8 else "bf16"),
                   "d": d, "T": T, "batch": B, "model": 6},
        "mfma_frac_end_to_end": total / (ms * 1e-3) / (peak * 1e12),
        "stage_ms": {"unpack": stages[0], **{"block%d" % (k + 1): stages[1 + k] for k in range(len(blocks))},
                     "residual_repack": stages[-1]},
        "roofline": {"kernel": "block 2: two conv3d 3x3x3 512->512 (%s MFMA, four 128-channel output slices in one launch each)"
                               % ("fp8" if fp8 else "bf16"),
                     "bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None},
    }
    print(json.dumps(out), flush=True)


def bench_stream(args, torch, pdx, workload):
    """The temporal window driver (Sec. VI, parallel windows in time): a model
    of Table models over --stream rounds at distance --d, --batch streams,
    windows of d x d x 3d (core d, buffer d), everything on one GPU."""
    d, n, B = args.d or 13, args.stream, args.batch or 1
    core, buf = args.core or d, d if args.buffer is None else args.buffer
    dtype = args.dtype or "bf16"
    layers = workload.paper_model_layers(args.paper_model)
    weights = workload.he_normal_weights(layers, 4000 + args.paper_model)
    det, _ = workload.make_inputs(d, n, B, 0.003, 0.003, 6000 + d)
    torch.cuda.set_device(0)
    s = pdx.Stream(weights, d, n, layers, core, buf, dtype, n_streams=B, layout="paper", first="Z", last="Z")
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    flips = torch.empty((B, s.flip_words), dtype=torch.int64, device="cuda")
    res = torch.empty((B, s.det_words), dtype=torch.int64, device="cuda")
    cur = torch.cuda.current_stream()
    for _ in range(args.warmup):
        s.run(ddet, flips, res, stream=cur)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(cur)
    for _ in range(args.steps):
        s.run(ddet, flips, res, stream=cur)
    e1.record(cur)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    s.close()
    plan = pdx.stream_windows(n, core, buf)
    nwin = len(plan)
    h = sum((k - 1) // 2 for (_, _, k, _) in layers)  # receptive-field half-width: buffer >= h is exact
    # Table Time_Like_Parallel_Table (GB300, FP8, one GPU per d x d x 3d block
    # or `batch` blocks per GPU): us/round for 1000 rounds -- context only
    ctx = {(1, 13, 1): 0.11, (1, 13, 2): 0.13, (1, 13, 4): 0.179, (1, 21, 1): 0.179, (1, 21, 2): 0.244,
           (1, 21, 4): 0.423, (4, 13, 1): 0.138, (4, 13, 2): 0.211, (4, 13, 4): 0.282, (4, 21, 1): 0.231,
           (4, 21, 2): 0.324, (4, 21, 4): 0.551}
    out = {
        "metric": "us/round over a %d-round stream, temporal windows (Table models Model %d, paper layout, d=%d)"
                  % (n, args.paper_model, d),
        "value": ms * 1e3 / n, "unit": "us/round", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp8": "fp8-e4m3"}[dtype],
        "data": "synthetic (seeded phenomenological noise p=q=0.003, He-normal random weights)",
        "config": {"workload": "%d stream(s) of %d rounds at d=%d, Model %d (%s); %d windows per stream (core %d, "
                               "buffer %d rounds; exact for buffer >= %d), all run on one GPU as one batch per "
                               "window length" % (B, n, d, args.paper_model, layers, nwin, core, buf, h),
                   "d": d, "rounds": n, "streams": B, "model": args.paper_model, "windows_per_stream": nwin,
                   "core": core, "buffer": buf, "computed_rounds_per_stream": sum(w[1] for w in plan)},
        "us_per_round_per_stream": ms * 1e3 / n / B,
        "paper_context_us_per_round": ctx.get((args.paper_model, d, B)) if (core, buf) == (d, d) else None,
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="workload id (1..5)")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--stage-iters", type=int, default=5)
    ap.add_argument("--cpu-samples", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (calibrates HBM byte counters)")
    ap.add_argument("--paper-model", type=int, default=None,
                    help="time a model of Table models (1 to 5; 6: the residual network) in the paper's own layout "
                         "(D x D grid, four input channels, 3x3x3 (Model 3: 5x5x5) output layer) at d = T = --d "
                         "instead of a workload")
    ap.add_argument("--d", type=int, default=None,
                    help="distance and rounds d = T: for --paper-model (default 13), or to run a workload's "
                         "network and noise at another distance (a sweep over d)")
    ap.add_argument("--stream", type=int, default=None,
                    help="with --paper-model: time the temporal window driver over a stream of this many rounds "
                         "(windows of d x d x 3d rounds: core d, buffer d), --batch streams at once")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of a recorded run (HIP graph) instead of predecoder_run calls")
    ap.add_argument("--core", type=int, default=None, help="--stream: committed rounds per window (default d)")
    ap.add_argument("--buffer", type=int, default=None, help="--stream: rounds read on each side (default d)")
    ap.add_argument("--replays", type=int, default=100,
                    help="recorded-run (HIP graph) replays timed one by one for the median / p10 / p90 (0: skip)")
    ap.add_argument("--replay-warmup", type=int, default=200, help="untimed replays before them")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured MFMA / HBM ceilings")
    ap.add_argument("--peaks", action="store_true",
                    help="only measure the MFMA and HBM ceilings of this device and print them")
    ap.add_argument("--dtype", choices=["bf16", "fp8"], default=None,
                    help="operand precision (default: the workload's, bf16 for the benchmark workload); fp8 = "
                         "E4M3 weights and activations with fp32 accumulation, the paper's deployment precision")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the path is data-parallel over independent volumes and "
              "this build runs on a single MI355X; --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2604_12841_amd as pdx
    from paper_2604_12841_amd import workload

    if args.peaks:
        torch.cuda.set_device(0)
        pk = measure_peaks(torch, pdx, torch.cuda.current_stream())
        print(json.dumps({"metric": "measured MI355X ceilings", "measured_peaks": pk,
                          "published": {"mfma_bf16_tflops": PEAK_BF16_TFLOPS, "mfma_fp8_tflops": PEAK_FP8_TFLOPS,
                                        "hbm_gbs": PEAK_HBM_GBS}}), flush=True)
        return
    paper = args.paper_model is not None
    if args.paper_model == 6:
        return bench_model6(args, torch, pdx, workload)
    if args.stream is not None:
        if not paper:
            print("--stream needs --paper-model", file=sys.stderr)
            sys.exit(2)
        return bench_stream(args, torch, pdx, workload)
    if paper:
        # Table models in the paper's layout: memory experiment in the Z basis
        # (x_present cleared in the first and last round), d = T
        d = T = args.d or 13
        B = args.batch or 1
        layers = workload.paper_model_layers(args.paper_model)
        weights = workload.he_normal_weights(layers, 4000 + args.paper_model)
        det, _ = workload.make_inputs(d, T, B, 0.003, 0.003, 5000 + d)
        cfg = dict(dtype=args.dtype or "bf16", p=0.003, n_hidden=len(layers) - 1, width=layers[0][1])
        grid = d
    else:
        cfg = workload.CONFIGS[args.workload]
        if args.d:
            cfg = dict(cfg, d=args.d, T=args.d)
        d, T = cfg["d"], cfg["T"]
        B = args.batch or cfg["batch"]
        layers = workload.config_layers(args.workload)
        weights = workload.config_weights(args.workload)
        det, _ = workload.make_inputs(d, T, B, cfg["p"], cfg["q"], 2000 + args.workload)
        grid = d + 1
        if args.dtype:
            if cfg["dtype"] == "fp32":
                print("--dtype applies to the bf16 workloads", file=sys.stderr)
                sys.exit(2)
            cfg = dict(cfg, dtype=args.dtype)
    fp8 = cfg["dtype"] == "fp8"
    peak = PEAK_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS

    torch.cuda.set_device(0)
    if paper:
        pre = pdx.Predecoder(weights, d, T, layers, cfg["dtype"], max_batch=B, layout="paper", first="Z", last="Z")
    else:
        pre = pdx.Predecoder(weights, d, T, layers, cfg["dtype"], max_batch=B)
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    flips = torch.empty((B, pre.flip_words), dtype=torch.int64, device="cuda")
    res = torch.empty((B, pre.det_words), dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream()

    graph = pre.graph(ddet, flips, res) if args.graph else None
    step = (lambda: graph.launch(stream=stream)) if graph else (lambda: pre.run(ddet, flips, res, stream=stream))
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print("step %.3f ms" % ms, file=sys.stderr, flush=True)
    if graph:
        graph.close()

    # Per-stage HIP-event times on the same stream (unpack, each layer, head, residual).
    stages = pre.stage_times(ddet, flips, res, args.stage_iters, stream=stream)
    # the paper's protocol: replays of a recorded run, each timed (median, p10, p90)
    replays = graph_replays(torch, pre, ddet, flips, res, stream, args.replays, args.replay_warmup) \
        if args.replays > 0 else None
    if replays:
        print("graph replays: median %.3f ms (p10 %.3f, p90 %.3f)" % (replays["median_ms"], replays["p10_ms"],
                                                                      replays["p90_ms"]), file=sys.stderr, flush=True)
    n = len(layers)
    # hidden C->C layers whose epilogue writes activations (with a 1x1x1 head
    # the last hidden layer also applies the head and is timed separately in
    # stage_ms; a 3x3x3 output layer is a stage of its own)
    last_hidden = n - 1 if layers[-1][2] == 3 else n - 2
    hidden = [i for i in range(1, last_hidden) if layers[i][0] == layers[i][1]]
    conv_ms = float(np.mean([stages[1 + i] for i in hidden]))
    ci, co, kk = layers[hidden[0]][0], layers[hidden[0]][1], layers[hidden[0]][2]
    V = T * grid ** 2
    conv_flops = 2.0 * ci * co * kk ** 3 * V * B
    achieved = conv_flops / (conv_ms * 1e-3) / 1e12
    print("stages ms:", ["%.3f" % s for s in stages], file=sys.stderr, flush=True)

    total_flops = flops_per_sample(layers, grid, T) * B
    in_bytes = layers[0][0] * (4 if cfg["dtype"] == "fp32" else 2)  # input planes: c_in channels, bf16 or fp32
    rounds = B * T
    out = {
        "metric": "syndrome rounds/sec and us/round (pre-decode+residual) at d=13,T=13; MFMA %",
        "value": rounds / (ms * 1e-3),
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "us_per_round": ms * 1e3 / rounds,
        "mfma_frac_end_to_end": total_flops / (ms * 1e-3) / (peak * 1e12),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp8": "fp8-e4m3", "fp32": "f32"}[cfg["dtype"]],
        "data": "synthetic (seeded phenomenological noise, He-normal random weights)",
        "timed": "HIP graph replays of predecoder_run" if args.graph else "predecoder_run calls",
        "config": {
            "workload": "rotated surface code d=%d, T=%d rounds, batch %d; %d conv3d 3x3x3 layers x %d "
                        "channels + 1x1x1 head, %s operands / fp32 accumulate; p=q=%g"
                        % (d, T, B, cfg["n_hidden"], cfg["width"], cfg["dtype"], cfg["p"]),
            "d": d, "T": T, "batch": B, "layers": cfg["n_hidden"], "width": cfg["width"],
        },
        "stage_ms": {"unpack": stages[0],
                     **{"layer%d" % (i + 1): stages[1 + i] for i in range(n - 1)},
                     "head_threshold": stages[n], "residual_repack": stages[n + 1]},
        # algorithmic HBM bytes of the two bit-moving stages / their event
        # times: unpack reads the packed detectors and writes the interior
        # input planes; residual+repack reads the flip nibbles (one byte per
        # voxel) and the detectors and writes the packed flip and residual rows
        "stage_gbs": {
            "unpack": B * (pre.det_words * 8 + V * in_bytes) / (stages[0] * 1e-3) / 1e9,
            "residual_repack": B * (V + pre.det_words * 16 + pre.flip_words * 8) / (stages[n + 1] * 1e-3) / 1e9,
        },
        "graph_replays": None if replays is None else dict(
            replays, rounds_per_s_median=rounds / (replays["median_ms"] * 1e-3),
            us_per_round_median=replays["median_ms"] * 1e3 / rounds,
            us_per_round_latency_median=replays["median_ms"] * 1e3 / T),
        "roofline": {
            "kernel": "conv3d %dx%dx%d %d->%d implicit GEMM (%s MFMA) + bias/GELU epilogue"
                      % (kk, kk, kk, ci, co, "fp8 e4m3" if fp8 else "bf16"),
            "bound": "mfma",
            "achieved": achieved,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": achieved / peak,
            "traffic": counted_traffic("conv_hidden_%dx%d_d%d_T%d_B%d%s_counters.md"
                                       % (ci, co, d, T, B, "_fp8" if fp8 else "")),
        },
    }

    if not args.no_peaks:
        pk = measure_peaks(torch, pdx, stream)
        mp = pk["mfma_%s_random_tflops" % ("fp8" if fp8 else "bf16")]
        out["measured_peaks"] = pk
        out["roofline"].update(measured_peak=mp, frac_of_measured=achieved / mp)
        out["mfma_frac_end_to_end_of_measured"] = total_flops / (ms * 1e-3) / (mp * 1e12)
        print("measured peaks:", {k: round(v, 1) for k, v in pk.items() if k != "how"}, file=sys.stderr, flush=True)

    if paper:
        # the paper times Table models at batch 1 (Table runtimes, GB300, FP8,
        # TensorRT): 13^3 / 21^3 / 31^3 = 2.397 / 1.872 / 2.609 us/round for
        # Model 1, 3.252 / 2.703 / 3.774 for Model 4 and 4.364 / 5.056 / 9.263
        # for Model 5 -- another machine and precision, context only
        ctx = {1: {13: 2.397, 21: 1.872, 31: 2.609}, 4: {13: 3.252, 21: 2.703, 31: 3.774},
               5: {13: 4.364, 21: 5.056, 31: 9.263}}
        out.update({
            "metric": "us/round (pre-decode+residual), Table models Model %d in the paper's layout at d=T=%d"
                      % (args.paper_model, d),
            "value": ms * 1e3 / rounds,
            "unit": "us/round",
            "higher_is_better": False,
            "rounds_per_s": rounds / (ms * 1e-3),
            "config": {"workload": "Model %d of Table models (%s), paper layout: D x D grid, 4 input channels, "
                                   "3x3x3 output layer; d=T=%d, batch %d; %s / fp32 accumulate; p=q=0.003"
                                   % (args.paper_model, layers, d, B, cfg["dtype"]),
                       "d": d, "T": T, "batch": B, "model": args.paper_model},
            "paper_context_us_per_round": ctx.get(args.paper_model, {}).get(d),
        })
        out["roofline"]["traffic"] = None
        out["stage_ms"] = {"unpack": stages[0], **{"layer%d" % (i + 1): stages[1 + i] for i in range(n)},
                           "residual_repack": stages[n + 1]}
        pre.close()
        print(json.dumps(out), flush=True)
        return

    if not args.no_cpu_baseline:
        # the oracle on a bounded sample of the same workload, built for this
        # host (-march=native), with all its threads and with one; and the
        # parity of the GPU's outputs for those samples (the timed launch
        # configuration: the whole batch, logits kept) against it
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from parity import compare
        ns = args.cpu_samples or {1: 64, 2: 128, 3: 48, 4: 1, 5: 4}[args.workload]
        ns = min(ns, B)
        oracle.use_native()
        oracle.unpack(d, T, det[:1])  # load the library outside the timed region
        bf16 = cfg["dtype"] == "bf16"
        t0 = time.perf_counter()
        ref = oracle.run(d, T, det[:ns], layers, weights, bf16=bf16, fp8=fp8)
        dt = time.perf_counter() - t0
        cores = oracle.num_threads()
        n1 = max(1, min(ns, int(round(ns / cores))))
        oracle.set_num_threads(1)
        t0 = time.perf_counter()
        oracle.run(d, T, det[:n1], layers, weights, bf16=bf16, fp8=fp8)
        dt1 = time.perf_counter() - t0
        oracle.set_num_threads(cores)
        out["cpu_baseline"] = {
            "value": ns * T / dt, "unit": "rounds/s", "cores": cores, "kind": "oracle",
            "sample": "%d of the %d samples (%.1f s, fp64 oracle with %s rounding points, gcc -O3 -march=native, "
                      "OpenMP over samples x output channels, %d host CPUs visible)"
                      % (ns, B, dt, cfg["dtype"], len(os.sched_getaffinity(0))),
            "single_thread": {"value": n1 * T / dt1, "unit": "rounds/s", "cores": 1,
                              "sample": "%d of the %d samples (%.1f s)" % (n1, B, dt1)},
        }
        logits = torch.empty((B, 4, T, grid, grid), dtype=torch.float32, device="cuda")
        pre.run(ddet, flips, res, logits, stream=stream)
        torch.cuda.synchronize()
        u64 = lambda t: t[:ns].cpu().numpy().view(np.uint64)
        st = compare(d, T, cfg["dtype"], *ref, u64(flips), u64(res), logits[:ns].cpu().numpy())
        out["parity"] = dict(st, samples=ns, rule="logits within the dtype's bound; flips and residual bit-exact "
                                                  "outside sites whose oracle |logit| <= it")
        del logits
    pre.close()
    if args.copy_mib:
        # a plain device copy of known size (HBM byte-counter calibration)
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        pdx.peak_copy(src, dst, n, stream=stream)
        torch.cuda.synchronize()
        out["copy_calibration_mib"] = args.copy_mib
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
