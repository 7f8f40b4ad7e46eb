"""Benchmark of the HIGGS inference hot path on one MI355X.

Default workload: the seven linear layers of Llama-3.1-8B (q, k, v, o, gate,
up, down), weights drawn as Student-t(5) at std 0.02 with 0.1% outlier input
columns, bf16, quantized on the GPU with the (p=2, n=256) grid (4 bits per
weight), g = 1024, one rotation seed per layer. One step = for every layer,
the output y = x W_hat^T of one bf16 activation row (batch 1): the activation
rotation and the lookup-table product in one launch. The timed steps rotate
over enough copies of the codes and scales (>= 1 GiB) that the 256 MB
Infinity Cache cannot hold them, so the codes stream from HBM. Timed launches
are replayed from HIP graphs, so host-side launch cost does not enter the
GPU time.

Printed: one JSON line with the headline figure (whole-step HBM GB/s over the
algorithmic bytes), the roofline of the dominant kernel (the batch-1 product),
the oracle timed on the host cores, and extra per-layer / per-batch figures
(among them the same layers as dense bf16 weights through hipBLASLt, as a
reference point measured on the same GPU).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
METRIC = "HIGGS qmatmul µs/layer and achieved HBM GB/s (bs=1), TFLOP/s (bs=64), 8B shapes"
G = 1024


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "qgemv_llama8b_bs1_traffic.json")
TRAFFIC_FILE_BS64 = os.path.join(ROOT, "profiles", "qgemm_llama8b_bs64_traffic.json")
PROBE_LIB = os.path.join(ROOT, "paper_2411_17525_amd", "libhiggs_bench.so")


def measured_traffic(path=TRAFFIC_FILE):
    """HBM bytes of one step (one launch per layer) from the committed
    FETCH_SIZE / WRITE_SIZE counter runs, scaled by the counters of a copy of
    known size; None when the kernel sources changed since they were taken."""
    import hashlib
    try:
        rec = json.load(open(path))
        h = hashlib.sha256()
        for f in rec["sources"]:
            h.update(open(os.path.join(ROOT, f), "rb").read())
    except (OSError, ValueError, KeyError):
        return None
    return rec["step_hbm_bytes"] if h.hexdigest() == rec["source_sha256"] else None


def stream_ceiling(dev, flush, sizes):
    """The memory ceiling per launch size: launch-to-launch time of a plain
    streaming read (libhiggs_bench.so) of `nbytes`, one launch on each of
    several distinct slices of a 2 GiB buffer, replayed from a graph after a
    cache flush, exactly as the product launches are timed. Returns
    {nbytes: GB/s}."""
    import ctypes
    import torch
    lib = ctypes.CDLL(PROBE_LIB)
    lib.higgs_bench_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                            ctypes.c_void_p]
    lib.higgs_bench_stream_read.restype = ctypes.c_int
    total = 2 << 30
    buf = torch.ones(total // 4, dtype=torch.float32, device=dev)
    sink = torch.zeros(64, dtype=torch.int32, device=dev)
    out = {}
    for nbytes in sizes:
        nbytes = nbytes // 256 * 256
        count = max(1, min(16, total // nbytes))

        def one(i, nbytes=nbytes):
            st = torch.cuda.current_stream().cuda_stream
            rc = lib.higgs_bench_stream_read(ctypes.c_void_p(buf.data_ptr() + i * nbytes), nbytes,
                                             ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(st))
            if rc != 0:
                raise RuntimeError(f"stream read probe failed ({rc})")
        us = graph_train_us(one, count, flush)
        out[nbytes] = nbytes / (us * 1e-6) / 1e9
    del buf
    return out


def ceiling_for(ceil, nbytes):
    return ceil[nbytes // 256 * 256]


def graph_train_us(fn, count, flush, replays=3):
    """Launch-to-launch time in µs of fn(0), ..., fn(count - 1) captured in one
    HIP graph: the mean over `replays` replays, each preceded (outside the
    timed region) by a read of `flush`, a buffer four times the 256 MB
    Infinity Cache. fn(i) reads the i-th of `count` distinct copies of its
    codes, so every timed launch streams its codes from HBM."""
    import torch
    stream = torch.cuda.current_stream()
    for i in range(count):
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(count):
            fn(i)
    g.replay()  # the first replay uploads the graph; untimed
    total = 0.0
    for _ in range(replays):
        flush.sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        total += e0.elapsed_time(e1)
    return total * 1e3 / (replays * count)


# Layers of a Llama block that read the same activations (indices into the
# seven 8B layers): the q, k and v projections, o, gate and up, down.
GROUPS = (("qkv", (0, 1, 2)), ("o", (3,)), ("gate_up", (4, 5)), ("down", (6,)))


def group_bytes(batch, shapes, p, n, g):
    """Algorithmic HBM bytes of layers that read one activation tensor:
    codes + fp16 scales + fp32 outputs of each, the bf16 activations once.
    shapes: [(out, in)] with a common in."""
    inp = shapes[0][1]
    return sum(qmm_bytes(batch, o, inp, p, n, g) - 2 * batch * inp for o, _ in shapes) \
        + 2 * batch * inp


def qmm_bytes(batch, out, inp, p, n, g):
    """Algorithmic HBM bytes of one layer's output from its activations: codes +
    fp16 scales + bf16 activations + fp32 output."""
    bits = int(round(math.log2(n)))
    return out * inp * bits // (8 * p) + 2 * out * (inp // g) + 2 * batch * inp + 4 * batch * out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-extra", action="store_true", help="headline line only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--profile-pass", action="store_true",
                    help="counter pass for a profiler: random codes of the same layers, three "
                         "products per layer group at --profile-batch rows, then a 64 MiB "
                         "elementwise copy of known traffic for calibration; prints nothing on "
                         "stdout")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="CPU only: HBM traffic per layer group from the rocprofv3 "
                         "counter_collection.csv files of a FETCH_SIZE and a WRITE_SIZE run of "
                         "--profile-pass at --profile-batch rows; writes the profiles/ traffic "
                         "record that the bench line reports")
    ap.add_argument("--summarize-trace", metavar="TRACE_CSV",
                    help="CPU only: per kernel and launch shape dispatch durations from a "
                         "rocprofv3 kernel_trace.csv, as a markdown table")
    ap.add_argument("--summarize-stats", metavar="STATS_CSV",
                    help="CPU only: every kernel of a whole run from a rocprofv3 "
                         "kernel_stats.csv (calls, mean / min / max / total time), as markdown")
    ap.add_argument("--profile-batch", type=int, default=1,
                    help="batch rows of the --profile-pass products (default 1)")
    ap.add_argument("--stamp-pass", action="store_true",
                    help="phase times of the batch-1 product launches from the phase-stamp "
                         "build of the library (libhiggs_stamps.so): per launch group, the "
                         "median over waves of each phase, as a markdown table")
    ap.add_argument("--encode-profile", action="store_true",
                    help="encoder pass for a profiler: per code format the search index built "
                         "seven times, then the seven 8B layer shapes encoded six times each "
                         "(and the (2,256) gate layer six times without an index); prints the "
                         "event-timed figures")
    ap.add_argument("--summarize-encode-trace", metavar="TRACE_CSV",
                    help="CPU only: the encoder table of profiles/quantize_llama8b.md from the "
                         "rocprofv3 kernel_trace.csv of an --encode-profile run")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_stats:
        summarize_stats(args.summarize_stats)
        return
    if args.summarize_encode_trace:
        summarize_encode_trace(args.summarize_encode_trace)
        return
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters, args.profile_batch,
                           TRAFFIC_FILE if args.profile_batch == 1 else
                           TRAFFIC_FILE_BS64 if args.profile_batch == 64 else
                           os.path.join(ROOT, "profiles",
                                        f"qgemm_llama8b_bs{args.profile_batch}_traffic.json"))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1 "
                          "(the path is single-GPU; multi-GPU sharding is a design note)"}))
        sys.exit(2)

    if args.stamp_pass:  # the debug build with the product kernel's phase stamps
        os.environ["HIGGS_LIB"] = os.path.join(ROOT, "paper_2411_17525_amd", "libhiggs_stamps.so")
    import torch
    from paper_2411_17525_amd import higgs as H
    from paper_2411_17525_amd import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    H.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    p, n = 2, 256
    if args.profile_pass:
        profile_pass(H, synth, dev, p, n, args.profile_batch)
        return
    if args.encode_profile:
        encode_profile(H, synth, dev)
        return
    if args.stamp_pass:
        stamp_pass(H, synth, dev, p, n)
        return
    t0 = time.time()
    grid_np, grid_mse, grid_iters = H.make_grid(p, n, 0, 1 << 20, 300)
    log(f"grid (2,256) from 2^20 samples: mse/dim={grid_mse:.6g} iters={grid_iters} "
        f"({time.time() - t0:.1f} s)")
    grid = torch.from_numpy(grid_np).to(dev)
    # the grid's search index: built once, used for every layer
    H.search_index(grid)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    gindex = H.search_index(grid)
    e1.record(stream)
    torch.cuda.synchronize()
    index_ms = e0.elapsed_time(e1)

    # ---- encode the seven 8B layers on the GPU (also timed: encode throughput) ----
    layers = []
    enc_ms = 0.0
    total_w = 0
    # options of the variable-bitwidth problem (Sec. 4): (p, n) with their grids
    dyn_opts = []
    if not args.no_extra:
        for fp, fn in [(2, 64), (1, 16), (2, 256), (2, 1024), (1, 256)]:
            fgrid = H.make_uniform_grid(fn)[0] if (fp, fn) == (1, 256) else \
                H.make_grid(fp, fn, 0, 1 << 18, 100)[0]
            fg = torch.from_numpy(fgrid).to(dev)
            dyn_opts.append((fp, fn, fg, H.search_index(fg)))
    dyn_t2, dyn_ms = [], 0.0
    for li, (name, out, inp) in enumerate(synth.LLAMA8B_LAYERS):
        wt = synth.student_t_weight(out, inp, seed=2000 + li, dtype="bf16")
        w_dev = torch.from_numpy(wt.bits.view(np.int16)).to(dev).view(torch.bfloat16)
        del wt
        H.quantize(w_dev, grid, G, li, index=gindex)          # warm-up of this shape
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        codes, scales = H.quantize(w_dev, grid, G, li, index=gindex)
        e1.record(stream)
        torch.cuda.synchronize()
        enc_ms += e0.elapsed_time(e1)
        total_w += out * inp
        # the layer's error under every option: quantize + error kernel (timed)
        row = []
        for fp, fn, fgrid, findex in dyn_opts:
            e0.record(stream)
            c2, s2 = H.quantize(w_dev, fgrid, G, li, index=findex)
            ge = torch.empty((out * (inp // G), 2), dtype=torch.float64, device=dev)
            t2d = torch.empty(1, dtype=torch.float64, device=dev)
            H.lib().higgs_layer_error(H._ptr(w_dev), 1, out, inp, H._ptr(c2), H._ptr(s2),
                                      H._ptr(fgrid), fp, fn, G, li, H._ptr(ge), H._ptr(t2d),
                                      H._stream(None))
            e1.record(stream)
            torch.cuda.synchronize()
            dyn_ms += e0.elapsed_time(e1)
            row.append(float(t2d.item()))
            del c2, s2, ge, t2d
        if dyn_opts:
            dyn_t2.append(row)
        del w_dev
        layers.append({"name": name, "out": out, "in": inp, "seed": li,
                       "codes": codes, "scales": scales})
    log(f"encoded {total_w} weights in {enc_ms:.2f} ms of kernel time")

    # ---- copies of the codes so the timed loop streams >= 1 GiB ----
    set_bytes = sum(L["codes"].numel() + 2 * L["scales"].numel() for L in layers)
    ncopies = max(16, math.ceil((1 << 30) / set_bytes))
    copies = [[(L["codes"], L["scales"]) for L in layers]]
    for _ in range(ncopies - 1):
        copies.append([(c.clone(), s.clone()) for c, s in copies[0]])
    log(f"{ncopies} copies of {set_bytes / 1e6:.1f} MB of codes + scales")
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)  # 1 GiB

    def make_io(batch):
        xs, ys = [], []
        for li, L in enumerate(layers):
            act = synth.activations(batch, L["in"], seed=2000 + li + 500 + batch)
            xs.append(torch.from_numpy(act.bits.view(np.int16)).to(dev).view(torch.bfloat16))
            ys.append(torch.empty((batch, L["out"]), dtype=torch.float32, device=dev))
        ws_bytes = max([H.qmatmul_fused_workspace_bytes(batch, L["out"], L["in"], p, n, G)
                        for L in layers] +
                       [H.qmatmul_fused_multi_workspace_bytes(
                           batch, [layers[li]["out"] for li in idx], layers[idx[0]]["in"], p, n,
                           G) for _, idx in GROUPS])
        ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
        return xs, ys, ws

    def run_group(io, copy, idx):
        """The outputs of the layers idx, which read the activations of the
        first of them: one launch (the multi-layer call for several)."""
        xs, ys, ws = io
        if len(idx) == 1:
            li = idx[0]
            c, s = copies[copy][li]
            H.qmatmul_fused(xs[li], c, s, grid, G, layers[li]["seed"], layers[li]["out"],
                            y=ys[li], workspace=ws)
        else:
            H.qmatmul_fused_multi(xs[idx[0]], [(*copies[copy][li], layers[li]["seed"],
                                                layers[li]["out"]) for li in idx],
                                  grid, G, ys=[ys[li] for li in idx], workspace=ws)

    def step(io, copy):
        """One pass of the hot path: the output of every layer of the block,
        one launch per group of layers that share their input."""
        for _, idx in GROUPS:
            run_group(io, copy, idx)

    def graph_of(fn):
        """fn's launches captured into a HIP graph (replays skip the host
        launch path, so the timing is the GPU's)."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        return g

    def timed(batch, steps, warmup):
        """`warmup` untimed steps, then exactly `steps` back-to-back steps
        (copies of the codes in turn) replayed from one graph between one
        event pair; returns ms per step."""
        io = make_io(batch)
        for i in range(warmup):
            step(io, i % ncopies)
        torch.cuda.synchronize()
        g = graph_of(lambda: [step(io, (warmup + i) % ncopies) for i in range(steps)])
        g.replay()  # first replay uploads the graph; untimed
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        g.replay()
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps

    def layer_us(batch):
        """Per-layer launch time: one layer's product launched once on each
        copy of its codes, replayed from a graph after a cache flush."""
        xs, ys, ws = make_io(batch)
        out = {}
        for li, L in enumerate(layers):
            def one(i, li=li, L=L):
                c, s = copies[i][li]
                H.qmatmul_fused(xs[li], c, s, grid, G, L["seed"], L["out"], y=ys[li],
                                workspace=ws)
            out[L["name"]] = graph_train_us(one, ncopies, flush)
        return out

    def step_bytes_of(batch):
        return sum(group_bytes(batch, [(layers[li]["out"], layers[li]["in"]) for li in idx],
                               p, n, G) for _, idx in GROUPS)

    def group_us(batch):
        """Launch time of each group of layers sharing an input (one launch),
        one launch on each copy of the codes, after a cache flush."""
        io = make_io(batch)
        return {name: graph_train_us(lambda i, idx=idx: run_group(io, i, idx), ncopies, flush)
                for name, idx in GROUPS}

    # ---- headline: batch 1 ----
    batch = 1
    ms_per_step = timed(batch, args.steps, args.warmup)
    step_bytes = step_bytes_of(batch)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    per_layer_us = layer_us(batch)
    groups_us = group_us(batch)
    # the memory ceiling at each launch's size: a plain streaming read of the
    # same number of bytes in one launch, timed like the products
    gbytes = {name: group_bytes(batch, [(layers[li]["out"], layers[li]["in"]) for li in idx],
                                p, n, G) for name, idx in GROUPS}
    ceil = stream_ceiling(dev, flush, sorted(set(gbytes.values())) + [1 << 30])
    ceiling_step_us = sum(b / (ceiling_for(ceil, b) * 1e9) * 1e6 for b in gbytes.values())
    # the timed region holds only the product kernel's launches (four per
    # step): algorithmic bytes per launch / average launch time over it
    achieved = step_bytes / (ms_per_step * 1e-3) / 1e9
    per_layer = {L["name"]: {"us": round(per_layer_us[L["name"]], 3),
                             "GBps": round(qmm_bytes(batch, L["out"], L["in"], p, n, G)
                                           / (per_layer_us[L["name"]] * 1e-6) / 1e9, 1)}
                 for L in layers}
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "llama3.1-8b-7-linear-layers-higgs-p2n256-g1024-batch1",
                   "layers": [f"{L['name']}:{L['out']}x{L['in']}" for L in layers],
                   "batch": batch, "grid": [p, n], "g": G,
                   "hbm_rotation_copies": ncopies,
                   "step": "per group of layers sharing an input (q/k/v, o, gate/up, down): "
                           "activation rotation + LUT product, one launch per group"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(), "algorithmic_bytes": step_bytes,
                     "kernel": "qgemv_kernel (batch 1, fused rotation), 4 launches per step "
                               "covering the 7 layer shapes: algorithmic bytes of a step / step "
                               "time over the timed region (launch to launch)",
                     "measured_ceiling_GBps": round(step_bytes / (ceiling_step_us * 1e-6) / 1e9, 1),
                     "frac_of_measured_ceiling": round(achieved / (step_bytes / (ceiling_step_us
                                                                             * 1e-6) / 1e9), 4),
                     "measured_ceiling": "a plain streaming-read kernel (libhiggs_bench.so) "
                                         "reading each launch's algorithmic bytes in one "
                                         "launch, timed the same way (graph replay, cold "
                                         "HBM): the step's bytes over the sum of those times"},
        "hbm_stream_read_GBps": {str(b): round(v, 1) for b, v in sorted(ceil.items())},
        "per_layer_bs1": per_layer,
        "groups_bs1": {name: {"us": round(groups_us[name], 3),
                              "GBps": round(group_bytes(batch, [(layers[li]["out"], layers[li]["in"])
                                                               for li in idx], p, n, G)
                                            / (groups_us[name] * 1e-6) / 1e9, 1)}
                       for name, idx in GROUPS},
    }

    extra = {}
    if not args.no_extra:
        extra["encode"] = {"weights": total_w, "kernel_ms": round(enc_ms, 3),
                           "weights_per_s": total_w / (enc_ms * 1e-3),
                           "search_index_ms": round(index_ms, 4),
                           "note": "per-layer quantize calls with the grid's search index, "
                                   "built once per grid (search_index_ms, not included)"}
        extra["grid"] = {"mse_per_dim": grid_mse, "iters": grid_iters}
        for b in (4, 16, 32, 64):
            ms = timed(b, max(20, args.steps // 4), 5)
            lus = layer_us(b)
            flops = sum(2 * b * L["out"] * L["in"] for L in layers)
            byts = sum(qmm_bytes(b, L["out"], L["in"], p, n, G) for L in layers)
            step_b = step_bytes_of(b)
            ksum = sum(lus.values())
            extra[f"batch{b}"] = {"ms_per_step": round(ms, 5),
                                  "step_GBps": round(step_b / (ms * 1e-3) / 1e9, 1),
                                  "step_TFLOPs": round(flops / (ms * 1e-3) / 1e12, 2),
                                  "layers_us_sum": round(ksum, 2),
                                  "GBps": round(byts / (ksum * 1e-6) / 1e9, 1),
                                  "TFLOPs": round(flops / (ksum * 1e-6) / 1e12, 2),
                                  "per_layer_us": {k: round(v, 2) for k, v in lus.items()}}
            if b == 64:
                # the batched roofline: the step's matrix work against the
                # fp16 matrix-core peak, and against the lower bound that its
                # arithmetic intensity sets at the HBM peak
                tflops = flops / (ms * 1e-3) / 1e12
                intensity = flops / step_b
                hbm_bound = intensity * HBM_PEAK_GBS * 1e9 / 1e12
                result["roofline_bs64"] = {
                    "bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_F16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4),
                    "traffic": measured_traffic(TRAFFIC_FILE_BS64),
                    "algorithmic_flops": flops, "algorithmic_bytes": step_b,
                    "intensity_flop_per_byte": round(intensity, 1),
                    "hbm_bound_TFLOPs": round(hbm_bound, 1),
                    "frac_of_min_bound": round(tflops / min(MFMA_F16_PEAK_TFLOPS, hbm_bound), 4),
                    "kernel": "the batch-64 step of the 7 layers in 4 groups: per group the "
                              "activation conversion, qgemm_kernel (32x32x16 fp16 MFMA, "
                              "dominant) and the split reduction where K is split; "
                              "algorithmic flops (2 batch out in) over the step time"}
        # variable bitwidth (Sec. 4): exact allocation over the measured errors
        # with synthetic per-layer coefficients (real ones need a model + data)
        bits = [math.log2(fn) / fp + 16.0 / G for fp, fn, _, _ in dyn_opts]
        t2 = np.array(dyn_t2)
        sizes = np.array([L["out"] * L["in"] for L in layers], dtype=np.int64)
        alpha = np.random.default_rng(11).uniform(0.5, 2.0, len(layers))
        plans = {}
        for b_max in (3.5, 4.0, 4.5, 5.0, 6.0):
            t_a = time.perf_counter()
            choice, obj, avg = H.allocate_bits(alpha, t2, bits, sizes, b_max)
            dt = (time.perf_counter() - t_a) * 1e3
            plans[str(b_max)] = {"choice": [f"p{dyn_opts[c][0]}n{dyn_opts[c][1]}" for c in choice],
                                 "avg_bits": round(avg, 5), "objective": obj, "host_ms": round(dt, 3)}
        reps = 32  # a 32-block model: the 7 shapes repeated, coefficients per block
        alpha224 = np.random.default_rng(12).uniform(0.5, 2.0, reps * len(layers))
        t_a = time.perf_counter()
        choice224, obj224, avg224 = H.allocate_bits(alpha224, np.tile(t2, (reps, 1)), bits,
                                                    np.tile(sizes, reps), 4.0)
        dp224_ms = (time.perf_counter() - t_a) * 1e3
        extra["dynamic_bits"] = {
            "options": [f"p{fp}n{fn}" for fp, fn, _, _ in dyn_opts], "bits": bits,
            "t2": {L["name"]: [round(v, 6) for v in row] for L, row in zip(layers, dyn_t2)},
            "database_kernel_ms": round(dyn_ms, 3), "alpha": "uniform(0.5, 2), seed 11",
            "plans_7_layers": plans,
            "plan_224_layers_b4": {"avg_bits": round(avg224, 5), "objective": obj224,
                                   "host_ms": round(dp224_ms, 2)}}
        # GPTQ rounding (Sec. 3.5) on two 8B shapes with synthetic correlated
        # calibration activations: factor + quantize time, and the output error
        # on the calibration inputs (through the LUT product) against RTN
        gptq = {}
        for li in (0, 4):
            name, out, inp = synth.LLAMA8B_LAYERS[li]
            wt = synth.student_t_weight(out, inp, seed=2000 + li, dtype="bf16")
            w_dev = torch.from_numpy(wt.bits.view(np.int16)).to(dev).view(torch.bfloat16)
            rng = np.random.default_rng(40 + li)
            mix = torch.from_numpy((np.eye(inp) + 0.8 * rng.standard_normal((inp, inp))
                                    / math.sqrt(inp)).astype(np.float32)).to(dev)
            xc = torch.randn((1024, inp), device=dev) @ mix
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(stream)
            x_rot = H.rht_activations(xc, G, li)
            factor = H.gptq_factor(x_rot, 0.01)
            e1.record(stream)
            cg, sg = H.quantize_gptq(w_dev, grid, G, li, factor)
            e2.record(stream)
            torch.cuda.synchronize()
            cr, sr = H.quantize(w_dev, grid, G, li, index=gindex)
            y_true = xc.double() @ w_dev.double().T
            err = {}
            for tag, c, sc in (("gptq", cg, sg), ("rtn", cr, sr)):
                y = H.qmatmul(x_rot, c, sc, grid, G, out)
                err[tag] = float(((y.double() - y_true) ** 2).sum() / (y_true ** 2).sum())
            gptq[name] = {"shape": [out, inp], "calib_samples": 1024,
                          "factor_ms": round(e0.elapsed_time(e1), 2),
                          "quantize_ms": round(e1.elapsed_time(e2), 2),
                          "rel_output_err_gptq": err["gptq"], "rel_output_err_rtn": err["rtn"]}
            del w_dev, factor, xc, mix
            torch.cuda.synchronize()
        extra["gptq"] = gptq
        # other code formats (3-bit (2,64), 4-bit scalar (1,16), and the 8-bit
        # uniform CH8 grid (1,256)) at batch 1, 2, 8 and 64
        fmts = [(2, 64, H.make_grid(2, 64, 0, 1 << 18, 100)[0]),
                (1, 16, H.make_grid(1, 16, 0, 1 << 18, 100)[0]),
                (1, 256, H.make_uniform_grid(256)[0])]
        for fp, fn, fgrid in fmts:
            lus = format_layers_us(H, synth, dev, fp, fn, fgrid, (1, 2, 8, 64), flush)
            for b, per in lus.items():
                ksum = sum(per.values())
                byts = sum(qmm_bytes(b, L["out"], L["in"], fp, fn, G) for L in layers)
                flops = sum(2 * b * L["out"] * L["in"] for L in layers)
                extra[f"p{fp}n{fn}_batch{b}"] = {
                    "layers_us_sum": round(ksum, 2),
                    "GBps": round(byts / (ksum * 1e-6) / 1e9, 1),
                    "TFLOPs": round(flops / (ksum * 1e-6) / 1e12, 2),
                    "per_layer_us": {k: round(v, 2) for k, v in per.items()}}
        extra["llama70b_mixed"] = llama70b_extra(H, synth, dev, flush)
        dense = dense_bf16_extra(synth, dev, flush)
        for b, key in ((1, None), (16, "batch16"), (64, "batch64")):
            ours = result["ms_per_step"] if key is None else extra[key]["ms_per_step"]
            dense[f"batch{b}"]["higgs_step_us"] = round(ours * 1e3, 2)
            dense[f"batch{b}"]["dense_sum_over_higgs_step"] = round(
                dense[f"batch{b}"]["layers_us_sum"] / (ours * 1e3), 2)
        extra["dense_bf16_reference"] = dense
        result["extra"] = extra

    if not args.no_extra:
        extra["cfg1"] = cfg1_gpu(H, synth, dev, grid_np)
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(layers, grid_np, p, n)
        result["cpu_baseline"]["legs"] = cpu_legs(layers, grid_np, p, n)

    print(json.dumps(result), flush=True)


def format_layers_us(H, synth, dev, p, n, grid_np, batches, flush, reps=16):
    """Per-layer launch time of the fused product for another code format on
    the seven 8B shapes: random codes (every bit pattern is a valid code, so
    random bytes are the same traffic as encoded ones), `reps` distinct copies,
    one launch on each, replayed from a graph after a cache flush. Returns
    {batch: {layer: us}}."""
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    grid = torch.from_numpy(grid_np).to(dev)
    res = {b: {} for b in batches}
    for li, (name, out, inp) in enumerate(synth.LLAMA8B_LAYERS):
        rb = H.codes_row_bytes(inp, p, n)
        sets = [(torch.randint(0, 256, (out, rb), dtype=torch.uint8, device=dev, generator=gen),
                 (torch.rand((out, inp // G), device=dev, generator=gen) * 1e-3 + 1e-3).half())
                for _ in range(reps)]
        for b in batches:
            x = torch.randn((b, inp), device=dev, generator=gen).bfloat16()
            y = torch.empty((b, out), device=dev)
            wsb = H.qmatmul_fused_workspace_bytes(b, out, inp, p, n, G)
            ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
            res[b][name] = graph_train_us(
                lambda i: H.qmatmul_fused(x, *sets[i], grid, G, li, out, y=y, workspace=ws),
                reps, flush)
        del sets
        torch.cuda.synchronize()
    return res


def dense_bf16_extra(synth, dev, flush, batches=(1, 16, 64), reps=4):
    """A reference point on the same GPU: the seven 8B layers as dense bf16
    weights through torch.mm (hipBLASLt on ROCm), x [batch][in] times W
    [in][out]. Per-layer launch-to-launch time from graph trains over `reps`
    distinct weight copies after a cache flush, and the sum per batch. The
    quantized path reads a quarter of these weight bytes (plus scales) and
    rotates the activations."""
    import torch
    res = {}
    for b in batches:
        per = {}
        for name, out, inp in synth.LLAMA8B_LAYERS:
            ws = [torch.randn((inp, out), device=dev, dtype=torch.bfloat16) for _ in range(reps)]
            x = torch.randn((b, inp), device=dev, dtype=torch.bfloat16)
            ys = [torch.empty((b, out), device=dev, dtype=torch.bfloat16) for _ in range(reps)]
            per[name] = graph_train_us(lambda i: torch.mm(x, ws[i], out=ys[i]), reps, flush)
            del ws, ys
            torch.cuda.synchronize()
        res[f"batch{b}"] = {"layers_us_sum": round(sum(per.values()), 2),
                            "per_layer_us": {k: round(v, 2) for k, v in per.items()}}
    return res


def llama70b_extra(H, synth, dev, flush, batches=(1, 64), reps=12):
    """Llama-3.1-70B shapes with per-layer grids drawn by seed from p = 2,
    n in {64, 256, 1024}, g = 1024. Weights: the Student-t + outlier recipe
    drawn on the GPU (seed 5000 + layer), encoded by the library (kernel time
    recorded). Per layer and batch, launch-to-launch times from graph trains
    over `reps` distinct copies of the codes after a cache flush: the end-to-end
    layer (activation rotation + product, the fused call), and its two parts
    run separately: the rotation kernel, and the product on pre-rotated
    activations."""
    import torch
    stream = torch.cuda.current_stream()
    ns = synth.mixed_n_for_70b()
    grids, indexes = {}, {}
    for n in sorted(set(ns)):
        grids[n] = torch.from_numpy(H.make_grid(2, n, 0, 1 << 18, 100)[0]).to(dev)
        indexes[n] = H.search_index(grids[n])  # once per grid

    layers, enc_ms, weights = {}, 0.0, 0
    tot = {b: {"fused": 0.0, "rht": 0.0, "product": 0.0} for b in batches}
    for li, (name, out, inp) in enumerate(synth.LLAMA70B_LAYERS):
        n = ns[li]
        grid = grids[n]
        w, _ = synth.student_t_weight_device(out, inp, 5000 + li, dev)
        H.quantize(w, grid, G, li, index=indexes[n])  # warm-up of this shape
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        codes, scales = H.quantize(w, grid, G, li, index=indexes[n])
        e1.record(stream)
        torch.cuda.synchronize()
        enc_ms += e0.elapsed_time(e1)
        weights += out * inp
        del w
        sets = [(codes, scales)] + [(codes.clone(), scales.clone()) for _ in range(reps - 1)]
        rec = {"shape": [out, inp], "grid": [2, n]}
        for b in batches:
            act = synth.activations(b, inp, seed=5000 + li + 500 + b)
            x = torch.from_numpy(act.bits.view(np.int16)).to(dev).view(torch.bfloat16)
            x_rot = torch.empty((b, inp), dtype=torch.float32, device=dev)
            y = torch.empty((b, out), dtype=torch.float32, device=dev)
            wsb = max(H.qmatmul_fused_workspace_bytes(b, out, inp, 2, n, G),
                      H.qmatmul_workspace_bytes(b, out, inp, 2, n, G))
            ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
            fused = graph_train_us(lambda i: H.qmatmul_fused(x, *sets[i], grid, G, li, out,
                                                             y=y, workspace=ws), reps, flush)
            rht = graph_train_us(lambda i: H.rht_activations(x, G, li, out=x_rot), reps, flush)
            prod = graph_train_us(lambda i: H.qmatmul(x_rot, *sets[i], grid, G, out, y=y,
                                                      workspace=ws), reps, flush)
            byts = qmm_bytes(b, out, inp, 2, n, G)
            rec[f"batch{b}"] = {"fused_us": round(fused, 2), "rht_us": round(rht, 2),
                                "product_us": round(prod, 2),
                                "GBps": round(byts / (fused * 1e-6) / 1e9, 1),
                                "TFLOPs": round(2 * b * out * inp / (fused * 1e-6) / 1e12, 2)}
            tot[b]["fused"] += fused
            tot[b]["rht"] += rht
            tot[b]["product"] += prod
        layers[name] = rec
        del sets, codes, scales
        torch.cuda.synchronize()
    summary = {}
    for b in batches:
        byts = sum(qmm_bytes(b, out, inp, 2, ns[li], G)
                   for li, (_, out, inp) in enumerate(synth.LLAMA70B_LAYERS))
        flops = sum(2 * b * out * inp for _, out, inp in synth.LLAMA70B_LAYERS)
        t = tot[b]
        summary[f"batch{b}"] = {
            "layers_fused_us_sum": round(t["fused"], 2),
            "two_step_us_sum": round(t["rht"] + t["product"], 2),
            "rht_share_of_two_step": round(t["rht"] / (t["rht"] + t["product"]), 4),
            "GBps": round(byts / (t["fused"] * 1e-6) / 1e9, 1),
            "TFLOPs": round(flops / (t["fused"] * 1e-6) / 1e12, 2)}
    return {"grids": {nm: [2, n] for (nm, _, _), n in zip(synth.LLAMA70B_LAYERS, ns)},
            "encode": {"weights": weights, "kernel_ms": round(enc_ms, 3),
                       "weights_per_s": weights / (enc_ms * 1e-3)},
            "summary": summary, "per_layer": layers}


def kernel_sources(batch):
    """Sources of the kernels a --profile-pass at `batch` rows runs."""
    k = "qgemv.hip" if batch == 1 else "qgemm.hip"
    return [f"paper_2411_17525_amd/csrc/{k}", "paper_2411_17525_amd/csrc/wave_fwht.h",
            "paper_2411_17525_amd/csrc/internal.h"]


def summarize_counters(fetch_csv, write_csv, batch, out_json):
    """HBM traffic of the --profile-pass products from two rocprofv3 counter
    runs of it (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch). Per layer
    group the median over its three calls of the summed dispatches, each
    counter scaled by what it reads for the 64 MiB elementwise copy at the
    end of the pass (64 MiB in, 64 MiB out). Writes out_json (with the
    SHA-256 of the kernel sources: bench.py reports the traffic only while
    they are unchanged) and prints a markdown table. CPU only."""
    import csv
    import hashlib
    import statistics
    from paper_2411_17525_amd import synth

    def rows(path, counter):
        out = []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
        out.sort()
        return out

    def calls_and_copy(rs):
        ours = [r for r in rs if "higgs" in r[1]]  # demangled or not (templates)
        calls = []
        for _, name, v in ours:
            # a call starts with its activation conversion on the matrix-core
            # path, or is the one small-batch launch
            if "xprep" in name or "qgemv" in name or not calls:
                calls.append([])
            calls[-1].append((name, v))
        copies = [r for r in rs if "elementwise" in r[1] and "distribution" not in r[1]]
        return calls, copies[-1][2]

    fcalls, fcopy = calls_and_copy(rows(fetch_csv, "FETCH_SIZE"))
    wcalls, wcopy = calls_and_copy(rows(write_csv, "WRITE_SIZE"))
    if len(fcalls) != 3 * len(GROUPS) or len(wcalls) != 3 * len(GROUPS):
        raise SystemExit(f"expected {3 * len(GROUPS)} calls, got {len(fcalls)} / {len(wcalls)}")
    fscale, wscale = 65536.0 / fcopy, 65536.0 / wcopy
    shapes = synth.LLAMA8B_LAYERS
    p, n = 2, 256
    groups, step_hbm, step_alg = {}, 0, 0
    print("| group | algorithmic MB | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM MB (scaled) | HBM / algorithmic |")
    print("|---|---|---|---|---|---|")
    for gi, (gname, idx) in enumerate(GROUPS):
        fk = statistics.median(sum(v for _, v in c) for c in fcalls[3 * gi:3 * gi + 3])
        wk = statistics.median(sum(v for _, v in c) for c in wcalls[3 * gi:3 * gi + 3])
        hbm = (fk * fscale + wk * wscale) * 1024
        alg = group_bytes(batch, [(shapes[li][1], shapes[li][2]) for li in idx], p, n, G)
        groups[gname] = {"fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
                         "hbm_bytes": int(hbm), "algorithmic_bytes": int(alg),
                         "kernels": [nm.split("(")[0] for nm, _ in fcalls[3 * gi]]}
        step_hbm += hbm
        step_alg += alg
        print(f"| {gname} | {alg / 1e6:.1f} | {fk:.1f} | {wk:.1f} | {hbm / 1e6:.1f} | "
              f"{hbm / alg:.3f} |")
    print(f"\nstep: {step_hbm / 1e6:.1f} MB HBM vs {step_alg / 1e6:.1f} MB algorithmic "
          f"({step_hbm / step_alg:.3f}x); counter scale: fetch x{fscale:.4f}, write x{wscale:.4f}")
    h = hashlib.sha256()
    for f in kernel_sources(batch):
        h.update(open(os.path.join(ROOT, f), "rb").read())
    rec = {"workload": f"Llama-3.1-8B seven linear layers in four layer groups (q/k/v, o, "
                       f"gate/up, down), (p,n)=(2,256), g=1024, batch {batch}",
           "source_sha256": h.hexdigest(), "sources": kernel_sources(batch),
           "calibration": {"fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
                           "kernel": "torch.add(src, 0, out=dst), 64 MiB fp32 in / 64 MiB out",
                           "fetch_kib_read": fcopy, "write_kib_read": wcopy},
           "per_group": groups, "step_hbm_bytes": int(step_hbm),
           "step_algorithmic_bytes": int(step_alg)}
    with open(out_json, "w") as f:
        json.dump(rec, f, indent=1)
    print(f"wrote {out_json}")


def summarize_trace(trace_csv):
    """Per (kernel, grid) dispatch durations of this library's kernels in a
    rocprofv3 kernel_trace.csv: count, mean, median, p10, p90 (us), as a
    markdown table. CPU only."""
    import csv
    import statistics
    by = {}
    for r in csv.DictReader(open(trace_csv)):
        name = r["Kernel_Name"]
        if "higgs" not in name and "stream_read" not in name:
            continue
        short = name.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        key = (short[:72],
               int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"])),
               int(r["Workgroup_Size_X"]))
        by.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    print("| kernel | blocks x threads | dispatches | mean us | median us | p10 us | p90 us |")
    print("|---|---|---|---|---|---|---|")
    for (name, blocks, threads), ds in sorted(by.items()):
        ds.sort()
        q = lambda f: ds[min(len(ds) - 1, int(f * len(ds)))]
        print(f"| {name} | {blocks} x {threads} | {len(ds)} | {statistics.mean(ds):.2f} | "
              f"{statistics.median(ds):.2f} | {q(0.1):.2f} | {q(0.9):.2f} |")


def summarize_stats(stats_csv, top=45):
    """Every kernel of a rocprofv3 kernel_stats.csv (a whole run): calls and
    mean / min / max / total time, the `top` longest in total, then this
    library's search-index builds, as markdown tables. CPU only."""
    import csv
    import re

    def short(n):
        m = re.search(r"(xprep4?_kernel)ILi(\d+)E([tf])Lb([01])E", n)
        if m:
            return (f"{m.group(1)}<{m.group(2)}, {'bf16' if m.group(3) == 't' else 'float'}, "
                    f"{'rotate' if m.group(4) == '1' else 'no rotation'}>")
        if "stream_read_kernel" in n:
            return "stream_read_kernel (the measured ceiling)"
        if "higgs::" in n:
            n = n.replace("void ", "").replace("higgs::(anonymous namespace)::", "")
            n = n.replace("higgs::", "")
            i = n.find(">(")
            return n[:i + 1] if i >= 0 else n.split("(")[0]
        if n.startswith("void at::native::reduce_kernel<512, 1") and "sum_functor" in n:
            return ("at::native::reduce_kernel (torch sum: the 1 GiB cache-evicting read "
                    "before timed trains)")
        n = n.replace("void ", "")
        return n if len(n) <= 117 else n[:117] + "..."

    recs = [(short(r["Name"]), int(r["Calls"]), float(r["AverageNs"]) / 1e3,
             float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["TotalDurationNs"]) / 1e6)
            for r in csv.DictReader(open(stats_csv))]
    print("| kernel | calls | mean us | min us | max us | total ms |")
    print("|---|---|---|---|---|---|")
    for nm, c, a, mn, mx, tot in sorted(recs, key=lambda t: -t[5])[:top]:
        print(f"| `{nm}` | {c} | {a:.1f} | {mn:.1f} | {mx:.1f} | {tot:.2f} |")
    print()
    print("Search-index builds in the same run (once per grid):")
    print()
    print("| kernel | calls | mean us |")
    print("|---|---|---|")
    idx = [t for t in recs if t[0].startswith(("index_finish_kernel", "index_slots_kernel"))]
    for nm, c, a, *_ in sorted(idx, key=lambda t: (t[0].split("<")[1], t[0])):
        print(f"| `{nm}` | {c} | {a:.1f} |")


def profile_pass(H, synth, dev, p, n, batch=1):
    """Dispatches for hardware-counter runs (FETCH_SIZE / WRITE_SIZE per
    dispatch): the four layer groups of a step at `batch` rows (q/k/v, o,
    gate/up, down; at batch 1 one launch per group, on the matrix-core path
    the group's activation conversion, product and split reduction) over
    random codes (the same bytes as encoded ones), three copies each so each
    dispatch reads its codes from HBM, then one elementwise copy of 64 MiB in
    and 64 MiB out whose counters give the scale of the counters."""
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    grid = torch.randn((n, p), device=dev, generator=gen)
    shapes = synth.LLAMA8B_LAYERS
    for _, idx in GROUPS:
        inp = shapes[idx[0]][2]
        rb = H.codes_row_bytes(inp, p, n)
        x = torch.randn((batch, inp), device=dev, generator=gen).bfloat16()
        for c in range(3):
            lay = []
            for li in idx:
                out = shapes[li][1]
                codes = torch.randint(0, 256, (out, rb), dtype=torch.uint8, device=dev,
                                      generator=gen)
                scales = (torch.rand((out, inp // G), device=dev, generator=gen) * 1e-3
                          + 1e-3).half()
                lay.append((codes, scales, li, out))
            H.qmatmul_fused_multi(x, lay, grid, G)
            torch.cuda.synchronize()
            del lay
    src = torch.randn(16 << 20, device=dev, generator=gen)  # 64 MiB of fp32
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.add(src, 0.0, out=dst)
    torch.cuda.synchronize()
    log("profile pass done")


STAMP_PHASES = (
    ("arguments", 0, 1, False),
    ("table and loads issued", 1, 2, False),
    ("activations arrive", 2, 3, True),
    ("rotation", 3, 4, True),
    ("wait for the rotation", 4, 5, False),
    ("decode", 5, 6, False),
    ("wait for the block's last wave", 6, 7, False),
    ("K-wave sum and store", 7, 8, False),
)


def stamp_pass(H, synth, dev, p, n, reps=5):
    """Per batch-1 launch group (the step's four launches, random codes of the
    same shapes, a 1 GiB cache-evicting write before each call): the median
    over waves of each phase of qgemv_kernel, from the per-wave s_memrealtime
    stamps (100 MHz) of the phase-stamp build, then the median over `reps`
    calls; also the launch's span (first wave's start to last wave's end) and
    how long its waves take to start."""
    import ctypes
    import torch
    L = H.lib()
    if not hasattr(L, "higgs_debug_set_stamps"):
        raise SystemExit("--stamp-pass needs the phase-stamp build (libhiggs_stamps.so)")
    L.higgs_debug_set_stamps.argtypes = [ctypes.c_void_p]
    L.higgs_debug_set_stamps.restype = ctypes.c_int
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    grid = torch.randn((n, p), device=dev, generator=gen)
    buf = torch.zeros(2048 * 16 * 16, dtype=torch.int64, device=dev)
    if L.higgs_debug_set_stamps(ctypes.c_void_p(buf.data_ptr())) != 0:
        raise SystemExit("higgs_debug_set_stamps failed")
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    shapes = synth.LLAMA8B_LAYERS
    tick_us = 0.01  # s_memrealtime runs at 100 MHz
    rows = []
    for gname, idx in GROUPS:
        inp = shapes[idx[0]][2]
        x = torch.randn((1, inp), device=dev, generator=gen).bfloat16()
        per_call = []
        for c in range(reps + 1):
            lay = []
            for li in idx:
                out = shapes[li][1]
                codes = torch.randint(0, 256, (out, H.codes_row_bytes(inp, p, n)),
                                      dtype=torch.uint8, device=dev, generator=gen)
                scales = (torch.rand((out, inp // G), device=dev, generator=gen) * 1e-3
                          + 1e-3).half()
                lay.append((codes, scales, li, out))
            buf.zero_()
            flush.fill_(1.0)
            torch.cuda.synchronize()
            H.qmatmul_fused_multi(x, lay, grid, G)
            torch.cuda.synchronize()
            st = buf.view(-1, 16).cpu().numpy()
            st = st[st[:, 0] != 0]
            conv = (st[:, 9] & 1) == 1
            blocks = int((buf.view(-1, 16, 16)[:, :, 0] != 0).any(dim=1).sum().item())
            rec = {"waves": len(st), "blocks": blocks,
                   "kw": int((st[0, 9] >> 8) & 0xff), "rg": int((st[0, 9] >> 16) & 0xff),
                   "span": (st[:, 8].max() - st[:, 0].min()) * tick_us,
                   "start_spread": (st[:, 0].max() - st[:, 0].min()) * tick_us}
            for name, a, b, conv_only in STAMP_PHASES:
                sel = st[conv] if conv_only else st
                rec[name] = float(np.median(sel[:, b] - sel[:, a])) * tick_us
            if c > 0:
                per_call.append(rec)
            del lay
        med = {k: float(np.median([r[k] for r in per_call])) for k in per_call[0]}
        rows.append((gname, med))
    print("| phase (median over waves, us) | " + " | ".join(g for g, _ in rows) + " |")
    print("|---|" + "---|" * len(rows))
    print("| blocks x waves (K-waves x row groups) | " + " | ".join(
        f"{int(m['blocks'])} x {int(m['waves'] / max(m['blocks'], 1))} ({int(m['kw'])} x {int(m['rg'])})"
        for _, m in rows) + " |")
    for name, _, _, conv_only in STAMP_PHASES:
        label = name + (" (row group 0)" if conv_only else "")
        print(f"| {label} | " + " | ".join(f"{m[name]:.2f}" for _, m in rows) + " |")
    print("| launch span: first wave's start to last wave's end | "
          + " | ".join(f"{m['span']:.2f}" for _, m in rows) + " |")
    print("| waves' start spread | " + " | ".join(f"{m['start_spread']:.2f}" for _, m in rows)
          + " |")


ENCODE_FORMATS = ((2, 256), (2, 1024), (2, 64), (1, 256), (1, 16))


def encode_profile(H, synth, dev, reps=6):
    """Encoder dispatches in a fixed order (see --encode-profile): per format
    seven index builds, then `reps` encodes of each 8B layer shape (bf16
    weights N(0, 0.02^2) drawn on the GPU), and for (2, 256) `reps` encodes
    of the gate shape with no index. Prints event-timed medians to stderr."""
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)

    def t_us(fn):
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts[1:]))
    for p, n in ENCODE_FORMATS:
        g = H.make_uniform_grid(256)[0] if (p, n) == (1, 256) else H.make_grid(p, n, 0, 1 << 16, 30)[0]
        grid = torch.from_numpy(g).to(dev)
        idx = H.search_index(grid)
        log(f"({p},{n}) index build {t_us(lambda: H.search_index(grid, index=idx)):.1f} us")
        for name, out, inp in synth.LLAMA8B_LAYERS:
            w = (torch.randn((out, inp), device=dev, generator=gen) * 0.02).bfloat16()
            log(f"({p},{n}) {name} {out}x{inp}: "
                f"{t_us(lambda: H.quantize(w, grid, G, 0, index=idx)):.1f} us")
        if (p, n) == (2, 256):
            w = (torch.randn((14336, 4096), device=dev, generator=gen) * 0.02).bfloat16()
            log(f"(2,256) gate without index: "
                f"{t_us(lambda: H.quantize(w, grid, G, 0, index=False)):.1f} us")


def summarize_encode_trace(trace_csv, reps=6):
    """Markdown table of an --encode-profile trace: dispatches are matched to
    (format, layer) by their order; medians over all but the first of each
    run of `reps`."""
    import csv
    from paper_2411_17525_amd import synth
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    ev = []
    for r in rows:
        name = r["Kernel_Name"]
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        kind = ("slots" if "index_slots_kernel" in name else
                "finish" if "index_finish_kernel" in name else
                "q" if ("quantize_kernel" in name or "quantize_scan_kernel" in name) else None)
        if kind:
            ev.append((kind, name, d, r))
    i = 0

    def take(kind):
        nonlocal i
        assert ev[i][0] == kind, (i, ev[i][1])
        i += 1
        return ev[i - 1]
    print("| grid (p, n) | kernel | threads per block | index build us (lists + layout) | "
          + " | ".join(name for name, _, _ in synth.LLAMA8B_LAYERS)
          + " | seven layers us | G weights/s |")
    print("|---|---|---|---|" + "---|" * len(synth.LLAMA8B_LAYERS) + "---|---|")
    noidx = None
    for p, n in ENCODE_FORMATS:
        builds = [(take("slots")[2], take("finish")[2]) for _ in range(reps + 1)][2:]
        per, kern, threads, weights = [], "", "", 0
        for _, out, inp in synth.LLAMA8B_LAYERS:
            q = [take("q") for _ in range(reps)]
            per.append(float(np.median([e[2] for e in q[1:]])))
            kern = q[0][1].replace("higgs::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
            threads = q[0][3]["Workgroup_Size_X"]
            weights += out * inp
        if (p, n) == (2, 256):
            noidx = float(np.median([take("q")[2] for _ in range(reps)][1:]))
        tot = sum(per)
        print(f"| ({p}, {n}) | `{kern}` | {threads} | "
              f"{np.median([a for a, _ in builds]):.1f} + {np.median([b for _, b in builds]):.1f} | "
              + " | ".join(f"{x:.1f}" for x in per) + f" | {tot:.1f} | {weights / tot / 1e3:.1f} |")
    assert i == len(ev), (i, len(ev))
    print()
    print(f"(2, 256) gate shape with no index (every vector scans the grid): {noidx:.1f} us")


def cfg1_gpu(H, synth, dev, grid_np, reps=20):
    """The single 1024 x 1024 layer (fp32 Student-t weights, seed 0; grid
    (2, 256), g = 1024, rotation seed 0; one bf16 activation row, seed 1):
    GPU latency of the encoder, the activation rotation, the product on the
    rotated activations and the fused call (median over `reps` launches,
    HIP events; the layer fits in the caches, so these are warm latencies)."""
    import torch
    stream = torch.cuda.current_stream()
    wt = synth.student_t_weight(1024, 1024, seed=0, dtype="f32", outliers=False)
    act = synth.activations(1, 1024, seed=1)
    w = torch.from_numpy(wt.values).to(dev)
    x = torch.from_numpy(act.bits.view(np.int16)).to(dev).view(torch.bfloat16)
    grid = torch.from_numpy(grid_np).to(dev)
    gindex = H.search_index(grid)
    codes, scales = H.quantize(w, grid, G, 0, index=gindex)
    x_rot = H.rht_activations(x, G, 0)
    y = torch.empty((1, 1024), dtype=torch.float32, device=dev)

    def med_us(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        return round(float(np.median(ts)), 2)
    res = {"encode_us": med_us(lambda: H.quantize(w, grid, G, 0, codes=codes, scales=scales,
                                                  index=gindex)),
           "search_index_us": med_us(lambda: H.search_index(grid, index=gindex)),
           "rht_us": med_us(lambda: H.rht_activations(x, G, 0, out=x_rot)),
           "qmatmul_us": med_us(lambda: H.qmatmul(x_rot, codes, scales, grid, G, 1024, y=y)),
           "fused_us": med_us(lambda: H.qmatmul_fused(x, codes, scales, grid, G, 0, 1024, y=y))}
    res["encode_rht_qmatmul_us"] = round(res["encode_us"] + res["rht_us"] + res["qmatmul_us"], 2)
    res["note"] = ("each call timed alone between HIP events (launch included), median of "
                   f"{reps}; 1024x1024 fp32 weights encoded with g = 1024, batch 1")
    return res


def cpu_legs(layers, grid_np, p, n, reps=3):
    """The oracle's three parts timed on their own (median of `reps`): the
    encoder (explicit-H rotation + brute-force nearest point), the
    dequantisation (explicit inverse rotation) and the fp64 matmul on the
    dequantised weights (the fair 'CPU given dequantised weights' figure).
    The 1024 x 1024 layer in full; for the seven 8B layers, a 128-row
    matrix of each layer's width drawn with the same recipe (the oracle's
    cost per weight does not depend on the row count)."""
    from oracle import higgs_oracle as O
    from paper_2411_17525_amd import synth

    def med(fn):
        ts = []
        for _ in range(reps):
            t = time.perf_counter()
            r = fn()
            ts.append(time.perf_counter() - t)
        return float(np.median(ts)), r
    grid64 = grid_np.astype(np.float64)
    out = {}
    wt = synth.student_t_weight(1024, 1024, seed=0, dtype="f32", outliers=False)
    x = synth.activations(1, 1024, seed=1).values.astype(np.float64)
    t_enc, q = med(lambda: O.quantize(wt.values.astype(np.float64), grid64, G, 0))
    t_deq, w_hat = med(lambda: O.dequantize(q["codes"], q["scales"], grid64, G, 0))
    t_mm, _ = med(lambda: x @ w_hat.T)
    out["cfg1_1024x1024"] = {"encode_s": round(t_enc, 4), "dequantize_s": round(t_deq, 4),
                             "matmul_s": round(t_mm, 6),
                             "encode_weights_per_s": round(1024 * 1024 / t_enc, 1)}
    rows = 128
    tot = {"encode_s": 0.0, "dequantize_s": 0.0, "matmul_s": 0.0}
    wsum = 0
    for li, L in enumerate(layers):
        w_rows = synth.student_t_weight(rows, L["in"], seed=2000 + li,
                                        dtype="bf16").values.astype(np.float64)
        xb = synth.activations(1, L["in"], seed=2000 + li + 501).values.astype(np.float64)
        te, ql = med(lambda: O.quantize(w_rows, grid64, G, L["seed"]))
        td, wh = med(lambda: O.dequantize(ql["codes"], ql["scales"], grid64, G, L["seed"]))
        tm, _ = med(lambda: xb @ wh.T)
        tot["encode_s"] += te
        tot["dequantize_s"] += td
        tot["matmul_s"] += tm
        wsum += rows * L["in"]
    out["llama8b_128_row_samples"] = {
        **{k: round(v, 4) for k, v in tot.items()},
        "weights": wsum,
        "encode_weights_per_s": round(wsum / tot["encode_s"], 1),
        "dequantize_weights_per_s": round(wsum / tot["dequantize_s"], 1),
        "matmul_weights_per_s": round(wsum / tot["matmul_s"], 1)}
    out["note"] = f"median of {reps} runs per leg, fp64 NumPy on the host"
    return out


def cpu_baseline(layers, grid_np, p, n, budget_s=12.0):
    """The oracle (fp64 NumPy: dequantize through the explicit inverse Hadamard,
    then x W_hat^T) on a bounded sample of the same layers at batch 1: blocks of
    256 consecutive rows of every layer, round after round (rows wrap around),
    until `budget_s` seconds of oracle time have been spent."""
    import threadpoolctl
    from oracle import higgs_oracle as O
    from paper_2411_17525_amd import synth

    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    rows_per_block = 256
    host = []
    for li, L in enumerate(layers):
        act = synth.activations(1, L["in"], seed=2000 + li + 501)
        host.append((L["codes"].cpu().numpy(), L["scales"].cpu().numpy(),
                     act.values.astype(np.float64)))
    grid64 = grid_np.astype(np.float64)
    done_bytes = 0
    t_total = 0.0
    rounds = 0
    while t_total < budget_s:
        for li, L in enumerate(layers):
            codes_all, scales_all, x = host[li]
            r0 = (rounds * rows_per_block) % L["out"]
            sl = slice(r0, r0 + rows_per_block)
            c = O.unpack_codes(codes_all[sl], n, L["in"] // p)
            t = time.perf_counter()
            O.qmatmul(x, c, scales_all[sl], grid64, G, L["seed"])
            t_total += time.perf_counter() - t
            done_bytes += qmm_bytes(1, rows_per_block, L["in"], p, n, G)
        rounds += 1
    return {"value": round(done_bytes / t_total / 1e9, 6), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{rounds} blocks of {rows_per_block} rows of each of the 7 layers, batch 1 "
                      f"(dequantize + fp64 matmul; rows wrap), {t_total:.1f} s of oracle time"}


if __name__ == "__main__":
    main()
