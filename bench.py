#!/usr/bin/env python3
"""Throughput of the rotating-hypercube mixing stack on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload lm256_step]

The default workload is the language-model-shaped stack's whole training
step (window 256, width 512, batch 64, 16 rotated causal layers, byte-token
embedding, 256-way output head and cross-entropy): one step = the embedding
gather, the stack forward, the head with its loss and dlogits, the head's
gradients, the stack backward and the embedding's scatter sum over one batch
of synthetic inputs already resident in HBM, replayed as a HIP graph.
`--workload lm256` times the stack alone (one hcmix_stack_forward and one
hcmix_stack_backward call); the other workloads are the method's other
shapes (reach, long4096, hybrids, decode).
Prints one JSON line: positions*layers per second, the roofline of the
dominant kernel (timed live with HIP events on the stream it runs on) and the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("positions·layers/sec (fwd+bwd) + % bf16 MFMA peak / % HBM BW, window 256")
UNIT = "positions·layers/s"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

WORKLOADS = {
    "lm256": "window n=256, width 512, batch 64, 16 rotated causal layers, bf16, fwd+bwd",
    "reach": "window n=256, width 64, batch 64, 8 rotated bidirectional layers, bf16, fwd+bwd",
    "long4096": "window n=4096, width 1024, batch 8, 24 rotated causal layers, bf16, fwd+bwd",
    "hybrid": ("window n=256, width 512, batch 64, 16 rotated causal layers with 2 causal "
               "softmax attention layers (8 heads x 64) at slots 3 and 9 of 18, bf16, fwd+bwd"),
    "decode256": ("decode: window n=256, width 512, batch 64, 16 rotated causal layers, bf16; "
                  "positions 0..255 one step each (all windows, every layer)"),
    "lm256_step": ("window n=256, width 512, batch 64, 16 rotated causal layers, bf16: the whole "
                   "language-model training step, Zipf byte-token embedding, the stack forward and "
                   "backward, 256-way output head with bias and cross-entropy"),
    "hy256": ("window n=256, width 512, batch 64, the hybrid256 schedule: 8 local layers, 6 "
              "causal jumps 128..1 and 2 causal softmax attention layers (8 heads x 64), 16 "
              "layers, bf16, fwd+bwd"),
    "shared256": ("window n=256, width 512, batch 64, 16 rotated causal channel-shared layers "
                  "(per-position scalar maps from one 256 x 256 table per layer), Zipf byte-token "
                  "embedding inputs, bf16, fwd+bwd"),
    "field256": ("window n=256, width 512, batch 64, the field coupling of Section 3.4 (scaled "
                 "Gaussian distance kernel, 32 coordinates, tau 1, mean squared distance 100) "
                 "applied T = 8 times in a chain, each application with its own coordinates, "
                 "Zipf byte-token embedding inputs, bf16 with fp32 coordinates, fwd+bwd"),
}
# hybrid: positions of the attention layers in the 18-layer list
HYBRID_ATTN_SLOTS = (3, 9)
HYBRID_LAYERS = 18
# the paper's window-256 hybrid schedule string (Appendix A), by layer name
HY256 = ("near jump128 near attn near jump32 near jump16 near attn near jump4 near jump2 "
         "near jump1").split()


def algorithmic_work(batch, n, width, layers, causal):
    """Flops and HBM bytes per step counting only the links the method has:
    per position-layer forward 3w^2 (causal) or 4w^2 (bidir) flops, backward
    twice that; bytes 2 (fwd: read x, write y) + 3 (bwd: read dy, x, write dx)
    activation rows of w bf16 values."""
    pl = batch * n * layers
    f_fwd = (3 if causal else 4) * width * width
    return pl * 3 * f_fwd, pl * 5 * width * 2


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="lm256_step", choices=sorted(WORKLOADS))
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's batch (windows), e.g. for a batch sweep")
    ap.add_argument("--graph", type=int, default=1, help="replay the step as a HIP graph")
    ap.add_argument("--cpu-baseline", type=int, default=1)
    ap.add_argument("--cpu-windows", type=int, default=0,
                    help="windows in the oracle sample (0: sized for ~10-30 s)")
    ap.add_argument("--kernel-reps", type=int, default=20)
    ap.add_argument("--mode", default="preset", choices=["preset", "causal", "bidir"],
                    help="lm256, reach, long4096: run the stack causal or bidirectional instead "
                         "of the preset's mode")
    ap.add_argument("--attention", default="native", choices=["native", "sdpa"],
                    help="hybrid workloads: the library's attention core, or PyTorch SDPA")
    ap.add_argument("--proj", default="library", choices=["library", "torch"],
                    help="hybrids: the attention layers' projections in the library's kernels "
                         "(the whole step in library calls) or as PyTorch GEMMs under autograd")
    ap.add_argument("--head-grad", default="library", choices=["library", "torch"],
                    help="lm256_step: the head's input and weight gradients in the library's "
                         "kernels or as PyTorch GEMMs")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    return ap.parse_args()


def kernel_source_hash() -> str:
    """Hash of the HIP sources; a traffic figure is valid only for the same sources."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2609_18145_amd", "csrc", "*"))):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def profiled_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (profiles/traffic_<workload>.json), or None if it was taken on different
    kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch", {}).get(kernel)


def calibration_copy(torch, dev, mib):
    """One plain device copy of `mib` MiB: the reference that scales the
    profiler's FETCH_SIZE and WRITE_SIZE counters to bytes."""
    src = torch.empty(mib << 20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def device_copy_context(torch, dev):
    """Measured context for the HBM roofline: a plain device-to-device copy of
    1 GiB (read + write counted), timed with HIP events after one warm-up --
    the practical ceiling a streaming kernel can reach on this device, beside
    the 8 TB/s specification the fractions are quoted against."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 5 * 2 * n / (e0.elapsed_time(e1) / 1e3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"device_copy_GBps": round(gbs, 1), "device_copy_frac_of_peak": round(gbs / PEAK_HBM_GBS, 4),
            "note": "a 1 GiB device-to-device copy, read + write bytes over its time"}


def fused_path(n, w, L):
    """Shapes the library runs as one LDS-resident kernel per stack direction."""
    return w == 64 and n in (64, 128, 256) and L <= 64


def deferred_path(n, w, L):
    """Shapes whose stack backward runs the dX chain (one mix launch per
    layer) and then every layer's weight gradients in one dw_batch_kernel
    launch (bf16, two or more layers, width a multiple of 128)."""
    return not fused_path(n, w, L) and L > 1 and w % 128 == 0


def profiled_mfma(workload: str, kernel: str, sec: float, flops: int):
    """MFMA counter evidence for `kernel` from the committed counter summary
    (profiles/mfma_<workload>.json; the LM step's stack kernels run at the
    lm256 launch configuration and use its file): the flops the MFMA units
    issued per launch (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) against the
    algorithmic count, and MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES over the 1024
    SIMDs x 2.4 GHz x this launch's measured duration.  None if the counters
    were taken on different kernel sources."""
    wl = "lm256" if workload == "lm256_step" else workload
    path = os.path.join(ROOT, "profiles", f"mfma_{wl}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    k = rec.get("kernels", {}).get(kernel)
    if rec.get("source_hash") != kernel_source_hash() or k is None:
        return None
    return {"issued_flops": k["mops_bf16_x512"], "issued_equals_algorithmic":
            k["mops_bf16_x512"] == flops,
            "mfma_busy": round(k["mfma_busy_cycles"] / (sec * 2.4e9 * 1024), 4),
            "source": f"profiles/mfma_{wl}.json"}


def graph_timed(torch, fn, count, replays=3):
    """Seconds per call of fn: `count` calls captured back to back in one
    graph, replayed `replays` times between HIP events on the stream the
    kernels run on (a stream of its own that first waits for the caller's).
    Graph replay is how the timed steps run: the binding's host-side operand
    checks stay out of the timed region, consecutive kernels start within
    about 0.3 us of each other (kernel traces), and one graph launch is
    spread over `count` calls, so the figure is the kernels' own time plus the
    dependent-launch gaps of the step itself."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        fn()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            for _ in range(count):
                fn()
        graph.replay()
        torch.cuda.synchronize()
        k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        k0.record(side)
        for _ in range(replays):
            graph.replay()
        k1.record(side)
        torch.cuda.synchronize()
    del graph
    return k0.elapsed_time(k1) / 1e3 / (count * replays)


def dominant_kernel(args, hcmix, stream, x0, ws, wo, dy, xs_out, dx_out, dws, dwo, workspace,
                    layers, B, n, w, L, causal):
    """Roofline entries, timed with HIP events on the stream the kernels run
    on over calls captured back to back in one graph (graph_timed): {name:
    entry}, the dominant one under "roofline".

    Small width (the fused path): the backward stack call (fused_bwd_kernel
    plus its fixed-order partial reduction), against HBM bandwidth; its
    algorithmic bytes are dY, the L saved inputs and dX (bf16), the 2L weight
    matrices (bf16) read and the 2L weight gradients (fp32) written.

    Wider layers: the mix GEMM (mix_bf16_kernel), which runs every forward
    layer and every dX and so holds most of the step, timed on its forward
    instance (hcmix_forward launches of the stack's layers, the launch
    configuration the stack uses): flops B n w^2 x 3 causal / x 4
    bidirectional per launch (2 w^2 for the self map of every position, 2 w^2
    for the partner map of each receiver).  Beside it ("roofline_dw", deferred
    path only) the all-layer weight-gradient launch (hcmix_stack_weight_
    gradients, dw_batch_kernel): flops B n L w^2 x 3 causal / x 4 bidirectional
    (dW_self 2 w^2 per position, dW_off 2 w^2 per receiver)."""
    import torch
    reps = args.kernel_reps
    xs = [x0, *xs_out[:L - 1]]
    # committed counter figures belong to the preset's mode only
    pkey = args.workload if args.mode == "preset" else f"{args.workload} ({args.mode})"

    def timed(fn, count):
        return graph_timed(torch, fn, count)

    if fused_path(n, w, L):
        sec = timed(lambda: hcmix.stack_backward(xs, ws, wo, layers, dy, causal, dx=dx_out[0],
                                                 dws=dws, dwo=dwo, workspace=workspace), reps)
        act = B * n * w * 2
        nbytes = act * (L + 2) + 2 * L * w * w * 2 + 2 * L * w * w * 4
        gbs = nbytes / sec / 1e9
        kname = "fused_bwd_kernel + fused_dw_reduce_kernel"
        return {"roofline": {"bound": "hbm", "kernel": kname + " (one hcmix_stack_backward call)",
                             "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                             "frac": round(gbs / PEAK_HBM_GBS, 4),
                             "traffic": profiled_traffic(pkey, kname),
                             "avg_launch_us": round(sec * 1e6, 2), "algorithmic_bytes": nbytes}}

    def fwd_layers():
        for l in range(L):
            hcmix.forward(xs_out[l - 1] if l else x0, ws[l], wo[l], layers[l], causal,
                          out=xs_out[l])

    sec = timed(fwd_layers, reps) / L
    flops = B * n * (3 if causal else 4) * w * w
    tflops = flops / sec / 1e12
    kname = "mix_bf16_kernel<forward>"
    out = {"roofline": {"bound": "mfma", "kernel": kname + " (one forward layer launch)",
                        "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                        "traffic": profiled_traffic(pkey, kname),
                        "avg_launch_us": round(sec * 1e6, 2), "algorithmic_flops": flops,
                        "counters": profiled_mfma(pkey, kname, sec, flops)}}
    if deferred_path(n, w, L):
        # the saved activations stand in for the output gradients: the same
        # shapes and magnitudes, and the kernel's work does not depend on values
        gs = [*xs_out[1:L], dy]
        sec = timed(lambda: hcmix.stack_weight_gradients(xs, gs, layers, causal, dws=dws,
                                                         dwo=dwo), reps)
        flops = B * n * L * (3 if causal else 4) * w * w
        tflops = flops / sec / 1e12
        kname = "dw_batch_kernel"
        out["roofline_dw"] = {"bound": "mfma", "kernel": kname + f" (weight gradients of all {L} "
                              "layers, one launch)", "achieved": round(tflops, 2),
                              "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                              "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                              "traffic": profiled_traffic(pkey, kname),
                              "avg_launch_us": round(sec * 1e6, 2), "algorithmic_flops": flops,
                              "counters": profiled_mfma(pkey, kname, sec, flops)}
    sec = timed(lambda: hcmix.stack_backward(xs, ws, wo, layers, dy, causal, dx=dx_out[0],
                                             dws=dws, dwo=dwo, workspace=workspace), reps)
    out["backward_call_us"] = round(sec * 1e6, 2)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the hot path runs on one GPU only (asked for --gpus {args.gpus}); "
              "sharding across GPUs is not implemented.", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2609_18145_amd import hcmix, inputs

    if args.mode != "preset" and args.workload not in inputs.PRESETS:
        print(f"bench.py: --mode applies to the stack workloads {sorted(inputs.PRESETS)}",
              file=sys.stderr)
        return 2

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    hcmix.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.workload in ("hybrid", "hy256"):
        return run_hybrid(args, torch, hcmix, inputs, dev)
    if args.workload == "decode256":
        return run_decode(args, torch, hcmix, inputs, dev)
    if args.workload == "lm256_step":
        return run_lm_step(args, torch, hcmix, inputs, dev)
    if args.workload == "field256":
        return run_field(args, torch, hcmix, inputs, dev)
    if args.workload == "shared256":
        return run_shared(args, torch, hcmix, inputs, dev)
    over = {"batch": args.batch} if args.batch > 0 else {}
    if args.mode != "preset":
        over["causal"] = args.mode == "causal"
    cfg = dict(inputs.PRESETS[args.workload], **over)
    s = inputs.make_preset(args.workload, **over)
    B, n, w, L, causal = cfg["batch"], cfg["n"], cfg["width"], cfg["num_layers"], cfg["causal"]
    dt = torch.bfloat16

    def dev_t(a):
        return torch.from_numpy(a).to(dt).to(dev)

    x0 = dev_t(s.x)
    ws = [dev_t(a) for a in s.w_self]
    wo = [dev_t(a) for a in s.w_off]
    dy = dev_t(s.dy)
    xs_out = [torch.empty_like(x0) for _ in range(L)]
    dx_out = [torch.empty_like(x0) for _ in range(L)]
    dws = [torch.empty((w, w), dtype=torch.float32, device=dev) for _ in range(L)]
    dwo = [torch.empty((w, w), dtype=torch.float32, device=dev) for _ in range(L)]
    workspace = hcmix.alloc_stack_workspace(B, n, w, L, dt, dev)

    def step():
        xs = hcmix.stack_forward(x0, ws, wo, s.layers, causal, outs=xs_out)
        hcmix.stack_backward(xs, ws, wo, s.layers, dy, causal, dx=dx_out[0], dws=dws, dwo=dwo,
                             workspace=workspace)

    stream = torch.cuda.Stream(device=dev)
    graph = None
    with torch.cuda.stream(stream):
        step()
        torch.cuda.synchronize()
        if args.graph:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                step()
        run = graph.replay if graph is not None else step
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        gpu_s = e0.elapsed_time(e1) / 1e3
        t = max(wall, gpu_s)

        kernels = dominant_kernel(args, hcmix, stream, x0, ws, wo, dy, xs_out, dx_out, dws, dwo,
                                  workspace, s.layers, B, n, w, L, causal)

    if args.calib_copy_mb > 0:
        calibration_copy(torch, dev, args.calib_copy_mb)

    flops, nbytes = algorithmic_work(B, n, w, L, causal)
    pl_per_step = B * n * L
    value = pl_per_step * args.steps / t
    ms = t / args.steps * 1e3
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOADS[args.workload]}"
                               + (f" (batch overridden to {B})" if args.batch > 0 else "")
                               + (f" (mode overridden to {args.mode})" if args.mode != "preset"
                                  else ""), "batch": B,
                   "n": n, "width": w, "layers": L, "mode": "causal" if causal else "bidir",
                   "graph": bool(args.graph)},
        "pct_bf16_peak": round(flops / t * args.steps / 1e12 / PEAK_BF16_TFLOPS * 100, 2),
        "pct_hbm": round(nbytes / t * args.steps / 1e9 / PEAK_HBM_GBS * 100, 2),
    }
    out.update(kernels)
    if args.cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(s, n, w, L, causal, args.cpu_windows)
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def native_segment_split(torch, hstack, x0, dy, nattn, reps):
    """Seconds per step of the sparse and the attention segments of a
    library-only hybrid step (HybridStack): one eager step records every
    segment's input and output gradient, then each segment's forward call and
    backward call, and the closing all-layer weight-gradient call, is timed on
    its own over calls captured back to back in a graph with those inputs
    (graph_timed; the kernels' work does not depend on the values).  The
    stack's saved state is restored around each timing, since a segment call
    appends to it."""
    hstack._saved = []
    xin, x = [], x0
    for k in range(len(hstack.segments)):
        xin.append(x)
        x = hstack.forward_segment(k, x)
    saved = list(hstack._saved)
    hstack._dw_in = []
    hstack.dw_attn = [None] * nattn
    gin, g = {}, dy
    for k in reversed(range(len(hstack.segments))):
        gin[k] = g
        g = hstack.backward_segment(k, g)
    dw_in = list(hstack._dw_in)
    torch.cuda.synchronize()
    res = {"sparse": 0.0, "attn": 0.0}
    for k, (kind, _) in enumerate(hstack.segments):
        def fwd(k=k):
            hstack._saved = list(saved[:k])
            hstack.forward_segment(k, xin[k])
        t_f = graph_timed(torch, fwd, reps)
        hstack._saved = saved

        def bwd(k=k):
            hstack._dw_in = []
            hstack.backward_segment(k, gin[k])
        t_b = graph_timed(torch, bwd, reps)
        res[kind] += t_f + t_b
    hstack._dw_in = dw_in
    res["sparse"] += graph_timed(torch, hstack.sparse_weight_gradients, reps)
    return res


def run_hybrid(args, torch, hcmix, inputs, dev):
    """Sparse layers with two causal softmax attention layers among them:
    "hybrid", the lm256 stack with attention inserted at slots 3 and 9 of 18
    (the rotated layers keep d = their index among the rotated layers mod 8),
    or "hy256", the paper's window-256 hybrid schedule string (local layers,
    one causal jump per scale, attention at two of sixteen; weights are the
    lm256 workload's first 14).  An attention layer is the QKV projection and
    the output projection (the library's linear maps, hcmix_linear_forward /
    _backward) around the library's causal attention core
    (hcmix_attention_forward / _backward): by default the whole step is
    library calls (paper_2609_18145_amd.hybrid); --proj torch runs the
    projections as PyTorch GEMMs and --attention sdpa swaps in PyTorch's
    scaled-dot-product attention, both under torch autograd, for comparison.
    The sparse segments are hcmix stack calls: forward per segment, the dX
    chain per segment (hcmix_stack_backward_data), and the weight gradients of
    every sparse layer in one hcmix_stack_weight_gradients call at the end.  Forward and backward are chained by hand
    so that every segment can be timed on its own.  value = positions x
    (sparse + attention) layers per second of the whole step; beside it the
    sparse and attention segments' times (native_segment_split)."""
    import torch.nn.functional as F
    cfg = dict(inputs.PRESETS["lm256"])
    if args.batch > 0:
        cfg["batch"] = args.batch
    s = inputs.make_preset("lm256", **({"batch": args.batch} if args.batch > 0 else {}))
    B, n, w = cfg["batch"], cfg["n"], cfg["width"]
    dt = torch.bfloat16
    heads, hd = 8, 64
    assert heads * hd == w

    def dev_t(a):
        return torch.from_numpy(a).to(dt).to(dev)

    x0, dy = dev_t(s.x), dev_t(s.dy)
    ws = [dev_t(a) for a in s.w_self]
    wo = [dev_t(a) for a in s.w_off]
    gen = torch.Generator(device="cpu").manual_seed(1)
    attn_w = [((torch.randn(3 * w, w, generator=gen) / w ** 0.5).to(dt).to(dev),
               (torch.randn(w, w, generator=gen) / w ** 0.5).to(dt).to(dev))
              for _ in range(2)]
    # the schedule as entries: a layer code, or "attn"
    if args.workload == "hybrid":
        sched, rot = [], 0
        for slot in range(HYBRID_LAYERS):
            if slot in HYBRID_ATTN_SLOTS:
                sched.append("attn")
            else:
                sched.append(rot)   # rotated: dimension = index among rotated layers mod 8
                rot += 1
    else:
        sched = []
        for name in HY256:
            if name == "attn":
                sched.append("attn")
            elif name == "near":
                sched.append(hcmix.LAYER_NEAR)
            else:
                sched.append(int(name[len("jump"):]).bit_length() - 1)
    # segments: runs of sparse layers (weight indices, layer codes) and attention layers
    segs, cur, nsparse, nattn = [], [], 0, 0
    for e in sched:
        if e == "attn":
            segs.append(("sparse", cur))
            segs.append(("attn", nattn))
            cur, nattn = [], nattn + 1
        else:
            cur.append((nsparse, e))
            nsparse += 1
    segs.append(("sparse", cur))
    segs = [sg for sg in segs if sg[0] == "attn" or sg[1]]
    Ls = nsparse
    assert Ls <= len(ws) and nattn == len(attn_w)

    from torch.nn.attention import SDPBackend, sdpa_kernel
    backend = {"name": None}

    def sdpa(q, k, v):
        if backend["name"] is None:
            for name, be in (("flash", SDPBackend.FLASH_ATTENTION),
                             ("efficient", SDPBackend.EFFICIENT_ATTENTION)):
                try:
                    with sdpa_kernel([be]):
                        out = F.scaled_dot_product_attention(q, k, v, is_causal=True)
                    backend["name"], backend["be"] = name, be
                    return out
                except RuntimeError:
                    continue
            backend["name"] = "fp32 math"
        if backend["name"] == "fp32 math":
            # plain fp32 products on contiguous operands
            qf, kf, vf = (t.float().contiguous() for t in (q, k, v))
            att = torch.matmul(qf, kf.transpose(-1, -2).contiguous()) / hd ** 0.5
            mask = torch.ones(n, n, dtype=torch.bool, device=dev).triu(1)
            att = att.masked_fill(mask, float("-inf")).softmax(-1)
            return torch.matmul(att, vf).to(q.dtype)
        with sdpa_kernel([backend["be"]]):
            return F.scaled_dot_product_attention(q, k, v, is_causal=True)

    class Linear(torch.autograd.Function):
        """y = x W^T under autograd (the comparison paths: --proj torch or
        --attention sdpa).  --proj library: the library's linear map
        (hcmix_linear_forward / _backward); --proj torch: PyTorch GEMMs, the
        weight gradient's K = rows split into 16 batched products (a single GEMM
        with K = 16384 and a 512-wide output leaves most of the chip idle in its
        kernel choice)."""

        @staticmethod
        def forward(ctx, x2, wt):
            ctx.save_for_backward(x2, wt)
            if args.proj == "library":
                return hcmix.linear_forward(x2.contiguous(), wt)
            return torch.matmul(x2, wt.t())

        @staticmethod
        def backward(ctx, g):
            x2, wt = ctx.saved_tensors
            g = g.contiguous()
            if args.proj == "library":
                dx, dw = hcmix.linear_backward(x2, wt, g)
                return dx, dw.to(wt.dtype)
            kch = 16
            r = x2.shape[0] // kch
            dw = torch.bmm(g.view(kch, r, -1).transpose(1, 2), x2.view(kch, r, -1)).sum(0)
            return torch.matmul(g, wt), dw

    def attention(x, i):
        wqkv, wout = attn_w[i]
        qkv = Linear.apply(x.reshape(B * n, w), wqkv).view(B, n, 3, heads, hd)
        if args.attention == "native":
            o = hcmix.Attention.apply(qkv).reshape(B * n, w)
        else:
            q, k, v = (qkv[:, :, j].transpose(1, 2).contiguous() for j in range(3))
            o = sdpa(q, k, v).transpose(1, 2).reshape(B * n, w)
        return Linear.apply(o, wout).view(B, n, w)

    wsp = {}
    stream = torch.cuda.current_stream(dev)
    ev = torch.cuda.Event

    native = args.proj == "library" and args.attention == "native"
    from paper_2609_18145_amd.hybrid import HybridStack
    hstack = HybridStack(sched, ws[:Ls], wo[:Ls], attn_w[:nattn], heads)

    def step_native(times):
        """One step, every part a library call (paper_2609_18145_amd.hybrid):
        sparse stacks, linear maps and attention cores forward, the reverse
        backward (sparse dX chains, attention backward products), then all
        sparse weight gradients in one call."""
        cur = torch.cuda.current_stream(dev)

        def timed(kind, phase, fn):
            if times is None:
                return fn()
            e0, e1 = ev(enable_timing=True), ev(enable_timing=True)
            e0.record(cur)
            out = fn()
            e1.record(cur)
            times.append((kind, phase, e0, e1))
            return out

        hstack._saved = []
        x = x0
        for k, (kind, _) in enumerate(hstack.segments):
            x = timed(kind, "fwd", lambda: hstack.forward_segment(k, x))
        hstack._dw_in = []
        hstack.dw_attn = [None] * nattn
        g = dy
        for k in reversed(range(len(hstack.segments))):
            g = timed(hstack.segments[k][0], "bwd", lambda: hstack.backward_segment(k, g))
        timed("sparse", "dw", hstack.sparse_weight_gradients)
        return g

    def step(times):
        """One step; with `times` a list, every segment is bracketed by events
        on the current stream (left out under graph capture, times=None)."""
        if native:
            return step_native(times)
        cur = torch.cuda.current_stream(dev)

        def bracket():
            if times is None:
                return None, None
            e0, e1 = ev(enable_timing=True), ev(enable_timing=True)
            e0.record(cur)
            return e0, e1

        saved, x = [], x0
        for kind, arg in segs:                      # forward
            e0, e1 = bracket()
            if kind == "sparse":
                xs = hcmix.stack_forward(x, [ws[j] for j, _ in arg], [wo[j] for j, _ in arg],
                                         [c for _, c in arg], True)
                saved.append(xs)
                x = xs[-1]
            else:
                xin = x.detach().requires_grad_(True)
                params = [p.requires_grad_(True) for p in attn_w[arg]]
                with torch.enable_grad():
                    out = attention(xin, arg)
                saved.append((xin, out, params))
                x = out.detach()
            if times is not None:
                e1.record(cur)
                times.append((kind, "fwd", e0, e1))
        g = dy
        # the sparse segments run their dX chains only; the weight gradients of
        # all sparse layers follow in one library call
        dw_x, dw_g, dw_codes = [], [], []
        for (kind, arg), sv in zip(reversed(segs), reversed(saved)):   # backward
            e0, e1 = bracket()
            if kind == "sparse":
                L = len(arg)
                g_out = g
                g, grads = hcmix.stack_backward_data([ws[j] for j, _ in arg],
                                                     [wo[j] for j, _ in arg],
                                                     [c for _, c in arg], g_out, True)
                dw_x += sv[:L]
                dw_g += [*grads, g_out]
                dw_codes += [c for _, c in arg]
            else:
                xin, out, params = sv
                grads = torch.autograd.grad(out, [xin, *params], grad_outputs=g)
                g = grads[0].contiguous()
            if times is not None:
                e1.record(cur)
                times.append((kind, "bwd", e0, e1))
        e0, e1 = bracket()
        if "dw" not in wsp:
            wsp["dw"] = ([torch.empty((w, w), dtype=torch.float32, device=dev) for _ in dw_x],
                         [torch.empty((w, w), dtype=torch.float32, device=dev) for _ in dw_x])
        hcmix.stack_weight_gradients(dw_x, dw_g, dw_codes, True, dws=wsp["dw"][0],
                                     dwo=wsp["dw"][1])
        if times is not None:
            e1.record(cur)
            times.append(("sparse", "dw", e0, e1))
        return g

    for _ in range(args.warmup):
        step([])
    torch.cuda.synchronize()
    per_step = []
    t0 = time.perf_counter()
    c0, c1 = ev(enable_timing=True), ev(enable_timing=True)
    c0.record(stream)
    for _ in range(args.steps):
        times = []
        step(times)
        per_step.append(times)
    c1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_eager = max(wall, c0.elapsed_time(c1) / 1e3)
    sparse = sum(e0.elapsed_time(e1) for st in per_step for k, _, e0, e1 in st if k == "sparse") / 1e3
    attn = sum(e0.elapsed_time(e1) for st in per_step for k, _, e0, e1 in st if k == "attn") / 1e3
    total = total_eager
    if args.graph:
        # the same step (forward, attention autograd, library backward) captured
        # once and replayed: the step time without host launch overhead
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(stream)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            step(None)
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                step(None)
            for _ in range(args.warmup):
                graph.replay()
            torch.cuda.synchronize()
            g0, g1 = ev(enable_timing=True), ev(enable_timing=True)
            t0 = time.perf_counter()
            g0.record(side)
            for _ in range(args.steps):
                graph.replay()
            g1.record(side)
            torch.cuda.synchronize()
        total = max(time.perf_counter() - t0, g0.elapsed_time(g1) / 1e3)
    seg_split = None
    if native:
        seg_split = native_segment_split(torch, hstack, x0, dy, nattn, args.kernel_reps)
    pl = B * n * (Ls + nattn)
    core_us = None
    if args.attention == "native":
        # the attention core alone (forward + backward of one layer), back to back
        gen_q = torch.Generator(device="cpu").manual_seed(2)
        qkv = torch.randn(B, n, 3, heads, hd, generator=gen_q).to(dt).to(dev)
        gout = torch.randn(B, n, heads, hd, generator=gen_q).to(dt).to(dev)
        o_, l_ = hcmix.attention_forward(qkv)
        dq_ = hcmix.attention_backward(qkv, o_, l_, gout)

        def core():
            hcmix.attention_forward(qkv, out=o_, lse=l_)
            hcmix.attention_backward(qkv, o_, l_, gout, dqkv=dq_)
        core_us = round(graph_timed(torch, core, args.kernel_reps) * 1e6, 2)
        backend["name"] = "hcmix_attention (library kernels)"
    out = {
        "metric": METRIC, "value": round(pl * args.steps / total, 1), "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(total / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOADS[args.workload]}", "batch": B, "n": n,
                   "width": w, "layers": Ls, "attention_layers": nattn, "mode": "causal",
                   "graph": bool(args.graph), "attention_backend": backend["name"],
                   "projections": "hcmix_linear (library kernels)" if args.proj == "library"
                   else "PyTorch GEMMs"},
        "hybrid": {"step_ms": round(total / args.steps * 1e3, 4),
                   "step_ms_eager": round(total_eager / args.steps * 1e3, 4),
                   "attention_core_fwd_bwd_us_per_layer": core_us},
    }
    if seg_split is not None:
        out["hybrid"].update({
            "sparse_ms": round(seg_split["sparse"] * 1e3, 4),
            "attention_ms": round(seg_split["attn"] * 1e3, 4),
            "sparse_share": round(seg_split["sparse"] / (seg_split["sparse"] + seg_split["attn"]), 4),
            "sparse_positions_layers_per_s": round(B * n * Ls / seg_split["sparse"], 1),
            "note": "value = positions * (sparse + attention) layers per second of the whole step "
                    "(one captured graph, when graph); the split times every segment's forward and "
                    "backward call and the sparse weight-gradient call on its own, each over "
                    "calls captured back to back in one graph (graph_timed)"})
    else:
        out["hybrid"].update({
            "sparse_ms_eager": round(sparse / args.steps * 1e3, 4),
            "attention_ms_eager": round(attn / args.steps * 1e3, 4),
            "note": "value = positions * (sparse + attention) layers per second of the whole step; "
                    "the split from eager steps with HIP events around every segment (host "
                    "overhead included)"})
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def run_shared(args, torch, hcmix, inputs, dev):
    """The channel-shared stack at the LM shape: one hcmix_shared_stack_forward
    and one hcmix_shared_stack_backward call per step, replayed as a graph.
    HBM-bound, so its roofline is bytes: the forward kernel reads x_0 and
    writes every layer's output, (L + 1) activations; the backward kernel
    reads dy and every layer input and writes dx, (L + 2) activations, plus
    the L fp32 table gradients (n^2 each).  Each call is timed on its own
    with HIP events around graph replays of calls of it (graph_timed), on the stream
    it runs on."""
    B, n, w, L = 64, 256, 512, 16
    if args.batch > 0:
        B = args.batch
    s = inputs.make_shared_stack(B, n, w, L, True, "bf16", kind="zipf_bytes", seed=0)
    dt = torch.bfloat16
    x0 = torch.from_numpy(s.x).to(dt).to(dev)
    dy = torch.from_numpy(s.dy).to(dt).to(dev)
    tabs = [torch.from_numpy(t).to(dev) for t in s.tables]
    outs = [torch.empty_like(x0) for _ in range(L)]
    dx = torch.empty_like(x0)
    dts = [torch.empty((n, n), dtype=torch.float32, device=dev) for _ in range(L)]
    nbytes = hcmix.load().hcmix_shared_stack_backward_workspace_bytes(B, n, w, L, hcmix.HCMIX_BF16)
    wsp = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    xs = [x0, *outs]

    def fwd():
        hcmix.shared_stack_forward(x0, tabs, s.layers, True, outs=outs)

    def bwd():
        hcmix.shared_stack_backward(xs[:L], tabs, s.layers, dy, True, dx=dx, dtables=dts,
                                    workspace=wsp)

    def step():
        fwd()
        bwd()

    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        step()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        t = max(time.perf_counter() - t0, e0.elapsed_time(e1) / 1e3)
    us = {name: graph_timed(torch, fn, args.kernel_reps) * 1e6
          for name, fn in (("forward", fwd), ("backward", bwd))}
    if args.calib_copy_mb > 0:
        calibration_copy(torch, dev, args.calib_copy_mb)
    act = B * n * w * 2
    bytes_fwd = (L + 1) * act + L * n * 8
    bytes_bwd = (L + 2) * act + L * n * 8 + L * n * n * 4
    entries = {}
    for name, nb, kname in (("forward", bytes_fwd, "shared_fwd_kernel"),
                            ("backward", bytes_bwd, "shared_bwd_kernel + shared_dt_reduce_kernel")):
        gbs = nb / (us[name] * 1e-6) / 1e9
        entries[name] = {"bound": "hbm", "kernel": f"{kname} (one {name} call, all {L} layers)",
                         "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": profiled_traffic(args.workload, kname),
                         "avg_launch_us": round(us[name], 2), "algorithmic_bytes": nb}
    dom = "backward" if us["backward"] >= us["forward"] else "forward"
    out = {
        "metric": METRIC, "value": round(B * n * L * args.steps / t, 1), "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"shared256: {WORKLOADS['shared256']}", "batch": B, "n": n,
                   "width": w, "layers": L, "mode": "causal", "graph": True},
        "pct_hbm": round((bytes_fwd + bytes_bwd) / t * args.steps / 1e9 / PEAK_HBM_GBS * 100, 2),
        "roofline": entries[dom],
        "roofline_" + ("forward" if dom == "backward" else "backward"):
            entries["forward" if dom == "backward" else "backward"],
    }
    if args.cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_shared(s, n, L, args.cpu_windows)
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def run_field(args, torch, hcmix, inputs, dev):
    """The field coupling (Section 3.4) at the window-256 LM shape: T = 8
    applications x_t = C(p_t) x_{t-1} in a chain, each with its own
    coordinates (the force that moves them between applications is the
    model's and stays out), then the backward in reverse (dx chained, dp per
    application); one step = T hcmix_field_forward and T hcmix_field_backward
    calls, replayed as a graph.  Both calls are HBM-bound (about 60 flops per
    byte against the bf16 ridge near 315), so the roofline is bytes: forward
    reads p and x and writes y and two fp32 row statistics; backward reads p,
    x, dy and the statistics and writes dp and dx (the couplings, the fp32
    squared-distance gradient and each window's coordinate table are
    workspace, not algorithmic traffic).  Each application has its own workspace: the
    forward leaves the coordinate tables there and the backward of the same
    application takes them (reuse_table).  Each call is timed on its own with
    graph_timed, on the stream it runs on."""
    B, n, w, c, T = 64, 256, 512, 32, 8
    if args.batch > 0:
        B = args.batch
    x_h, ps_h, dy_h, tau, scaled = inputs.make_field_chain(B, n, w, c, T, seed=0)
    x0 = torch.from_numpy(x_h).to(torch.bfloat16).to(dev)
    dy = torch.from_numpy(dy_h).to(torch.bfloat16).to(dev)
    ps = [torch.from_numpy(p).to(dev) for p in ps_h]
    xs = [x0] + [torch.empty_like(x0) for _ in range(T)]
    ms = [torch.empty((B, n), dtype=torch.float32, device=dev) for _ in range(T)]
    lses = [torch.empty((B, n), dtype=torch.float32, device=dev) for _ in range(T)]
    dps = [torch.empty_like(p) for p in ps]
    gs = [torch.empty_like(x0) for _ in range(T)]
    wsps = [torch.empty(hcmix.field_workspace_bytes(B, n, c), dtype=torch.uint8, device=dev)
            for _ in range(T)]

    def fwd(t):
        hcmix.field_forward(ps[t], xs[t], tau, scaled, y=xs[t + 1], row_mean=ms[t], lse=lses[t],
                            workspace=wsps[t])

    def bwd(t, g):
        hcmix.field_backward(ps[t], xs[t], ms[t], lses[t], g, tau, scaled, dp=dps[t], dx=gs[t],
                             workspace=wsps[t], reuse_table=True)

    def step():
        for t in range(T):
            fwd(t)
        g = dy
        for t in reversed(range(T)):
            bwd(t, g)
            g = gs[t]

    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        step()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        t = max(time.perf_counter() - t0, e0.elapsed_time(e1) / 1e3)
    us = {"forward": graph_timed(torch, lambda: fwd(0), args.kernel_reps) * 1e6,
          "backward": graph_timed(torch, lambda: bwd(0, dy), args.kernel_reps) * 1e6}
    if args.calib_copy_mb > 0:
        calibration_copy(torch, dev, args.calib_copy_mb)
    rows = B * n
    bytes_fwd = rows * (c * 4 + 2 * w * 2 + 2 * 4)
    bytes_bwd = rows * (2 * c * 4 + 3 * w * 2 + 2 * 4)
    # causal products with x or dy: sum over rows of (i + 1) w multiply-adds
    pv_flops = B * n * (n + 1) * w
    entries = {}
    for name, nb, fl, kname in (
            ("forward", bytes_fwd, pv_flops, "field_couple_kernel + field_readout_kernel"),
            ("backward", bytes_bwd, 2 * pv_flops, "field_bwd_rows_kernel + field_bwd_tail_kernel")):
        sec = us[name] * 1e-6
        gbs = nb / sec / 1e9
        entries[name] = {"bound": "hbm", "kernel": f"{kname} (one {name} call)",
                         "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": profiled_traffic(args.workload, kname),
                         "avg_launch_us": round(us[name], 2), "algorithmic_bytes": nb,
                         "mfma_frac_bf16": round(fl / sec / 1e12 / PEAK_BF16_TFLOPS, 4)}
    dom = "backward" if us["backward"] >= us["forward"] else "forward"
    out = {
        "metric": METRIC, "value": round(B * n * T * args.steps / t, 1), "unit": UNIT,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"field256: {WORKLOADS['field256']}", "batch": B, "n": n,
                   "width": w, "coord_dim": c, "applications": T, "tau": tau,
                   "form": "scaled" if scaled else "unscaled", "graph": True},
        "roofline": entries[dom],
        "roofline_" + ("forward" if dom == "backward" else "backward"):
            entries["forward" if dom == "backward" else "backward"],
    }
    if args.cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_field(x_h, ps_h, dy_h, tau, scaled, n, T,
                                                 args.cpu_windows)
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def run_lm_step(args, torch, hcmix, inputs, dev):
    """The lm256 stack inside a whole training step of the byte-level language
    model: embedding (library gather), the 16-layer stack forward, the 256-way
    head with bias and cross-entropy (library kernel: logits, loss and
    dlogits and the bias gradient), the head's weight and input gradients
    (the library's hcmix_head_backward; --head-grad torch runs them as
    PyTorch GEMMs instead, for comparison), the stack backward and the
    embedding's scatter sum (library), replayed as a HIP graph.  value = positions * sparse layers / step time;
    the sparse stack's share of the step is reported beside it."""
    over = {"batch": args.batch} if args.batch > 0 else {}
    cfg = dict(inputs.PRESETS["lm256"], **over)
    s = inputs.make_preset("lm256", **over)
    B, n, w, L = cfg["batch"], cfg["n"], cfg["width"], cfg["num_layers"]
    V = 256
    dt = torch.bfloat16
    rows = B * n
    gen = torch.Generator(device="cpu").manual_seed(3)
    table = (torch.randn(V, w, generator=gen)).to(dt).to(dev)
    head_w = (torch.randn(V, w, generator=gen) / w ** 0.5).to(dt).to(dev)
    head_b = torch.zeros(V, dtype=torch.float32, device=dev)
    tokens = torch.from_numpy(s.tokens.astype("int32")).to(dev)
    targets = torch.from_numpy(s.targets.astype("int32")).to(dev)
    ws = [torch.from_numpy(a).to(dt).to(dev) for a in s.w_self]
    wo = [torch.from_numpy(a).to(dt).to(dev) for a in s.w_off]
    x0 = torch.empty(B, n, w, dtype=dt, device=dev)
    xs_out = [torch.empty_like(x0) for _ in range(L)]
    dx0 = torch.empty_like(x0)
    dws = [torch.empty((w, w), dtype=torch.float32, device=dev) for _ in range(L)]
    dwo = [torch.empty((w, w), dtype=torch.float32, device=dev) for _ in range(L)]
    loss = torch.empty(rows, dtype=torch.float32, device=dev)
    dlogits = torch.empty(rows, V, dtype=dt, device=dev)
    d_table = torch.empty(V, w, dtype=torch.float32, device=dev)
    gx_buf = torch.empty(B, n, w, dtype=dt, device=dev)
    d_bias = torch.empty(V, dtype=torch.float32, device=dev)
    head_ws = torch.empty(hcmix.load().hcmix_head_cross_entropy_workspace_bytes(rows, V),
                          dtype=torch.uint8, device=dev)
    stack_ws = hcmix.alloc_stack_workspace(B, n, w, L, dt, dev)
    emb_ws = torch.empty(hcmix.load().hcmix_embedding_backward_workspace_bytes(rows, w, V),
                         dtype=torch.uint8, device=dev)
    d_head = torch.empty(V, w, dtype=torch.float32, device=dev)
    head_bws = torch.empty(hcmix.load().hcmix_head_backward_workspace_bytes(rows, w, V),
                           dtype=torch.uint8, device=dev)

    def step(times=None):
        ev = []

        def mark():
            if times is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record(stream)
                ev.append(e)
        mark()
        hcmix.embedding_forward(table, tokens, out=x0)
        mark()
        xs = hcmix.stack_forward(x0, ws, wo, s.layers, True, outs=xs_out)
        mark()
        xl = xs[-1].view(rows, w)
        # logits, loss, dlogits and the bias gradient in the library's kernel
        hcmix.head_cross_entropy(xl, head_w, head_b, targets, 1.0 / rows, loss=loss,
                                 dlogits=dlogits, dbias=d_bias, workspace=head_ws)
        if args.head_grad == "library":
            # the head's input and weight gradients in the library's kernels
            hcmix.head_backward(xl, head_w, dlogits, gx=gx_buf.view(rows, w), dw=d_head,
                                workspace=head_bws)
        else:
            # the same as PyTorch GEMMs; the weight gradient's K = rows is split
            # into 16 batched products (one GEMM over all rows leaves the chip idle)
            kch = 16
            torch.bmm(xl.view(kch, rows // kch, w).transpose(1, 2),
                      dlogits.view(kch, rows // kch, V)).sum(0).t()
            torch.matmul(dlogits, head_w, out=gx_buf.view(rows, w))
        gx = gx_buf
        mark()
        hcmix.stack_backward(xs, ws, wo, s.layers, gx, True, dx=dx0, dws=dws, dwo=dwo,
                             workspace=stack_ws)
        mark()
        hcmix.embedding_backward(tokens, dx0, V, dtable=d_table, workspace=emb_ws)
        mark()
        if times is not None:
            times.append(ev)

    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        step()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        t = max(time.perf_counter() - t0, e0.elapsed_time(e1) / 1e3)
        # phase split from eager steps with events between the phases
        per = []
        for _ in range(5):
            step(per)
        torch.cuda.synchronize()
        # the stack's dominant kernels, timed as in the stack-only workload
        kernels = dominant_kernel(args, hcmix, stream, x0, ws, wo, gx_buf, xs_out, [dx0], dws,
                                  dwo, stack_ws, s.layers, B, n, w, L, True)
    if args.calib_copy_mb > 0:
        calibration_copy(torch, dev, args.calib_copy_mb)
    names = ["embedding", "stack_forward", "head_and_cross_entropy", "stack_backward",
             "embedding_backward"]
    phase_ms = {nm: round(sum(ev[i].elapsed_time(ev[i + 1]) for ev in per) / len(per), 4)
                for i, nm in enumerate(names)}
    sparse = phase_ms["stack_forward"] + phase_ms["stack_backward"]
    eager = sum(phase_ms.values())
    flops, nbytes = algorithmic_work(B, n, w, L, True)
    # the two ends: head logits, dlogits x W and dW_head (2 V w flops each per
    # position); bytes: embedding gather (read the row, write x0) and its
    # backward (read dx), head (read x twice, write dlogits, read it twice,
    # write the input gradient)
    flops += rows * 3 * 2 * V * w
    nbytes += rows * (3 * 2 * w + 4 * w + 2 * w + 3 * 2 * V)
    out = {
        "metric": METRIC, "value": round(rows * L * args.steps / t, 1), "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"lm256_step: {WORKLOADS['lm256_step']}"
                               + (f" (batch overridden to {B})" if over else ""), "batch": B,
                   "n": n, "width": w, "layers": L, "vocab": V, "mode": "causal", "graph": True},
        "pct_bf16_peak": round(flops / t * args.steps / 1e12 / PEAK_BF16_TFLOPS * 100, 2),
        "pct_hbm": round(nbytes / t * args.steps / 1e9 / PEAK_HBM_GBS * 100, 2),
    }
    out.update(kernels)
    out["lm_step"] = {"phase_ms_eager": phase_ms,
                      "sparse_share_of_eager_step": round(sparse / eager, 4),
                      "loss_mean": round(float(loss.mean()), 5),
                      "note": "value = positions * sparse layers per second of the whole training "
                              "step (graph replay); phases timed on eager steps with HIP events"}
    if args.cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_lm(s, table, head_w, n, w, L, V, args.cpu_windows)
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def run_decode(args, torch, hcmix, inputs, dev):
    """Incremental decode at the lm256 shape: one hcmix_decode_step per
    position, positions 0..n-1 of a window in order (every window of the batch
    advances one position per step).  A step is one position of all windows
    through all layers; value = windows * layers * steps / time."""
    cfg = dict(inputs.PRESETS["lm256"])
    if args.batch > 0:
        cfg["batch"] = args.batch
    s = inputs.make_preset("lm256", **({"batch": args.batch} if args.batch > 0 else {}))
    B, n, w, L = cfg["batch"], cfg["n"], cfg["width"], cfg["num_layers"]
    dt = torch.bfloat16
    x = torch.from_numpy(s.x).to(dt).to(dev)
    cols = [x[:, p].contiguous() for p in range(n)]
    ws = [torch.from_numpy(a).to(dt).to(dev) for a in s.w_self]
    wo = [torch.from_numpy(a).to(dt).to(dev) for a in s.w_off]
    cache = hcmix.alloc_decode_cache(B, n, w, s.layers, dt, dev)
    y = torch.empty(B, w, dtype=dt, device=dev)
    stream = torch.cuda.current_stream(dev)

    def window(npos):
        for p in range(npos):
            hcmix.decode_step(cols[p], ws, wo, s.layers, n, p, cache, out=y)

    window(n)
    torch.cuda.synchronize()
    steps = max(args.steps, n)          # whole windows
    steps = (steps + n - 1) // n * n

    def timed(run):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(steps // n):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        return max(time.perf_counter() - t0, e0.elapsed_time(e1) / 1e3)

    t_eager = timed(lambda: window(n))
    # one graph holding a whole window: n positions x L layer launches in
    # order (the position is a launch argument), replayed once per window
    graphs = []
    if args.graph:
        side = torch.cuda.Stream(device=dev)
        with torch.cuda.stream(side):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                window(n)
            graphs.append(g)
        torch.cuda.synchronize()

        def replay():
            graphs[0].replay()
        replay()
        torch.cuda.synchronize()
        t_graph = timed(replay)
    t = t_graph if graphs else t_eager
    out = {
        "metric": METRIC, "value": round(B * L * steps / t, 1), "unit": UNIT, "n_gpus": 1,
        "steps": steps, "warmup": n, "ms_per_step": round(t / steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"decode256: {WORKLOADS['decode256']}", "batch": B, "n": n,
                   "width": w, "layers": L, "mode": "causal", "graph": bool(graphs)},
        "decode": {"us_per_position": round(t / steps * 1e6, 2),
                   "us_per_position_eager": round(t_eager / steps * 1e6, 2),
                   "launches_per_position": L,
                   "note": "value from one captured graph per window (n positions x layers "
                           "launches, the position a launch argument); eager launches beside it"},
    }
    if not args.calib_copy_mb:       # counter runs: the calibration copy stays the largest
        out["context"] = device_copy_context(torch, dev)
    print(json.dumps(out), flush=True)
    return 0


def cpu_model() -> str:
    """The host CPU's model name (as lscpu prints it, from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def timed_oracle_legs(run, B, n, L, windows, what, single_threaded=False):
    """Time `run(k)` (the oracle over k windows, every layer, forward and
    backward) on all host threads and on one thread.

    All threads: with windows == 0 the sample is sized to 10-30 s of CPU work
    from a timed pilot of a few windows; when the whole workload takes less
    than that, it is run repeatedly (the sample then says how many passes).
    One thread: one window, repeated until about 5 s have passed (at most
    once more than needed), so the whole baseline stays within about 35 s.
    An oracle that runs on one thread anyway (single_threaded) gets the first
    leg only, reported with one core."""
    import oracle

    passes = 1
    if windows <= 0:
        # a few-window pilot overstates the per-window cost (fewer rows to
        # spread over the threads), so aim above the 10-30 s band's floor
        target = 25.0
        pilot = min(B, 4)
        per_window = run(pilot) / pilot
        windows = max(1, min(B, int(target / max(per_window, 1e-4))))
        if windows == B:
            passes = max(1, min(200, int(round(target / max(per_window * B, 1e-4)))))
    dt, done = 0.0, 0
    while done < passes or (dt < 10.0 and done < 200):   # the pilot may overestimate
        dt += run(windows)
        done += 1
    passes = done
    threads = 1 if single_threaded else oracle.num_threads()
    sample = (f"{windows} of the workload's {B} windows" if windows < B
              else f"all {B} windows") + (f", {passes} passes" if passes > 1 else "")
    out = {"value": round(passes * windows * n * L / dt, 1), "unit": UNIT, "cores": threads,
           "kind": "oracle", "sample": f"{sample}{what}, {dt:.1f} s", "cpu_model": cpu_model(),
           "host_cpus": os.cpu_count()}
    if single_threaded:
        return out
    oracle.set_num_threads(1)
    try:
        dt1, done1 = 0.0, 0
        while dt1 < 5.0 and done1 < 200:
            dt1 += run(1)
            done1 += 1
    finally:
        oracle.set_num_threads(threads)
    out["single_thread"] = {"value": round(done1 * n * L / dt1, 1), "unit": UNIT, "cores": 1,
                            "sample": f"1 window, {done1} passes{what}, {dt1:.1f} s"}
    return out


def cpu_baseline(s, n, w, L, causal, windows):
    """The CPU oracle (plain fp64 loops) on a bounded sample of the same
    workload: windows through every layer, forward and backward, on all host
    threads and on one."""
    import oracle

    def run(k):
        t0 = time.perf_counter()
        xs = oracle.stack_forward(s.x[:k], s.w_self, s.w_off, s.layers, causal)
        oracle.stack_backward(xs, s.w_self, s.w_off, s.layers, s.dy[:k], causal)
        return time.perf_counter() - t0

    return timed_oracle_legs(run, s.x.shape[0], n, L, windows,
                             f", all {L} layers, forward+backward")


def cpu_baseline_lm(s, table, head_w, n, w, L, V, windows):
    """The CPU oracle on a bounded sample of the whole LM step: windows
    through the embedding, every layer, the head and cross-entropy, the head's
    gradients (plain products on dlogits), the stack backward and the
    embedding's scatter sum; all host threads and one thread, as cpu_baseline."""
    import numpy as np

    import oracle
    from oracle import lm_head

    tab = table.float().cpu().numpy().astype(np.float64)
    hw = head_w.float().cpu().numpy().astype(np.float64)
    B = s.tokens.shape[0]

    def run(k):
        t0 = time.perf_counter()
        x = lm_head.embedding_forward(tab, s.tokens[:k])
        xs = oracle.stack_forward(x, s.w_self, s.w_off, s.layers, True)
        xl = xs[-1].reshape(-1, w)
        _, dlog = lm_head.head_cross_entropy(xl, hw, np.zeros(V), s.targets[:k], 1.0 / (B * n))
        _ = dlog.T @ xl, dlog.sum(axis=0)
        gx = (dlog @ hw).reshape(k, n, w)
        dx, _, _ = oracle.stack_backward(xs, s.w_self, s.w_off, s.layers, gx, True)
        lm_head.embedding_backward(s.tokens[:k], dx, V)
        return time.perf_counter() - t0

    return timed_oracle_legs(run, B, n, L, windows,
                             f": embedding, all {L} layers, head and cross-entropy, "
                             "forward+backward")


def cpu_baseline_shared(s, n, L, windows):
    """The channel-shared oracle (oracle/shared_mix.py, float64) on a bounded
    sample of the workload, all host threads and one thread."""
    from oracle import shared_mix

    def run(k):
        t0 = time.perf_counter()
        xs = shared_mix.stack_forward(s.x[:k], s.tables, s.layers, True)
        shared_mix.stack_backward(xs, s.tables, s.layers, s.dy[:k], True)
        return time.perf_counter() - t0

    return timed_oracle_legs(run, s.x.shape[0], n, L, windows,
                             f", all {L} layers, forward+backward (numpy, one thread)",
                             single_threaded=True)


def cpu_baseline_field(x, ps, dy, tau, scaled, n, T, windows):
    """The field oracle (oracle/field.py, float64 numpy) on a bounded sample of
    the workload: windows through all T applications, forward and backward,
    with numpy's BLAS held to one thread."""
    from threadpoolctl import threadpool_limits

    from oracle import field

    def run(k):
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            xs = [x[:k]]
            for t in range(T):
                xs.append(field.forward(ps[t][:k], xs[-1], tau, scaled)[0])
            g = dy[:k]
            for t in reversed(range(T)):
                _, g = field.backward(ps[t][:k], xs[t], g, tau, scaled)
            return time.perf_counter() - t0

    return timed_oracle_legs(run, x.shape[0], n, T, windows,
                             f", all {T} applications, forward+backward (numpy, one thread)",
                             single_threaded=True)


if __name__ == "__main__":
    sys.exit(main())
