"""Benchmark: block-sparse ResNet-50 backbone frames at 2048x1024 on one MI355X.

One step = one sparse frame of the whole hot path: the execution grid is compacted
into the active-block index (bc_build_block_index), then all 53 convolutions and
the max pooling run block-sparsely on the frame's active blocks, each reading its
input buffer (halo from neighbours) and writing its persistent output buffer in
place. Inputs (frame, weights, mask, previous buffers) are resident in HBM before
timing starts; frame 0 of the clip runs on every block, untimed.

Workload: ResNet-50 (stem 7x7/2, max pool, bottlenecks [3,4,6,3], BN folded, ReLU),
random He-normal weights, bf16 channels-last, N(0,1) synthetic 2048x1024x3 frame,
128-px blocks (16x8 grid), clustered mask with round(0.3 * 128) = 38 active blocks.

Printed: one JSON line with the effective TFLOP/s over active blocks (algorithmic
conv FLOPs of the active output pixels / frame time), ms per frame, the roofline
fraction of the dominant kernel (the matrix-core sparse conv, timed per launch with
HIP events on its stream), the frame time at other active fractions, and the CPU
oracle's rate on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--frac", type=float, default=0.3, help="active-block fraction of the timed frames")
    ap.add_argument("--sweep", default="0.1,0.5,1.0", help="extra active fractions timed (comma list, '' for none)")
    ap.add_argument("--no-graph", action="store_true", help="launch layer by layer instead of a HIP graph replay")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=0,
                    help="run only N plain steps (for rocprofv3) and print nothing else")
    return ap.parse_args()


def cpu_baseline(mask):
    """The CPU oracle (dense convolution then masked select, fp64, OpenMP) on a bounded
    sample of the workload: the four convolutions of ResNet-50 layer1.0 (1x1 64->64,
    3x3 64->64, 1x1 64->256, 1x1 64->256 shortcut) at their real 256x512 size with
    the frame's mask. Rate = active-block FLOPs of the sample / oracle time."""
    import numpy as np

    import oracle
    import synth
    r = synth.rng(5)
    h, w = 256, 512
    layers = [(64, 64, 1, False), (64, 64, 3, False), (64, 256, 1, True), (64, 256, 1, False)]
    x = synth.to_storage_bits(synth.normal(r, (1, 64, h, w)), "bf16")
    gh, gw = mask.shape[1:]
    act = int((mask != 0).sum()) / (gh * gw)
    flops = 0.0
    t0 = time.perf_counter()
    for cin, cout, k, res in layers:
        wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), "bf16")
        prev = np.zeros((1, cout, h, w), np.uint16)
        rb = synth.to_storage_bits(synth.normal(r, (1, cout, h, w)), "bf16") if res else None
        oracle.sparse_conv2d(x, wt, mask, prev, "bf16", 1, k // 2, np.zeros(cout, np.float32), rb, True)
        flops += 2.0 * cin * cout * k * k * h * w * act
    dt = time.perf_counter() - t0
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "ResNet-50 layer1.0 (4 convs) at 256x512x64 bf16, dense-then-select in fp64, "
                      f"{int((mask != 0).sum())}/{gh * gw} blocks active; {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    from paper_2108_09376_amd import resnet

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    H, W, BLOCK = 1024, 2048, 128
    net = resnet.SparseResNet(50, H, W, BLOCK, device=dev)
    gh, gw = net.grid
    frame = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_INPUT), (1, H, W, 3)), "bf16")
    x = torch.from_numpy(frame.view(np.int16)).view(torch.bfloat16).to(dev)
    stream = torch.cuda.current_stream()

    def masks_for(frac):
        return synth.frac_mask(synth.SEED_MASK0 + 1, gh, gw, frac)

    net.frame(x, sparse=False)           # frame 0 of the clip: every block
    torch.cuda.synchronize()

    if args.profile_steps:
        net.set_mask(masks_for(args.frac))
        for _ in range(args.profile_steps):
            net.frame(x, sparse=True)
        torch.cuda.synchronize()
        return

    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        net.set_mask(masks_for(args.frac))
        s = torch.cuda.Stream()
        s.wait_stream(stream)
        with torch.cuda.stream(s):
            net.frame(x, sparse=True)     # warm the capture stream
        stream.wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            net.frame(x, sparse=True)
        torch.cuda.synchronize()

    def step():
        if graph is not None:
            graph.replay()
        else:
            net.frame(x, sparse=True)

    def time_frames(frac, steps, warmup):
        net.set_mask(masks_for(frac))
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    mask = masks_for(args.frac)
    active = int(mask.sum())
    ms = time_frames(args.frac, args.steps, args.warmup)
    flops = net.conv_flops(active)
    value = flops / (ms * 1e-3) / 1e12

    sweep = {}
    for f in [float(v) for v in args.sweep.split(",") if v.strip()]:
        sweep[f"{f:g}"] = round(time_frames(f, max(10, args.steps // 2), 3), 4)
    sweep[f"{args.frac:g}"] = round(ms, 4)

    # Per-launch durations of the dominant kernel (sparse conv), HIP events on its stream.
    net.set_mask(mask)
    nl = len(net.layers)
    reps = max(5, args.steps // 5)
    conv_ms = [0.0] * nl
    for rep in range(reps + 2):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nl)]
        from paper_2108_09376_amd import bc
        bc.bc_build_block_index(net.mask, 1, net.grid, net.idx, net.count)
        for i in range(nl):
            ev[i][0].record()
            net.run_layer(i, x, net.idx, net.count)
            ev[i][1].record()
        torch.cuda.synchronize()
        if rep >= 2:
            for i in range(nl):
                conv_ms[i] += ev[i][0].elapsed_time(ev[i][1]) / reps
    conv_idx = [i for i, l in enumerate(net.layers) if l.kind == "conv"]
    conv_total_ms = sum(conv_ms[i] for i in conv_idx)
    achieved = flops / (conv_total_ms * 1e-3) / 1e12
    per_launch_us = conv_total_ms * 1e3 / len(conv_idx)

    out = {
        "metric": "effective TFLOP/s on active blocks + ms/frame at 2048x1024, 30% active",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "ResNet-50 backbone block-sparse frame, 2048x1024x3 bf16, 128-px blocks "
                               "(16x8 grid), clustered mask", "active_blocks": active,
                   "total_blocks": gh * gw, "active_fraction": round(active / (gh * gw), 4),
                   "batch": 1, "hip_graph": graph is not None},
        "conv_gflop_per_frame": round(flops / 1e9, 3),
        "frame_ms_by_active_fraction": sweep,
        "roofline": {"bound": "mfma", "kernel": "sparse conv (k_conv_mfma*, all 53 launches of a frame)",
                     "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 5),
                     "avg_launch_us": round(per_launch_us, 3), "traffic": None},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(mask)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
