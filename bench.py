"""Benchmark: block-sparse ResNet-50 backbone frames at 2048x1024 on one MI355X.

One step = one sparse frame of the whole hot path: the execution grid is compacted
into the active-block index (bc_build_block_index), then all 53 convolutions and
the max pooling run block-sparsely on the frame's active blocks (each block's shortcut
projection shares one launch with its branch's first 1x1 convolution: 49 conv
launches), each reading its
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
    ap.add_argument("--no-gather-scatter", action="store_true")
    ap.add_argument("--no-vendor-dense", action="store_true",
                    help="skip the dense frame through torch's own convolutions")
    ap.add_argument("--no-clip", action="store_true",
                    help="skip the 30-frame clip (ResNet-18 encoder; SwiftNet-18 full step)")
    ap.add_argument("--no-policy-steps", action="store_true",
                    help="skip sampling / frame state / information gain / rewards")
    ap.add_argument("--pmc-frames", type=int, default=0,
                    help="rocprofv3 --pmc helper: a 256 MiB float32 negation (calibration) then N sparse frames "
                         "at --frac launched layer by layer; prints nothing else")
    ap.add_argument("--no-layer-sweep", action="store_true",
                    help="skip the single-layer shapes (256x512x64 3x3; stride-16 C sweep)")
    ap.add_argument("--profile-steps", type=int, default=0,
                    help="run only N plain steps (for rocprofv3) and print nothing else")
    ap.add_argument("--counter-summary", nargs=2, metavar=("COUNTER_CSV", "AGENT_CSV"),
                    help="print the matrix-core / LDS counter table of a rocprofv3 --pmc run")
    ap.add_argument("--pmc-layers", type=int, default=0,
                    help="run only the single-layer sweep, each layer 1 + N times, for a rocprofv3 --pmc run")
    ap.add_argument("--layer-counter-summary", nargs=2, metavar=("COUNTER_CSV", "AGENT_CSV"),
                    help="print the matrix-core / LDS counter table of a --pmc-layers run")
    ap.add_argument("--pmc-gather-scatter", action="store_true",
                    help="run only the standalone gather/scatter cases for a rocprofv3 --pmc run")
    ap.add_argument("--gs-summary", nargs="+", metavar="CSV",
                    help="FETCH_CSV WRITE_CSV [KERNEL_TRACE_CSV]: print the gather/scatter traffic table "
                         "of two rocprofv3 --pmc runs (and rates over the kernel durations of a trace run)")
    ap.add_argument("--cpu-configs", action="store_true",
                    help="time the CPU oracle on configurations 1, 2, 4 and 5 (both modes) and exit")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the HBM-traffic summary of two counter_collection.csv files and exit")
    ap.add_argument("--rocprof-summary", nargs="+", metavar="CSV",
                    help="KERNEL_STATS_CSV [KERNEL_TRACE_CSV FIRST COUNT]: print a text summary of a "
                         "rocprofv3 --stats kernel table (and a window of conv dispatches) and exit")
    return ap.parse_args()


def cpu_model():
    """The host CPU's model name and thread count as the kernel reports them."""
    name, fam, mod = "unknown", "?", "?"
    try:
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k, v = k.strip(), v.strip()
            if k == "model name" and name == "unknown":
                name = v
            elif k == "cpu family" and fam == "?":
                fam = v
            elif k == "model" and mod == "?":
                mod = v
    except OSError:
        pass
    return f"{name} (family {fam}, model {mod}), {os.cpu_count()} logical CPUs"


def cpu_baseline(mask):
    """The CPU oracle (dense convolution then masked select, fp64, OpenMP) on a bounded
    sample of the workload: every convolution of ResNet-50's first two stages (layer1
    and layer2: 23 convs, stride 4 and 8) at their real sizes for a 2048x1024 frame, with
    the frame's mask; each layer gets seeded bf16 inputs of its shape. Rate = the
    sample's active-block FLOPs / oracle time. Beside it, the oracle's only-active mode
    on the same sample (same arithmetic, inactive blocks skipped: the fair sparse CPU
    comparison) and the configuration-1 layer (fp32, two frames) in both modes."""
    import numpy as np

    import oracle
    import synth
    from paper_2108_09376_amd import resnet
    layers = resnet.build_layers(50)
    shapes = resnet.layer_shapes(layers, 1024, 2048)
    r = synth.rng(5)
    gh, gw = mask.shape[1:]
    act = int((mask != 0).sum()) / (gh * gw)
    flops = 0.0
    n = 0
    dt = dt_act = 0.0
    for i, l in enumerate(layers):
        if l.kind != "conv" or not l.name.startswith(("layer1", "layer2")):
            continue
        ih, iw = shapes[l.src][:2]
        oh, ow = shapes[i][:2]
        x = synth.to_storage_bits(synth.normal(r, (1, l.cin, ih, iw)), "bf16")
        wt = synth.to_storage_bits(synth.he_normal(r, l.cout, l.cin, l.k, l.k), "bf16")
        prev = np.zeros((1, l.cout, oh, ow), np.uint16)
        rb = synth.to_storage_bits(synth.normal(r, (1, l.cout, oh, ow)), "bf16") if l.res is not None else None
        args = (x, wt, mask, prev, "bf16", l.stride, l.pad, np.zeros(l.cout, np.float32), rb, l.relu)
        t0 = time.perf_counter()           # the oracle only, not the input generation
        oracle.sparse_conv2d(*args)
        t1 = time.perf_counter()
        oracle.sparse_conv2d_active(*args)
        dt_act += time.perf_counter() - t1
        dt += t1 - t0
        flops += 2.0 * l.cin * l.cout * l.k * l.k * oh * ow * act
        n += 1
    c1 = config1_cpu()
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"ResNet-50 layer1 + layer2 ({n} convs) at their 2048x1024-frame sizes, bf16 "
                      f"values, dense-then-select in fp64, {int((mask != 0).sum())}/{gh * gw} blocks "
                      f"active; {dt:.1f} s",
            "cpu_model": cpu_model(),
            "only_active": {"value": round(flops / dt_act / 1e12, 6), "unit": "TFLOP/s",
                            "seconds": round(dt_act, 2)},
            "config1_us_per_frame": c1,
            "configs_recorded": recorded_cpu_configs()}


def config1_inputs():
    """Configuration 1: NCHW fp32 [1, 16, 64, 128], 3x3 16 -> 16, 8x16 grid of 8x8
    blocks, He-normal weights, N(0, 1) inputs and previous output, two frames with
    independent Bernoulli(0.25) grids."""
    import synth
    r = synth.rng(synth.SEED_INPUT)
    xs = [synth.to_storage_bits(synth.normal(r, (1, 16, 64, 128)), "f32") for _ in range(2)]
    wt = synth.to_storage_bits(synth.he_normal(synth.rng(synth.SEED_WEIGHT0), 16, 16, 3, 3), "f32")
    prev = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_PREV), (1, 16, 64, 128)), "f32")
    masks = [synth.bernoulli_mask(synth.rng(synth.SEED_MASK0 + t), 1, 8, 16, 0.25) for t in range(2)]
    return xs, wt, prev, masks


def config1_cpu():
    """The oracle on configuration 1's two frames (frame 1 on frame 0's output), both
    modes: microseconds per frame."""
    import oracle
    xs, wt, prev, masks = config1_inputs()
    out = {}
    for mode, fn in (("dense_then_select", oracle.sparse_conv2d), ("only_active", oracle.sparse_conv2d_active)):
        y = prev
        t0 = time.perf_counter()
        for x, m in zip(xs, masks):
            y = fn(x, wt, m, y, "f32", 1, 1, None, None, True)
        out[mode] = round((time.perf_counter() - t0) / 2 * 1e6, 1)
    return out


def config1_gpu(torch, bc, dev):
    """Configuration 1 on the GPU (fp32 NCHW path): one frame = index build + the layer,
    captured as a graph of 10 frames; microseconds per frame."""
    import numpy as np
    xs, wt, prev, masks = config1_inputs()
    x = torch.from_numpy(xs[0].view(np.float32)).to(dev)
    w = torch.from_numpy(wt.view(np.float32)).to(dev)
    y = torch.from_numpy(prev.view(np.float32)).to(dev)
    m = torch.from_numpy(masks[0]).to(dev)
    idx = torch.empty(128, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)

    def frame():
        bc.bc_build_block_index(m, 1, (8, 16), idx, cnt)
        bc.bc_sparse_conv2d((3, 3, 1, 1, 1), x, bc.BC_NCHW, w, None, None, y, (8, 16), idx, cnt)

    frame()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(10):
            frame()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return round(e0.elapsed_time(e1) * 1e3 / 100, 2)


CPU_CONFIGS_PROFILE = os.path.join(ROOT, "profiles", "cpu_oracle_configs.txt")


def cpu_configs():
    """The oracle on configurations 1, 2 and 4 (one frame each; configuration 4 every
    one of its 18 layers) and 5 (ResNet-18 on frames 0-3 of the synthetic clip), in
    both modes, on this host's cores. Prints a progress line per item and a summary."""
    import numpy as np

    import oracle
    import synth
    from oracle import network as onet
    lines = [f"host: {cpu_model()}; oracle threads: {oracle.num_threads()}"]

    def emit(s):
        print(s, flush=True)
        lines.append(s)

    def layer(tag, cin, cout, h, w, k, mask, seed):
        r = synth.rng(seed)
        x = synth.to_storage_bits(synth.normal(r, (1, cin, h, w)), "bf16")
        wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), "bf16")
        prev = synth.to_storage_bits(synth.normal(r, (1, cout, h, w)), "bf16")
        args = (x, wt, mask, prev, "bf16", 1, k // 2, np.zeros(cout, np.float32), None, True)
        act = int((mask != 0).sum()) / mask.size
        res = {}
        for mode, fn in (("dense_then_select", oracle.sparse_conv2d), ("only_active", oracle.sparse_conv2d_active)):
            t0 = time.perf_counter()
            fn(*args)
            res[mode] = time.perf_counter() - t0
        fl = 2.0 * cin * cout * k * k * h * w * act
        emit(f"{tag:28s} dense {res['dense_then_select']:8.2f} s  only-active {res['only_active']:8.2f} s  "
             f"active GFLOP {fl / 1e9:8.2f}")
        return res, fl

    c1 = config1_cpu()
    emit(f"config 1 (fp32 3x3 16->16 @64x128, 2 frames): dense {c1['dense_then_select']:.1f} us/frame, "
         f"only-active {c1['only_active']:.1f} us/frame")
    m30 = synth.frac_mask(synth.SEED_MASK0, 8, 16, 0.3)
    layer("config 2 3x3 64->64 @256x512", 64, 64, 256, 512, 3, m30, 2)
    tot = {"dense_then_select": 0.0, "only_active": 0.0}
    tf = 0.0
    for k in (1, 3):
        for cin in (256, 512, 1024):
            for cout in (256, 512, 1024):
                res, fl = layer(f"config 4 {k}x{k} {cin}->{cout} @64x128", cin, cout, 64, 128, k, m30, 4000 + cin + cout + k)
                for m in tot:
                    tot[m] += res[m]
                tf += fl
    emit(f"config 4 all 18 layers: dense {tot['dense_then_select']:.1f} s, only-active {tot['only_active']:.1f} s "
         f"({tf / 1e9:.1f} active GFLOP: {tf / tot['dense_then_select'] / 1e12:.5f} / "
         f"{tf / tot['only_active'] / 1e12:.5f} TFLOP/s)")
    table = onet.resnet_table(18)
    folded = onet.fold_params(table, onet.make_params(table, seed0=1000), "bf16")
    clip = synth.SyntheticClip(synth.SEED_INPUT + 4)
    sh = onet.shapes(table, 1024, 2048)
    for mode in ("dense_then_select", "only_active"):
        prev = [np.zeros((1,) + s_, np.uint16) for s_ in sh]
        ts = []
        for t in range(4):
            x = synth.to_storage_bits(clip.frame(t).transpose(0, 3, 1, 2).copy(), "bf16")
            t0 = time.perf_counter()
            prev = onet.frame(table, folded, x, clip.mask(t), prev, "bf16", only_active=(mode == "only_active"))
            ts.append(time.perf_counter() - t0)
            emit(f"config 5 ResNet-18 frame {t} ({mode}, {clip.mask(t).mean():.3f} active): {ts[-1]:.1f} s")
        emit(f"config 5 {mode}: frames 0-3 {', '.join(f'{v:.1f}' for v in ts)} s, mean {sum(ts) / 4:.1f} s")
    return "\n".join(lines)


def recorded_cpu_configs():
    """The per-configuration oracle timings committed under profiles/ (text lines), or None."""
    try:
        return [l for l in open(CPU_CONFIGS_PROFILE).read().splitlines() if l.startswith(("host", "config"))]
    except OSError:
        return None


def sweep_layers(torch, bc, dev):
    """The single-layer sweep's layers: the stride-4 3x3 64->64 layer (256x512, 32-px
    blocks) and the stride-16 sweep (64x128, 8-px blocks), 1x1 and 3x3 with Cin and Cout
    in {256, 512, 1024} (all nine pairs), on 38 of 128 clustered blocks. Yields (name,
    call, algorithmic FLOPs, algorithmic bytes) per layer, its tensors on the device."""
    import numpy as np

    import synth
    shapes = [("3x3 64->64 @256x512", 64, 64, 256, 512, 3)]
    for cin in (256, 512, 1024):
        for cout in (256, 512, 1024):
            for k in (1, 3):
                shapes.append((f"{k}x{k} {cin}->{cout} @64x128", cin, cout, 64, 128, k))
    mask = synth.frac_mask(synth.SEED_MASK0, 8, 16, 0.3)
    m = torch.from_numpy(mask).to(dev)
    idx = torch.empty(128, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    bc.bc_build_block_index(m, 1, (8, 16), idx, cnt)
    r = synth.rng(synth.SEED_WEIGHT0)
    n_act = int(mask.sum())
    for name, cin, cout, h, w, k in shapes:
        x = torch.from_numpy(synth.to_storage_bits(synth.normal(r, (1, h, w, cin)), "bf16").view(np.int16)).view(torch.bfloat16).to(dev)
        wt = torch.from_numpy(bc.bc_repack_weights(synth.he_normal(r, cout, cin, k, k), bc.BC_BF16).view(np.int16)).view(torch.bfloat16).to(dev)
        b = torch.zeros(cout, dtype=torch.float32, device=dev)
        y = torch.zeros((1, h, w, cout), dtype=torch.bfloat16, device=dev)
        call = (lambda k=k, x=x, wt=wt, b=b, y=y: bc.bc_sparse_conv2d(
            (k, k, 1, k // 2, 1), x, bc.BC_NHWC, wt, b, None, y, (8, 16), idx, cnt))
        fl = 2.0 * cin * cout * k * k * h * w * n_act / mask.size
        # algorithmic bytes: the active blocks' halo tiles, outputs and the weights, once
        bh, bw = h // 8, w // 16
        nb = n_act * ((bh + k - 1) * (bw + k - 1) * cin + bh * bw * cout) * 2 + cout * k * k * cin * 2
        yield name, call, fl, nb


def layer_sweep(torch, bc, dev):
    """Single block-sparse layers at their 2048x1024-frame shapes (sweep_layers), each
    timed as a captured graph of 10 launches; FLOPs are algorithmic (2*Cin*Cout*k*k per
    active output pixel)."""
    out = {}
    for name, call, fl, nb in sweep_layers(torch, bc, dev):
        call()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(10):
                call()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 50
        out[name] = {"us": round(us, 2), "tflops": round(fl / us / 1e6, 1),
                     "frac_of_mfma_peak": round(fl / us / 1e6 / PEAK_BF16_TFLOPS, 4),
                     "bytes": nb, "frac_of_hbm_peak": round(nb / us / 1e3 / PEAK_HBM_GBS, 4)}
        del g
    return out


def pmc_layers(torch, bc, dev, reps):
    """Counter run of the single-layer sweep: every layer of sweep_layers once to warm,
    then `reps` more times, eager, so each dispatch is one layer call."""
    for _, call, _, _ in sweep_layers(torch, bc, dev):
        for _ in range(1 + reps):
            call()
        torch.cuda.synchronize()


def layer_counter_summary(counter_csv, agent_csv):
    """Text summary of a rocprofv3 --pmc run of `bench.py --pmc-layers N` with the
    matrix-core and LDS counters of counter_summary. Per sweep layer, mean over the N
    timed calls: duration, mfma_util (MFMA busy cycles over SIMDs x duration x peak
    clock), rocprof's MfmaUtil / LdsUtil / LdsBankConflict, LDS instructions per
    matrix-core instruction, and the matrix-core FLOPs seen over the algorithmic ones."""
    import csv

    agent = [r for r in csv.DictReader(open(agent_csv)) if r.get("Name", "").startswith("gfx")][0]
    simds, clk = int(agent["Simd_Count"]), float(agent["Max_Engine_Clk_Fcompute"]) * 1e6
    per = {}
    for r in csv.DictReader(open(counter_csv)):
        d = per.setdefault(int(r["Dispatch_Id"]), {
            "name": r["Kernel_Name"],
            "dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    conv = [per[k] for k in sorted(per) if "k_conv_" in per[k]["name"]]
    shapes = [("3x3 64->64 @256x512", 64, 64, 256, 512, 3)]
    for cin in (256, 512, 1024):
        for cout in (256, 512, 1024):
            for k in (1, 3):
                shapes.append((f"{k}x{k} {cin}->{cout} @64x128", cin, cout, 64, 128, k))
    if len(conv) % len(shapes):
        raise SystemExit(f"{counter_csv}: {len(conv)} conv dispatches is not a whole number per layer")
    calls = len(conv) // len(shapes)
    out = [f"device: {simds} SIMDs, peak engine clock {clk / 1e9:.2f} GHz; one 16x16x32 bf16 MFMA "
           f"holds a SIMD's matrix core for 16 cycles, so busy cycles x 16384 / 16 = FLOPs at peak",
           f"{'layer':24s} {'us':>7s} {'mfma_util':>9s} {'MfmaUtil%':>9s} {'LdsUtil%':>8s} "
           f"{'LdsBank%':>8s} {'lds/mfma':>8s} {'flop/algo':>9s}"]
    for j, (name, cin, cout, h, w, k) in enumerate(shapes):
        runs = conv[j * calls + 1:(j + 1) * calls]

        def mean(key):
            return sum(d[key] for d in runs) / len(runs)

        fl = 2.0 * cin * cout * k * k * h * w * 38 / 128
        dur = mean("dur")
        out.append(f"{name:24s} {dur * 1e6:7.2f} {mean('SQ_VALU_MFMA_BUSY_CYCLES') / (simds * dur * clk):9.4f} "
                   f"{mean('MfmaUtil'):9.2f} {mean('LdsUtil'):8.2f} {mean('LdsBankConflict'):8.3f} "
                   f"{mean('SQ_INSTS_LDS') / mean('SQ_INSTS_VALU_MFMA_MOPS_BF16') * 32:8.3f} "
                   f"{mean('SQ_INSTS_VALU_MFMA_MOPS_BF16') * 512 / fl:9.3f}")
    out.append(f"conv_source_sha256={conv_source_sha()}")
    return "\n".join(out)


def vendor_dense_frame(torch, dev, layers):
    """The same ResNet-50 frame dense through torch's own convolutions (the vendor
    library, its default algorithm search), random weights of the same shapes, one
    captured graph per frame: what a dense frame costs without this library."""
    import torch.nn.functional as F
    params = []
    for l in layers:
        if l.kind != "conv":
            params.append(None)
            continue
        w = (torch.randn(l.cout, l.cin, l.k, l.k, device=dev) * (2.0 / (l.cin * l.k * l.k)) ** 0.5)
        params.append((w.to(torch.bfloat16).contiguous(memory_format=torch.channels_last),
                       torch.zeros(l.cout, device=dev, dtype=torch.bfloat16)))
    x = torch.randn(1, 3, 1024, 2048, device=dev).to(torch.bfloat16).contiguous(memory_format=torch.channels_last)

    def frame():
        outs = []
        for l, p in zip(layers, params):
            src = x if l.src < 0 else outs[l.src]
            if l.kind == "pool":
                y = F.max_pool2d(src, l.k, l.stride, l.pad)
            else:
                y = F.conv2d(src, p[0], p[1], stride=l.stride, padding=l.pad)
                if l.res is not None:
                    y = y + outs[l.res]
                if l.relu:
                    y = F.relu(y)
            outs.append(y)
        return outs[-1]

    for _ in range(3):
        frame()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        frame()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    del g
    return e0.elapsed_time(e1) / 10


def measured_ceilings(torch, dev):
    """Context for the roofline denominators (the published peaks stay the reference):
    torch's bf16 matrix product through the vendor library on an 8192-cube (the largest
    dense contraction rate a library reaches here), and torch's device copy of 1 GiB."""
    a = torch.randn((8192, 8192), device=dev).to(torch.bfloat16)
    b = torch.randn((8192, 8192), device=dev).to(torch.bfloat16)
    c = torch.empty((8192, 8192), device=dev, dtype=torch.bfloat16)
    src = torch.empty(1 << 29, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def per_call_ms(fn, reps):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    gemm_ms = per_call_ms(lambda: torch.matmul(a, b, out=c), 20)
    copy_ms = per_call_ms(lambda: dst.copy_(src), 20)
    gemm_tf = 2 * 8192 ** 3 / (gemm_ms * 1e-3) / 1e12
    copy_gbs = 2 * src.numel() * 2 / (copy_ms * 1e-3) / 1e9
    del a, b, c, src, dst
    return {"bf16_gemm_8192_TFLOPs": round(gemm_tf, 1),
            "bf16_gemm_frac_of_peak": round(gemm_tf / PEAK_BF16_TFLOPS, 3),
            "copy_1GiB_GBps": round(copy_gbs, 1),
            "copy_frac_of_peak": round(copy_gbs / PEAK_HBM_GBS, 3)}


def gather_scatter(torch, bc, dev):
    """Standalone halo gather and block scatter on the 256x512 stride-4 map of a
    2048x1024 frame (32-px blocks, 38 of 128 active, 3x3 halo), C = 64 and 256, bf16.
    Algorithmic bytes: gather reads and writes every halo tile element once, scatter
    reads and writes every block element once. 'warm': graph of 10 launches (inputs
    can stay in the 256 MB last-level cache); 'cold': each launch follows a 512 MiB
    read that evicts the caches (graph-differenced, see below). 'plain_copy': torch's
    contiguous device copy of the gather's byte count, timed the same way: what one
    launch can move at this size."""
    import numpy as np

    import synth
    mask = synth.frac_mask(synth.SEED_MASK0, 8, 16, 0.3)
    n_act = int(mask.sum())
    m = torch.from_numpy(mask).to(dev)
    idx = torch.empty(128, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    bc.bc_build_block_index(m, 1, (8, 16), idx, cnt)
    idx_all = torch.empty(128, dtype=torch.int32, device=dev)
    cnt_all = torch.empty(1, dtype=torch.int32, device=dev)
    bc.bc_build_block_index(torch.ones((1, 8, 16), dtype=torch.uint8, device=dev), 1, (8, 16), idx_all, cnt_all)
    flush = torch.ones((4096, 32768), dtype=torch.float32, device=dev)   # 512 MiB
    flush_out = torch.empty(4096, dtype=torch.float32, device=dev)
    out = {}
    for c in (64, 256):
        x = torch.randn((1, 256, 512, c), device=dev).to(torch.bfloat16)
        packed = torch.empty((128, 34, 34, c), dtype=torch.bfloat16, device=dev)
        blocks = torch.randn((128, 32, 32, c), device=dev).to(torch.bfloat16)
        dst = torch.empty_like(x)
        # the ceiling at this size: torch's device copy of the gather's bytes (one
        # contiguous read and write of the active tiles' size)
        csrc = torch.empty(n_act * 34 * 34 * c, dtype=torch.bfloat16, device=dev).normal_()
        cdst = torch.empty_like(csrc)
        ops = {
            "gather": (lambda: bc.bc_gather_halo(x, bc.BC_NHWC, (8, 16), (3, 3, 1, 1, 0), 0.0, idx, cnt, packed),
                       2 * n_act * 34 * 34 * c * 2),
            "scatter": (lambda: bc.bc_scatter_blocks(blocks, idx, cnt, (8, 16), dst, bc.BC_NHWC),
                        2 * n_act * 32 * 32 * c * 2),
            "plain_copy": (lambda: cdst.copy_(csrc), 2 * n_act * 34 * 34 * c * 2),
        }
        if c == 256:
            # every block (150 MB moved): the kernels' rate where launch latency is small
            asrc = torch.empty(128 * 34 * 34 * c, dtype=torch.bfloat16, device=dev).normal_()
            adst = torch.empty_like(asrc)
            ops["gather_all_blocks"] = (
                lambda: bc.bc_gather_halo(x, bc.BC_NHWC, (8, 16), (3, 3, 1, 1, 0), 0.0, idx_all, cnt_all, packed),
                2 * 128 * 34 * 34 * c * 2)
            ops["scatter_all_blocks"] = (
                lambda: bc.bc_scatter_blocks(blocks, idx_all, cnt_all, (8, 16), dst, bc.BC_NHWC),
                2 * 128 * 32 * 32 * c * 2)
            ops["plain_copy_all_blocks"] = (lambda: adst.copy_(asrc), 2 * 128 * 34 * 34 * c * 2)
        for name, (fn, nbytes) in ops.items():
            fn()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(10):
                    fn()
            g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(5):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            warm = e0.elapsed_time(e1) * 1e3 / 50
            # Cold: a graph of 5 x (cache-evicting read of 512 MiB, op) minus a graph of
            # the 5 reads alone, so launch latency is amortised as in a captured frame.
            # The eviction only reads (a row-wise max into 16 KB), so it leaves no dirty
            # lines whose write-back the measured op would pay for.
            def timed(with_op):
                gg = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gg):
                    for _ in range(5):
                        torch.amax(flush, dim=1, out=flush_out)
                        if with_op:
                            fn()
                gg.replay()
                torch.cuda.synchronize()
                ts = []
                for _ in range(3):
                    e0.record()
                    gg.replay()
                    e1.record()
                    torch.cuda.synchronize()
                    ts.append(e0.elapsed_time(e1) * 1e3 / 5)
                del gg
                return float(np.median(ts))
            cold_us = timed(True) - timed(False)
            out[f"{name}_C{c}"] = {"bytes": nbytes, "warm_us": round(warm, 2),
                                   "warm_GBps": round(nbytes / warm / 1e3, 1),
                                   "cold_us": round(cold_us, 2),
                                   "cold_GBps": round(nbytes / cold_us / 1e3, 1),
                                   "cold_frac_of_hbm_peak": round(nbytes / cold_us / 1e3 / PEAK_HBM_GBS, 3)}
            hb = (recorded_gs_bytes() or {}).get(f"{name}_C{c}")
            if hb is not None:
                # HBM bytes the counters saw for one cold launch, over the same cold time
                out[f"{name}_C{c}"].update({"counter_bytes": round(hb), "counter_GBps_cold": round(hb / cold_us / 1e3, 1),
                                            "counter_frac_of_hbm_peak": round(hb / cold_us / 1e3 / PEAK_HBM_GBS, 3)})
            del g
    return out


GS_CASES = (("C64", 64, False), ("C256", 256, False), ("all_blocks_C256", 256, True))
GS_PROFILE = os.path.join(ROOT, "profiles", "gather_scatter_traffic_256x512_bf16.txt")
GS_SOURCES = ("paper_2108_09376_amd/csrc/k_gather_scatter.hip",)


def gs_source_sha():
    """Hash of the gather/scatter kernel code (code_sha)."""
    return code_sha(GS_SOURCES)


def gs_algo_bytes(c, all_blocks, n_act=38):
    n = 128 if all_blocks else n_act
    return {"gather": 2 * n * 34 * 34 * c * 2, "scatter": 2 * n * 32 * 32 * c * 2}


def pmc_gather_scatter(torch, bc, dev, reps=3):
    """Counter runs of the standalone gather and scatter (rocprofv3 --pmc FETCH_SIZE,
    then WRITE_SIZE): the calibration negation (256 MiB read, 256 MiB written), then
    `reps` repetitions of gather / scatter on the tensors of gather_scatter() for C = 64,
    C = 256 and C = 256 with every block, each op after a 512 MiB cache-evicting read."""
    import synth
    mask = synth.frac_mask(synth.SEED_MASK0, 8, 16, 0.3)
    m = torch.from_numpy(mask).to(dev)
    idx = torch.empty(128, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    bc.bc_build_block_index(m, 1, (8, 16), idx, cnt)
    idx_all = torch.arange(128, dtype=torch.int32, device=dev)
    cnt_all = torch.full((1,), 128, dtype=torch.int32, device=dev)
    a0 = torch.ones(64 << 20, dtype=torch.float32, device=dev)
    a1 = torch.empty_like(a0)
    torch.cuda.synchronize()
    torch.neg(a0, out=a1)
    torch.cuda.synchronize()
    del a0, a1
    flush = torch.ones((4096, 32768), dtype=torch.float32, device=dev)
    flush_out = torch.empty(4096, dtype=torch.float32, device=dev)
    tens = {}
    for c in (64, 256):
        tens[c] = (torch.randn((1, 256, 512, c), device=dev).to(torch.bfloat16),
                   torch.empty((128, 34, 34, c), dtype=torch.bfloat16, device=dev),
                   torch.randn((128, 32, 32, c), device=dev).to(torch.bfloat16),
                   torch.empty((1, 256, 512, c), dtype=torch.bfloat16, device=dev))
    torch.cuda.synchronize()
    for _ in range(reps):
        for _, c, allb in GS_CASES:
            x, packed, blocks, dst = tens[c]
            i, n = (idx_all, cnt_all) if allb else (idx, cnt)
            torch.amax(flush, dim=1, out=flush_out)
            bc.bc_gather_halo(x, bc.BC_NHWC, (8, 16), (3, 3, 1, 1, 0), 0.0, i, n, packed)
            torch.amax(flush, dim=1, out=flush_out)
            bc.bc_scatter_blocks(blocks, i, n, (8, 16), dst, bc.BC_NHWC)
    torch.cuda.synchronize()


def gs_summary(fetch_csv, write_csv, trace_csv=None):
    """Text summary of the two counter runs of pmc_gather_scatter: calibrated FETCH and
    WRITE bytes per gather / scatter dispatch against the algorithmic bytes; with the
    kernel trace of a third run of the same command, each op's median kernel duration
    and the counters' bytes over it (GB/s and fraction of the 8 TB/s HBM peak)."""
    import csv
    res = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            rows[d] = (r["Kernel_Name"], rows.get(d, (None, 0.0))[1] + float(r["Counter_Value"]))
        seq = [rows[d] for d in sorted(rows)]
        cal = [v for n, v in seq if "neg" in n.lower()]
        factor = (256 << 10) / cal[-1]
        ops = [v * factor * 1024 for n, v in seq if "k_gather_" in n or "k_scatter_" in n]
        if len(ops) % 6:
            raise SystemExit(f"{path}: {len(ops)} gather/scatter dispatches is not a whole number of repetitions")
        res[counter] = (factor, [ops[i:i + 6] for i in range(0, len(ops), 6)])
    out = [f"calibration factors: FETCH_SIZE {res['FETCH_SIZE'][0]:.4f}, WRITE_SIZE {res['WRITE_SIZE'][0]:.4f}",
           f"{'op':26s} {'fetch_MB':>9s} {'write_MB':>9s} {'hbm_MB':>9s} {'algo_MB':>9s} {'ratio':>6s}"]
    kv = []
    for k, (tag, c, allb) in enumerate(GS_CASES):
        algo = gs_algo_bytes(c, allb)
        for j, op in enumerate(("gather", "scatter")):
            col = 2 * k + j
            f = sum(r[col] for r in res["FETCH_SIZE"][1]) / len(res["FETCH_SIZE"][1])
            w = sum(r[col] for r in res["WRITE_SIZE"][1]) / len(res["WRITE_SIZE"][1])
            out.append(f"{op + '_' + tag:26s} {f / 1e6:9.3f} {w / 1e6:9.3f} {(f + w) / 1e6:9.3f} "
                       f"{algo[op] / 1e6:9.3f} {(f + w) / algo[op]:6.2f}")
            kv.append(f"hbm_bytes_{op}_{tag}={f + w:.0f}")
    if trace_csv:
        tr = [r for r in csv.DictReader(open(trace_csv))
              if "k_gather_" in r["Kernel_Name"] or "k_scatter_" in r["Kernel_Name"]]
        tr.sort(key=lambda r: int(r["Start_Timestamp"]))
        out.append("kernel durations (trace run, each op after a 512 MiB cache-evicting read; median of "
                   f"{len(tr) // 6} repetitions) and counter bytes over them:")
        for k, (tag, c, allb) in enumerate(GS_CASES):
            for j, op in enumerate(("gather", "scatter")):
                ds = sorted((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
                            for r in tr[2 * k + j::6])
                us = ds[len(ds) // 2]
                hb = float(dict(x.split("=") for x in kv)[f"hbm_bytes_{op}_{tag}"])
                out.append(f"  {op + '_' + tag:26s} {us:7.2f} us  {hb / us / 1e3:8.1f} GB/s  "
                           f"{hb / us / 1e3 / PEAK_HBM_GBS:5.3f} of HBM peak")
    out += kv
    out.append(f"gs_source_sha256={gs_source_sha()}")
    return "\n".join(out)


def recorded_gs_bytes():
    """Counter HBM bytes per gather / scatter case from the committed summary (None if
    missing or taken on other kernel sources)."""
    try:
        kv = dict(l.split("=", 1) for l in open(GS_PROFILE).read().splitlines() if "=" in l
                  and " " not in l.split("=", 1)[0])
    except OSError:
        return None
    if kv.get("gs_source_sha256") != gs_source_sha():
        return None
    return {k[len("hbm_bytes_"):]: float(v) for k, v in kv.items() if k.startswith("hbm_bytes_")}


def policy_steps(torch, bc, dev):
    """The steps around the network at the workload's sizes (2048x1024 frame, 8x16 grid
    of 128-px blocks, 38 blocks active where a grid is given), each timed as a captured
    graph of 10 launches (5 replays):
      sample_grid       execution decisions from 128 block probabilities + index
      frame_state       executed blocks of the bf16 RGB frame copied into the state;
                        algorithmic bytes = 38 blocks x 128x128x3 x 2 B, read + written
      seg_information_gain  19-class fp32 scores of frame t and t-1 (2 x 159 MB read,
                        more than the 256 MB last-level cache holds), per-pixel KL and
                        block max; algorithmic bytes = both score maps once
      block_rewards     rewards, cost, moving average and loss over 128 blocks
      seg_information_gain_nhwc  the segmentation network's own output: bf16 scores at
                        stride 4 (512x256), 19 classes in 64 channels; algorithmic bytes
                        = the 19 class scores of both maps once; line bytes = the
                        128-byte lines that hold them (all 64 channels), fetched whole
      upsample_add      the decoder's largest merge (128x256 -> 256x512, 128 channels,
                        bf16, skip added, 38 blocks); algorithmic bytes = the active
                        blocks' coarse tiles with their one-pixel halo and skip read
                        once, the output blocks written once
      policy_forward    the policy network on a 2048x1024 frame (random init): S_t
                        assembly, eleven dense convolutions, the block probabilities;
                        FLOPs = 2 x its MACs
      policy_update     its online update at that forward pass: REINFORCE gradient of
                        the logits, the reverse pass (ReLU masks, weight, bias and
                        input gradients of every layer) and one RMSprop step"""
    import numpy as np

    import synth
    r = synth.rng(7)
    prob = torch.from_numpy(synth.block_probabilities(r, 1, 8, 16)).to(dev)
    mask = torch.empty((1, 8, 16), dtype=torch.uint8, device=dev)
    idx = torch.empty(128, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    m38 = torch.from_numpy(synth.frac_mask(synth.SEED_MASK0 + 1, 8, 16, 0.3)).to(dev)
    idx38 = torch.empty(128, dtype=torch.int32, device=dev)
    cnt38 = torch.empty(1, dtype=torch.int32, device=dev)
    bc.bc_build_block_index(m38, 1, (8, 16), idx38, cnt38)
    frame = torch.randn((1, 1024, 2048, 3), device=dev).to(torch.bfloat16)
    state = torch.zeros_like(frame)
    lt = torch.from_numpy(synth.seg_logits(r, 1, 19, 1024, 2048)).to(dev)
    lp = (lt + 0.1 * torch.randn_like(lt)).contiguous()
    ig = torch.empty((1, 8, 16), dtype=torch.float32, device=dev)
    lt4 = torch.randn((1, 256, 512, 64), device=dev).mul_(4).to(torch.bfloat16)
    lp4 = (lt4.float() + 0.1 * torch.randn_like(lt4, dtype=torch.float32)).to(torch.bfloat16)
    coarse = torch.randn((1, 128, 256, 128), device=dev).to(torch.bfloat16)
    skip = torch.randn((1, 256, 512, 128), device=dev).to(torch.bfloat16)
    upout = torch.zeros_like(skip)
    mavg = torch.full((1,), 0.3, device=dev)
    reward = torch.empty((1, 8, 16), device=dev)
    cost = torch.empty(1, device=dev)
    loss = torch.empty(1, device=dev)
    ops = {
        "sample_grid": (lambda: bc.bc_sample_execution_grid(prob, (8, 16), 2021, 5, mask, idx, cnt), None),
        "frame_state": (lambda: bc.bc_update_frame_state(frame, state, bc.BC_NHWC, (8, 16), idx38, cnt38),
                        2 * 38 * 128 * 128 * 3 * 2),
        "seg_information_gain": (lambda: bc.bc_seg_information_gain(lt, lp, (8, 16), ig),
                                 2 * 19 * 1024 * 2048 * 4),
        "block_rewards": (lambda: bc.bc_block_rewards(ig, mask, prob, (8, 16), 0.3, 5.0, 0.9, mavg, reward,
                                                      cost, loss), None),
        "seg_information_gain_nhwc": (lambda: bc.bc_seg_information_gain(lt4, lp4, (8, 16), ig, classes=19,
                                                                         layout=bc.BC_NHWC),
                                      2 * 19 * 256 * 512 * 2),
        "upsample_add": (lambda: bc.bc_sparse_upsample_add(coarse, bc.BC_NHWC, skip, upout, (8, 16), 0,
                                                           idx38, cnt38),
                         38 * 128 * 2 * ((16 + 2) * (16 + 2) + 2 * 32 * 32)),
    }
    from paper_2108_09376_amd import resnet
    pnet = resnet.PolicyNet(1024, 2048, device=dev)
    scores = torch.randn((1, 256, 512, 64), device=dev).to(torch.bfloat16)
    ops["policy_forward"] = (lambda: pnet.forward(frame, state, scores, mask), None)
    ops["policy_update"] = (lambda: pnet.train_step(reward, mask, prob), None)
    out = {}
    for name, (fn, nbytes) in ops.items():
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(10):
                fn()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 50
        row = {"us": round(us, 2)}
        if nbytes:
            row.update({"bytes": nbytes, "GBps": round(nbytes / us / 1e3, 1),
                        "frac_of_hbm_peak": round(nbytes / us / 1e3 / PEAK_HBM_GBS, 3)})
        if name == "seg_information_gain_nhwc":
            # every pixel's 19 class scores lie in one 128-byte line of its 64 channels:
            # both maps' lines are fetched whole
            lines = 2 * 256 * 512 * 128
            row.update({"line_bytes": lines, "line_GBps": round(lines / us / 1e3, 1),
                        "line_frac_of_hbm_peak": round(lines / us / 1e3 / PEAK_HBM_GBS, 3)})
        if name == "policy_forward":
            row.update({"gmac": round(pnet.macs() / 1e9, 3),
                        "tflops": round(2 * pnet.macs() / us / 1e6, 1)})
        out[name] = row
        del g
    return out


def resnet18_clip(torch, dev, frames=30):
    """ResNet-18 encoder (random init, bf16) on a 30-frame synthetic 2048x1024 clip:
    moving textured rectangles over a smooth background, execution grid = blocks
    touched by an object at t or t-1, frame 0 on every block. Frame 0 runs eagerly;
    every later frame replays one captured sparse-frame graph (block index built inside
    it) after the frame's image and grid are copied into the graph's fixed device
    buffers. Returns mean ms over frames 1..29 and the mean active fraction."""
    import numpy as np

    import synth
    from paper_2108_09376_amd import resnet
    clip = synth.SyntheticClip(synth.SEED_INPUT + 4)
    net = resnet.SparseResNet(18, 1024, 2048, 128, device=dev)
    x = torch.empty((1, 1024, 2048, 3), dtype=torch.bfloat16, device=dev)

    def load(t):
        img = synth.to_storage_bits(clip.frame(t), "bf16")
        x.copy_(torch.from_numpy(img.view(np.int16)).view(torch.bfloat16))
        mask = clip.mask(t)
        net.set_mask(mask)
        torch.cuda.synchronize()
        return mask

    load(0)
    net.frame(x, sparse=False)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        net.frame(x, sparse=True)
    times, fracs = [], []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    load(0)
    net.frame(x, sparse=False)           # the capture did not run; restart the clip
    for t in range(1, frames):
        mask = load(t)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
        fracs.append(float(mask.mean()))
    flops = sum(net.conv_flops(int(round(f * 128))) for f in fracs) / len(fracs)
    ms = float(np.mean(times))
    return {"frames": frames, "mean_ms_per_sparse_frame": round(ms, 4),
            "mean_active_fraction": round(float(np.mean(fracs)), 4),
            "effective_TFLOPs": round(flops / (ms * 1e-3) / 1e12, 2),
            "launch": "one HIP graph replay per sparse frame"}


def swiftnet_clip_step(torch, bc, dev, frames=30, seed=2021):
    """The whole BlockCopy step per frame on the same 30-frame clip, with the SwiftNet-18
    segmentation network (ResNet-18 encoder + decoder, 19 classes, random init, bf16):
      1. execution grid sampled from the policy's block probabilities, index built
         (bc_sample_execution_grid);
      2. frame state: executed blocks of the RGB frame copied (bc_update_frame_state);
      3. the previous class scores of the blocks about to run saved
         (bc_update_frame_state with the index);
      4. the sparse network on the sampled index (42 layers incl. 3 upsample merges);
      5. information gain of the stride-4 scores (19 of 64 channels) against the saved
         ones on the executed blocks, 0 elsewhere (bc_seg_information_gain with the grid);
      6. rewards, cost, moving average and REINFORCE loss (bc_block_rewards).
    The policy network is not part of the step: its stand-in output is p = 1 on the
    blocks the clip's objects touch at t or t-1 and 0.05 elsewhere (exploration),
    copied in with the frame. One HIP graph replay per frame; the graph fixes the
    generator's counter, so frames differ through their probabilities only. Also timed:
    the network alone (step 4) on the same grids, and the steps around it (1-3, 5, 6)
    alone, each replayed as its own graph."""
    import numpy as np

    import synth
    from paper_2108_09376_amd import resnet
    clip = synth.SyntheticClip(synth.SEED_INPUT + 4)
    net = resnet.SparseSwiftNet(18, 1024, 2048, 128, device=dev)
    grid = net.grid
    gh, gw = grid
    x = torch.empty((1, 1024, 2048, 3), dtype=torch.bfloat16, device=dev)
    state = torch.empty_like(x)
    prob = torch.empty((1, gh, gw), dtype=torch.float32, device=dev)
    mask = torch.empty((1, gh, gw), dtype=torch.uint8, device=dev)
    idx = torch.empty(gh * gw, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    prev_logits = torch.empty_like(net.logits)
    ig = torch.empty((1, gh, gw), dtype=torch.float32, device=dev)
    mavg = torch.full((1,), 0.3, device=dev)
    reward = torch.empty((1, gh, gw), device=dev)
    cost, loss = torch.empty(1, device=dev), torch.empty(1, device=dev)

    def load(t):
        img = synth.to_storage_bits(clip.frame(t), "bf16")
        x.copy_(torch.from_numpy(img.view(np.int16)).view(torch.bfloat16))
        prob.copy_(torch.from_numpy(np.where(clip.mask(t) != 0, 1.0, 0.05).astype(np.float32)))
        torch.cuda.synchronize()

    def before():
        bc.bc_sample_execution_grid(prob, grid, seed, 1, mask, idx, cnt)
        bc.bc_update_frame_state(x, state, bc.BC_NHWC, grid, idx, cnt)
        bc.bc_update_frame_state(net.logits, prev_logits, bc.BC_NHWC, grid, idx, cnt)

    def network():
        net.frame(x, sparse=True, index=(idx, cnt))

    def after():
        bc.bc_seg_information_gain(net.logits, prev_logits, grid, ig, classes=net.classes,
                                   layout=bc.BC_NHWC, mask=mask)
        bc.bc_block_rewards(ig, mask, prob, grid, 0.3, 5.0, 0.9, mavg, reward, cost, loss)

    def restart():
        load(0)
        net.frame(x, sparse=False)        # frame 0: every block
        state.copy_(x)
        torch.cuda.synchronize()

    restart()
    graphs = {}
    for name, fns in (("step", (before, network, after)), ("network", (network,)),
                      ("around", (before, after))):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for fn in fns:
                fn()
        graphs[name] = g
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res = {}
    for name in ("step", "network", "around"):
        restart()                         # the captures ran nothing; every pass starts the clip anew
        times, fracs = [], []
        for t in range(1, frames):
            load(t)
            if name == "network":         # the grid the step would sample, outside the timing
                bc.bc_sample_execution_grid(prob, grid, seed, 1, mask, idx, cnt)
            e0.record()
            graphs[name].replay()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
            fracs.append(float(mask.float().mean().item()))
        res[name] = (float(np.mean(times)), float(np.mean(fracs)))
    ms, frac = res["step"]
    flops = net.conv_flops(int(round(frac * gh * gw)))
    return {"frames": frames, "network": "SwiftNet-18 (ResNet-18 encoder + 3-level decoder), 19 classes",
            "mean_ms_per_step": round(ms, 4), "mean_ms_network_only": round(res["network"][0], 4),
            "mean_ms_steps_around_network": round(res["around"][0], 4),
            "mean_active_fraction": round(frac, 4),
            "effective_TFLOPs_network_in_step": round(flops / (ms * 1e-3) / 1e12, 2),
            "launch": "one HIP graph replay per step"}


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "sparse_conv_traffic_resnet50_2048x1024_active0.3.txt")
MFMA_PROFILE = os.path.join(ROOT, "profiles", "sparse_conv_mfma_lds_resnet50_2048x1024_active0.3.txt")
CONV_SOURCES = ("paper_2108_09376_amd/csrc/k_conv_mfma.hip", "paper_2108_09376_amd/csrc/bc_internal.h")


def code_sha(files):
    """SHA-256 over the code of C/C++/HIP sources: comments and blank lines are removed,
    so a change of wording leaves it alone and any change of code moves it."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in files:
        t = open(os.path.join(ROOT, f)).read()
        t = re.sub(r"/\*.*?\*/", "", t, flags=re.S)
        t = re.sub(r"//[^\n]*", "", t)
        h.update("\n".join(l.rstrip() for l in t.splitlines() if l.strip()).encode())
    return h.hexdigest()[:16]


def conv_source_sha():
    """Hash of the sparse-conv kernel code: counters taken on other code are stale."""
    return code_sha(CONV_SOURCES)


def pmc_summary(fetch_csv, write_csv):
    """Text summary of two rocprofv3 --pmc runs of `bench.py --pmc-frames N` (FETCH_SIZE,
    then WRITE_SIZE; KiB per dispatch). Both counters are scaled by what they read for
    the calibration kernel (float32 negation of 64 Mi elements: 256 MiB read, 256 MiB
    written). Sparse-conv dispatches are grouped into frames of 53 launches; the first
    frame runs every block, the others the 38-block grid."""
    import csv

    from paper_2108_09376_amd import resnet

    def load(path, counter):
        per = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            name, v = r["Kernel_Name"], float(r["Counter_Value"])
            per[d] = (name, per.get(d, (name, 0.0))[1] + v)
        return [per[d] for d in sorted(per)]

    out = []
    res = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = load(path, counter)
        cal = [v for n, v in rows if "neg" in n.lower()]
        if not cal:
            raise SystemExit(f"{path}: no calibration (neg) dispatch found")
        factor = (256 << 10) / cal[-1]
        conv = [v * factor * 1024 for n, v in rows if "k_conv_" in n]
        if len(conv) % 53:
            raise SystemExit(f"{path}: {len(conv)} conv dispatches is not a whole number of frames")
        frames = [conv[i:i + 53] for i in range(0, len(conv), 53)]
        res[counter] = (factor, cal[-1], frames)
    layers = resnet.build_layers(50)
    shapes = resnet.layer_shapes(layers, 1024, 2048)
    algo = [b for b in resnet.conv_algo_bytes(layers, shapes, (8, 16), 38) if b is not None]
    algo_full = [b for b in resnet.conv_algo_bytes(layers, shapes, (8, 16), 128) if b is not None]
    names = [l.name for l in layers if l.kind == "conv"]
    f_fac, f_raw, f_frames = res["FETCH_SIZE"]
    w_fac, w_raw, w_frames = res["WRITE_SIZE"]
    sparse_f = [sum(fr[i] for fr in f_frames[1:]) / len(f_frames[1:]) for i in range(53)]
    sparse_w = [sum(fr[i] for fr in w_frames[1:]) / len(w_frames[1:]) for i in range(53)]
    out.append(f"calibration: FETCH_SIZE read {f_raw:.0f} KiB for 262144 KiB (factor {f_fac:.4f}); "
               f"WRITE_SIZE read {w_raw:.0f} KiB for 262144 KiB (factor {w_fac:.4f})")
    out.append(f"{'layer':24s} {'fetch_MB':>9s} {'write_MB':>9s} {'hbm_MB':>9s} {'algo_MB':>9s} {'ratio':>6s}")
    for i in range(53):
        tot = sparse_f[i] + sparse_w[i]
        out.append(f"{names[i]:24s} {sparse_f[i] / 1e6:9.3f} {sparse_w[i] / 1e6:9.3f} {tot / 1e6:9.3f} "
                   f"{algo[i] / 1e6:9.3f} {tot / algo[i]:6.2f}")
    tf, tw_, ta = sum(sparse_f), sum(sparse_w), sum(algo)
    full = sum(f_frames[0]) + sum(w_frames[0])
    out.append(f"sparse frame (38/128 blocks): fetch {tf / 1e6:.1f} MB, write {tw_ / 1e6:.1f} MB, "
               f"total {(tf + tw_) / 1e6:.1f} MB vs algorithmic {ta / 1e6:.1f} MB (x{(tf + tw_) / ta:.2f})")
    out.append(f"full frame (128/128 blocks): total {full / 1e6:.1f} MB vs algorithmic "
               f"{sum(algo_full) / 1e6:.1f} MB (x{full / sum(algo_full):.2f})")
    out.append(f"traffic_bytes_per_conv_launch={(tf + tw_) / 53:.0f}")
    out.append(f"algo_bytes_per_conv_launch={ta / 53:.0f}")
    out.append(f"conv_source_sha256={conv_source_sha()}")
    return "\n".join(out)


def counter_summary(counter_csv, agent_csv):
    """Text summary of a rocprofv3 --pmc run of `bench.py --pmc-frames N` with the
    matrix-core and LDS counters (MfmaUtil LdsUtil LdsBankConflict
    SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_LDS SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE
    SQ_BUSY_CYCLES). Per conv layer, mean over the sparse frames: the kernel's duration;
    mfma_util = MFMA busy cycles summed over every SIMD / (SIMDs x duration x peak
    engine clock), the counters' utilisation over the kernel's own run time; rocprof's
    MfmaUtil / LdsUtil / LdsBankConflict (percent of GRBM_GUI_ACTIVE, a window that
    also holds the profiler's per-dispatch set-up, so they read lower); and the
    matrix-core FLOPs the counters saw (MOPS x 512) over the algorithmic FLOPs."""
    import csv

    from paper_2108_09376_amd import resnet
    agent = [r for r in csv.DictReader(open(agent_csv)) if r.get("Name", "").startswith("gfx")][0]
    simds, clk = int(agent["Simd_Count"]), float(agent["Max_Engine_Clk_Fcompute"]) * 1e6
    per = {}
    for r in csv.DictReader(open(counter_csv)):
        d = per.setdefault(int(r["Dispatch_Id"]), {
            "name": r["Kernel_Name"],
            "dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    conv = [per[k] for k in sorted(per) if "k_conv_" in per[k]["name"]]
    if len(conv) % 53:
        raise SystemExit(f"{counter_csv}: {len(conv)} conv dispatches is not a whole number of frames")
    frames = [conv[i:i + 53] for i in range(0, len(conv), 53)][1:]
    layers = resnet.build_layers(50)
    shapes = resnet.layer_shapes(layers, 1024, 2048)
    flops = [2.0 * l.cin * l.cout * l.k * l.k * oh * ow * 38 / 128
             for l, (oh, ow, _) in zip(layers, shapes) if l.kind == "conv"]
    names = [l.name for l in layers if l.kind == "conv"]

    def mean(i, key):
        return sum(f[i][key] for f in frames) / len(frames)

    out = [f"device: {simds} SIMDs, peak engine clock {clk / 1e9:.2f} GHz; one 16x16x32 bf16 MFMA "
           f"holds a SIMD's matrix core for 16 cycles, so busy cycles x 16384 / 16 = FLOPs at peak",
           f"{'layer':24s} {'us':>7s} {'mfma_util':>9s} {'MfmaUtil%':>9s} {'LdsUtil%':>8s} "
           f"{'LdsBank%':>8s} {'flop/algo':>9s}"]
    tb = td = 0.0
    for i in range(53):
        busy, dur = mean(i, "SQ_VALU_MFMA_BUSY_CYCLES"), mean(i, "dur")
        tb += busy
        td += dur
        out.append(f"{names[i]:24s} {dur * 1e6:7.2f} {busy / (simds * dur * clk):9.4f} "
                   f"{mean(i, 'MfmaUtil'):9.2f} {mean(i, 'LdsUtil'):8.2f} {mean(i, 'LdsBankConflict'):8.3f} "
                   f"{mean(i, 'SQ_INSTS_VALU_MFMA_MOPS_BF16') * 512 / flops[i]:9.3f}")
    out.append(f"sparse frame (38/128 blocks), mean of {len(frames)} frames: {td * 1e6:.1f} us of conv "
               f"kernels under the profiler (kernels serialised, counters set up per dispatch), MFMA "
               f"busy {tb / simds / clk * 1e6:.2f} us per SIMD; the algorithmic {sum(flops) / 1e9:.1f} GFLOP "
               f"take {sum(flops) / (simds * clk * 16384 / 16) * 1e6:.2f} us per SIMD at peak")
    out.append(f"mfma_util_over_conv_kernel_time={tb / (simds * td * clk):.4f}")
    out.append(f"mfma_busy_us_per_simd_per_frame={tb / simds / clk * 1e6:.3f}")
    out.append(f"conv_source_sha256={conv_source_sha()}")
    return "\n".join(out)


def recorded_mfma_busy_us():
    """Matrix-core busy time per SIMD of one sparse frame's convolutions (counters), from
    the committed summary, or None if it is missing or was taken on other kernel sources."""
    try:
        kv = dict(l.split("=", 1) for l in open(MFMA_PROFILE).read().splitlines() if "=" in l
                  and " " not in l.split("=", 1)[0])
    except OSError:
        return None
    if kv.get("conv_source_sha256") != conv_source_sha():
        return None
    return float(kv["mfma_busy_us_per_simd_per_frame"])


def recorded_traffic():
    """HBM bytes per sparse-conv launch from the committed counter summary, or None if
    it is missing or was taken on other kernel sources."""
    try:
        kv = dict(l.split("=", 1) for l in open(TRAFFIC_PROFILE).read().splitlines() if "=" in l
                  and " " not in l.split("=", 1)[0])
    except OSError:
        return None
    if kv.get("conv_source_sha256") != conv_source_sha():
        return None
    return float(kv["traffic_bytes_per_conv_launch"])


def rocprof_summary(path, trace=None, first=0, count=0):
    """Text summary of a rocprofv3 kernel_stats.csv: per-kernel calls / average / total,
    and the sparse-conv kernels (k_conv_*) pooled into one average launch duration. With
    the kernel_trace.csv of the same run and a window of conv dispatches (ordinals among
    k_conv dispatches in start order, as bench.py reports it), the window is pooled too."""
    import csv
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = [f"{'kernel':70s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>9s} {'pct':>6s}"]
    conv_n = conv_t = 0.0
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "")
        name = name.split("(bc::")[0]
        n, avg, tot = int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["TotalDurationNs"]) / 1e6
        lines.append(f"{name[:70]:70s} {n:7d} {avg:9.2f} {tot:9.3f} {float(r['Percentage']):6.2f}")
        if "k_conv_" in r["Name"]:
            conv_n += n
            conv_t += float(r["TotalDurationNs"])
    if conv_n:
        lines.append(f"sparse conv kernels pooled: {int(conv_n)} launches, average "
                     f"{conv_t / conv_n / 1e3:.2f} us per launch")
    if trace:
        tr = [r for r in csv.DictReader(open(trace)) if "k_conv_" in r["Kernel_Name"]]
        tr.sort(key=lambda r: int(r["Start_Timestamp"]))
        win = tr[first:first + count]
        if len(win) != count:
            raise SystemExit(f"{trace}: only {len(tr)} conv dispatches, window needs {first + count}")
        d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in win]
        lines.append(f"sparse conv dispatches {first}..{first + count - 1} (the per-layer timing phase): "
                     f"{count} launches, average {sum(d) / count:.2f} us per launch")
    return "\n".join(lines)


def main():
    args = parse()
    if args.rocprof_summary:
        a = args.rocprof_summary
        print(rocprof_summary(a[0], *(a[1:2] + [int(v) for v in a[2:4]])))
        return
    if args.pmc_summary:
        print(pmc_summary(*args.pmc_summary))
        return
    if args.counter_summary:
        print(counter_summary(*args.counter_summary))
        return
    if args.layer_counter_summary:
        print(layer_counter_summary(*args.layer_counter_summary))
        return
    if args.gs_summary:
        print(gs_summary(*args.gs_summary))
        return
    if args.cpu_configs:
        print(cpu_configs())
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    from paper_2108_09376_amd import resnet

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.pmc_gather_scatter:
        from paper_2108_09376_amd import bc
        pmc_gather_scatter(torch, bc, dev)
        return
    if args.pmc_layers:
        from paper_2108_09376_amd import bc
        pmc_layers(torch, bc, dev, args.pmc_layers)
        return
    H, W, BLOCK = 1024, 2048, 128
    net = resnet.SparseResNet(50, H, W, BLOCK, device=dev)
    # counter runs take one dispatch per conv layer (the per-layer traffic table)
    net.pair_launches = not args.pmc_frames
    conv_launches = sum(l.kind == "conv" for l in net.layers) - (len(net.pairs) if net.pair_launches else 0)
    gh, gw = net.grid
    frame = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_INPUT), (1, H, W, 3)), "bf16")
    x = torch.from_numpy(frame.view(np.int16)).view(torch.bfloat16).to(dev)
    stream = torch.cuda.current_stream()

    def masks_for(frac):
        return synth.frac_mask(synth.SEED_MASK0 + 1, gh, gw, frac)

    net.frame(x, sparse=False)           # frame 0 of the clip: every block
    torch.cuda.synchronize()

    if args.pmc_frames:
        a0 = torch.empty(64 << 20, dtype=torch.float32, device=dev)
        a1 = torch.empty_like(a0)
        a0.fill_(1.0)
        torch.cuda.synchronize()
        torch.neg(a0, out=a1)             # calibration: 256 MiB read + 256 MiB written
        torch.cuda.synchronize()
        net.set_mask(masks_for(args.frac))
        for _ in range(args.pmc_frames):
            net.frame(x, sparse=True)
        torch.cuda.synchronize()
        return

    if args.profile_steps:
        net.set_mask(masks_for(args.frac))
        for _ in range(args.profile_steps):
            net.frame(x, sparse=True)
        torch.cuda.synchronize()
        return

    # Per-launch durations of the dominant kernel (the sparse conv), measured first, right
    # after frame 0: each conv layer is captured as a graph of `reps` back-to-back launches
    # on the frame's index and timed with HIP events on the capture stream, so host-side
    # marshalling is not counted. Every launch of this phase is timed or warms its graph,
    # so a kernel trace of this command pools exactly these dispatches: conv dispatches
    # [F, F + 53 * (reps + 3 * reps)) in launch order, F = frame 0's 49 conv launches.
    mask = masks_for(args.frac)
    active = int(mask.sum())
    flops = net.conv_flops(active)
    net.set_mask(mask)
    from paper_2108_09376_amd import bc
    bc.bc_build_block_index(net.mask, 1, net.grid, net.idx, net.count)
    torch.cuda.synchronize()
    conv_idx = [i for i, l in enumerate(net.layers) if l.kind == "conv"]
    reps = 10
    layer_us = {}
    for i in conv_idx:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                net.run_layer(i, x, net.idx, net.count)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        layer_us[i] = e0.elapsed_time(e1) * 1e3 / (3 * reps)
        del g
    conv_total_us = sum(layer_us.values())
    achieved = flops / (conv_total_us * 1e-6) / 1e12
    per_launch_us = conv_total_us / len(conv_idx)
    slowest = sorted(layer_us.items(), key=lambda kv: -kv[1])[:5]

    conv_window = {"first": conv_launches, "count": len(conv_idx) * reps * 4}

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

    def time_frames(frac, steps, warmup, mask=None):
        net.set_mask(masks_for(frac) if mask is None else mask)
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

    ms = time_frames(args.frac, args.steps, args.warmup)
    value = flops / (ms * 1e-3) / 1e12

    sweep = {}
    for f in [float(v) for v in args.sweep.split(",") if v.strip()]:
        sweep[f"{f:g}"] = round(time_frames(f, max(10, args.steps // 2), 3), 4)
    sweep[f"{args.frac:g}"] = round(ms, 4)

    # Floors of the frame. Chain: one active block (the grid's centre), every layer still
    # launched. Launches: as many dependent minimal kernels (a one-element add) as the
    # frame launches (index build + one per layer), captured in one graph.
    import numpy as np
    one = np.zeros((1, gh, gw), np.uint8)
    one[0, gh // 2, gw // 2] = 1
    one_block_ms = time_frames(0.0, max(10, args.steps // 2), 3, mask=one)
    n_launch = 1 + len(net.layers) - (len(net.pairs) if net.pair_launches else 0)
    tick = torch.zeros(1, device=dev)
    lg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(lg):
        for _ in range(n_launch):
            tick.add_(1.0)
    lg.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        lg.replay()
    e1.record()
    torch.cuda.synchronize()
    launch_floor_ms = e0.elapsed_time(e1) / 10
    del lg
    floors = {"one_active_block_ms": round(one_block_ms, 4),
              "dependent_launches_per_frame": n_launch,
              "launch_floor_ms": round(launch_floor_ms, 4),
              "launch_floor_us_per_launch": round(launch_floor_ms * 1e3 / n_launch, 3),
              "roofline_frac_at_launch_floor": round(flops / (launch_floor_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}

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
        "frame_floors": floors,
        "roofline": {"bound": "mfma", "kernel": "sparse conv (k_conv_pipe / stem, each of a frame's 53 conv layers launched alone)",
                     "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 5),
                     "avg_launch_us": round(per_launch_us, 3), "conv_us_per_frame": round(conv_total_us, 2),
                     "traffic": recorded_traffic(),
                     "mfma_util": (None if recorded_mfma_busy_us() is None else
                                   round(recorded_mfma_busy_us() / conv_total_us, 4)),
                     "algo_bytes_per_launch": round(sum(b for b in resnet.conv_algo_bytes(
                         net.layers, net.shapes, net.grid, active) if b) / len(conv_idx)),
                     "trace_conv_dispatch_window": conv_window,
                     "slowest_layers_us": {net.layers[i].name: round(u, 2) for i, u in slowest}},
    }
    out["config1_gpu_us_per_frame"] = config1_gpu(torch, bc, dev)
    out["measured_ceilings"] = measured_ceilings(torch, dev)
    if not args.no_vendor_dense:
        vms = vendor_dense_frame(torch, dev, net.layers)
        out["vendor_dense_frame"] = {
            "library": "torch conv2d (MIOpen), bf16 channels-last, residual and ReLU as torch ops",
            "ms": round(vms, 4), "ours_every_block_ms": sweep.get("1"),
            "ours_at_active_fraction_ms": round(ms, 4),
            "speedup_of_this_frame": round(vms / ms, 2)}
    if not args.no_layer_sweep:
        out["single_layers_at_0.3"] = layer_sweep(torch, bc, dev)
    if not args.no_gather_scatter:
        out["gather_scatter"] = gather_scatter(torch, bc, dev)
    if not args.no_clip:
        out["resnet18_clip"] = resnet18_clip(torch, dev)
        out["swiftnet18_clip_step"] = swiftnet_clip_step(torch, bc, dev)
    if not args.no_policy_steps:
        out["policy_steps"] = policy_steps(torch, bc, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(mask)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
