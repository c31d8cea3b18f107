#!/usr/bin/env python3
"""Benchmark of the SegBlocks block-conv hot path on one MI355X (gfx950).

Workload: one block-conv layer shaped like ResNet-18 stage 1 of a
1024x2048 image (stride 4): fp16, N=1, C_in=C_out=64, 256x512 feature map,
32-pixel blocks (8x16 grid, 128 image pixels per block), 3x3 conv with bias,
Bernoulli(0.5) low-resolution mask, x ~ N(0,1), w ~ N(0, 1/(9*C_in)), seed 0,
channels_last.  Synthetic data standing in for Cityscapes-shaped maps.

One step = one pass of the whole hot path over the batch: the fused layer
kernel, which plans the mask, samples (split + 2x2 average), pads, convolves
and combines in one launch.  Every step reads a different input/output
buffer set, so that the working set rotates through more memory than the
256 MB Infinity Cache holds and the inputs stream from HBM.

Printed: one JSON line with the headline metric (effective block-conv
TFLOP/s = dense-equivalent FLOPs / step time), the per-kernel breakdown of
the unfused path (split / pad / conv3x3 / combine, the fused-pad conv), the
dense-conv comparators, the roofline of the timed kernel and the CPU
oracle's throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP16_PEAK_TFLOPS = 2516.6      # MI355X dense fp16 MFMA
MALL_BYTES = 256 << 20         # Infinity Cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_layer_stage1.json")
KERNEL_SOURCES = ["sb_conv_res.hip", "sb_common.h", "sb_pixel.h", "sb_kernels.h"]

WL = dict(N=1, C=64, H=256, W=512, bs=32, dtype="f16", p_low=0.5, seed=0)


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--breakdown-iters", type=int, default=100)
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="oracle sample length (0 = skip)")
    p.add_argument("--profile-run", action="store_true",
                   help="short run for rocprofv3 counters: a 256 MiB copy of known size, then the layer")
    return p.parse_args()


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2011_12025_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (got --gpus {args.gpus}); the block-conv path "
              "would shard over images or block rows, see the design notes", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2011_12025_amd as sb
    import paper_2011_12025_amd._binding as B
    from paper_2011_12025_amd import inputs

    lib = B.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    N, C, H, W, bs, dt = WL["N"], WL["C"], WL["H"], WL["W"], WL["bs"], WL["dtype"]
    lb = bs // 2
    es = 2
    mask_np = inputs.mask_bernoulli(WL["seed"], N, H // bs, W // bs, WL["p_low"])
    nh = int(mask_np.sum())
    nl = int(mask_np.size - nh)
    f_low = nl / mask_np.size
    x0 = inputs.feature_map(WL["seed"], N, C, H, W, dt)
    w0 = inputs.conv_weight(WL["seed"], C, C, 3, dt)
    b0 = inputs.conv_bias(WL["seed"], C, 9 * C, dt)

    cl = torch.channels_last
    mask = torch.from_numpy(mask_np).to(dev)
    ones = torch.ones_like(mask)
    wd, bd = w0.to(dev).contiguous(memory_format=cl), b0.to(dev).contiguous()  # OHWI for channels_last calls
    x_first = x0.to(dev).contiguous(memory_format=cl)

    map_bytes = N * C * H * W * es
    stk_bytes = (nh * bs * bs + nl * lb * lb) * C * es
    pad_bytes = (nh * (bs + 2) ** 2 + nl * (lb + 2) ** 2) * C * es
    # every timed op cycles through R buffer sets; R is sized so that even the op
    # touching the fewest bytes per launch sweeps more than twice the Infinity Cache
    min_op_bytes = min(2 * stk_bytes, stk_bytes + pad_bytes, 2 * map_bytes)
    R = max(2, -(-2 * MALL_BYTES // min_op_bytes))
    if args.profile_run:
        R = 2

    def empty_stack(S, e):
        return torch.empty((S, C, e, e), dtype=x_first.dtype, device=dev, memory_format=cl)

    sets = []
    for r in range(R):
        s = dict(x=x_first.clone(memory_format=cl), y=torch.empty_like(x_first),
                 hi=empty_stack(nh, bs), lo=empty_stack(nl, lb), hp=empty_stack(nh, bs + 2),
                 lp=empty_stack(nl, lb + 2), ho=empty_stack(nh, bs), lo_o=empty_stack(nl, lb), yc=torch.empty_like(x_first))
        sets.append(s)
    torch.cuda.synchronize()

    P = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    mk, on, wp, bp = P(mask), P(ones), P(wd), P(bd)
    DT, LAY = B.SB_F16, B.SB_NHWC

    def args_for(name, s):
        if name == "layer":
            return (P(s["x"]), DT, LAY, N, C, H, W, mk, bs, wp, bp, C, P(s["y"]), stream)
        if name == "layer_allhigh":
            return (P(s["x"]), DT, LAY, N, C, H, W, on, bs, wp, bp, C, P(s["yc"]), stream)
        if name == "split":
            return (P(s["x"]), DT, LAY, N, C, H, W, mk, bs, P(s["hi"]), nh, P(s["lo"]), nl, stream)
        if name == "pad":
            return (P(s["hi"]), P(s["lo"]), DT, LAY, N, C, H, W, mk, bs, P(s["hp"]), P(s["lp"]), nh, nl, stream)
        if name == "conv3x3":
            return (P(s["hp"]), P(s["lp"]), DT, LAY, N, C, H, W, mk, bs, wp, bp, C, P(s["ho"]), P(s["lo_o"]), nh, nl,
                    stream)
        if name == "combine":
            return (P(s["ho"]), P(s["lo_o"]), DT, LAY, N, C, H, W, mk, bs, nh, nl, P(s["yc"]), stream)
        if name == "block_conv3x3":
            return (P(s["hi"]), P(s["lo"]), DT, LAY, N, C, H, W, mk, bs, wp, bp, C, 0, None, None, P(s["ho"]),
                    P(s["lo_o"]), nh, nl, stream)
        raise KeyError(name)

    FN = dict(layer=lib.segblocks_layer, layer_allhigh=lib.segblocks_layer, split=lib.segblocks_split,
              pad=lib.segblocks_pad, conv3x3=lib.segblocks_conv3x3, combine=lib.segblocks_combine,
              block_conv3x3=lib.segblocks_block_conv3x3)
    ARGS = {k: [args_for(k, s) for s in sets] for k in FN}

    def launch(name, i):
        rc = FN[name](*ARGS[name][i % R])
        if rc:
            raise RuntimeError(f"{name}: {lib.segblocks_last_error().decode()}")

    # ---------------- profile run (for rocprofv3 --pmc): known copy, then the layer
    if args.profile_run:
        a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        bcp = torch.empty_like(a)
        for _ in range(3):
            bcp.copy_(a)
        for i in range(10):
            launch("layer", i)
        torch.cuda.synchronize()
        print(json.dumps({"profile_run": True, "copy_bytes": a.numel(), "layer_launches": 10}))
        return

    # ---------------- warmup + the timed steps (the contract's region)
    for i in range(args.warmup):
        launch("layer", i)
    torch.cuda.synchronize()
    # one HIP event pair on the launch stream around the whole region: its span / K is
    # the average launch duration of the fused kernel (the host only enqueues here)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for i in range(args.steps):
        launch("layer", i)
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    layer_ms = ev0.elapsed_time(ev1) / args.steps

    # ---------------- per-kernel breakdown (GPU run-ahead, events around a batch)
    def time_batch(name, iters):
        for i in range(5):
            launch(name, i)
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)          # lets the host queue the whole batch first
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(iters):
            launch(name, i)
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / iters

    it = args.breakdown_iters
    bd_ms = {k: time_batch(k, it) for k in ["split", "pad", "conv3x3", "combine", "block_conv3x3", "layer",
                                            "layer_allhigh"]}

    # dense comparator: MIOpen through torch (measurement only, not part of the path)
    import torch.nn.functional as F
    xs = [s["x"] for s in sets]
    for i in range(5):
        F.conv2d(xs[i % R], wd, bd, padding=1)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(it):
        F.conv2d(xs[i % R], wd, bd, padding=1)
    e1.record()
    e1.synchronize()
    miopen_ms = e0.elapsed_time(e1) / it

    # check the timed output once against the unfused chain (bit-identical by construction)
    torch.cuda.synchronize()
    launch("split", 0); launch("pad", 0); launch("conv3x3", 0); launch("combine", 0); launch("layer", 0)
    torch.cuda.synchronize()
    chain_equal = bool(torch.equal(sets[0]["yc"], sets[0]["y"]))

    # ---------------- derived numbers
    dense_flop = 2.0 * 9 * C * C * N * H * W
    block_flop = 2.0 * 9 * C * C * (nh * bs * bs + nl * lb * lb)
    w_bytes = 9 * C * C * es + C * es
    layer_bytes = 2 * map_bytes + w_bytes + mask_np.size
    kbytes = dict(split=map_bytes + stk_bytes, pad=stk_bytes + pad_bytes, conv3x3=pad_bytes + w_bytes + stk_bytes,
                  combine=stk_bytes + map_bytes, block_conv3x3=2 * stk_bytes + w_bytes, layer=layer_bytes,
                  layer_allhigh=layer_bytes)
    kflop = dict(conv3x3=block_flop, block_conv3x3=block_flop, layer=block_flop, layer_allhigh=dense_flop)
    breakdown = {}
    for k, ms in bd_ms.items():
        d = {"us": round(ms * 1e3, 3), "GB/s": round(kbytes[k] / (ms * 1e-3) / 1e9, 1),
             "hbm_frac": round(kbytes[k] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        if k in kflop:
            d["TFLOP/s"] = round(kflop[k] / (ms * 1e-3) / 1e12, 2)
            d["mfma_frac"] = round(kflop[k] / (ms * 1e-3) / 1e12 / FP16_PEAK_TFLOPS, 4)
        breakdown[k] = d
    chain_us = sum(bd_ms[k] for k in ["split", "pad", "conv3x3", "combine"]) * 1e3
    breakdown["unfused_chain_us"] = round(chain_us, 3)
    breakdown["miopen_conv2d_us"] = round(miopen_ms * 1e3, 3)

    achieved_gbs = layer_bytes / (layer_ms * 1e-3) / 1e9
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tr = json.load(open(TRAFFIC_FILE))
        if tr.get("kernel_source_hash") == kernel_source_hash():
            traffic = tr.get("bytes_per_launch")

    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        xf, wf, bf = x0.float().numpy(), w0.float().numpy(), b0.float().numpy()
        reps, tc0 = 0, time.perf_counter()
        while True:
            oracle.layer(xf, mask_np, bs, wf, bf, dt)
            reps += 1
            if time.perf_counter() - tc0 >= args.cpu_seconds:
                break
        tcpu = time.perf_counter() - tc0
        cpu = {"value": round(dense_flop * reps / tcpu / 1e12, 6), "unit": "TFLOP/s", "cores": 1, "kind": "oracle",
               "sample": f"{reps} full layer(s) of the benchmark workload (split, pad, fp64 conv, combine), "
                         f"{tcpu:.1f} s single-threaded C", "s_per_layer": round(tcpu / reps, 3)}

    out = {
        "metric": "effective block-conv TFLOP/s (dense-equivalent FLOPs / layer time) at 1024x2048 stage-1 shape",
        "value": round(dense_flop / (ms_per_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic",
        "config": {"workload": "block-conv layer, ResNet-18 stage-1 shape of a 1024x2048 image: N=1, C_in=C_out=64, "
                               "256x512, block 32 (8x16 grid), 3x3 conv + bias, Bernoulli(0.5) low-res mask, "
                               "channels_last",
                   "n_high": nh, "n_low": nl, "low_fraction": round(f_low, 4), "rotating_buffer_sets": R},
        "layer_latency_us": round(layer_ms * 1e3, 3),
        "vs_dense": {"ours_all_high_us": breakdown["layer_allhigh"]["us"], "miopen_conv2d_us": breakdown["miopen_conv2d_us"],
                     "speedup_vs_ours_all_high": round(bd_ms["layer_allhigh"] / bd_ms["layer"], 3),
                     "speedup_vs_miopen": round(miopen_ms / bd_ms["layer"], 3),
                     "theoretical_flop_speedup": round(dense_flop / block_flop, 3)},
        "pad_GBps": breakdown["pad"]["GB/s"],
        "roofline": {"bound": "hbm", "kernel": "k_conv_res<f16,SRC_DENSE,DST_DENSE> (segblocks_layer)",
                     "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": layer_bytes,
                     "algorithmic_flop_per_launch": block_flop,
                     "mfma_frac": round(block_flop / (layer_ms * 1e-3) / 1e12 / FP16_PEAK_TFLOPS, 4)},
        "breakdown": breakdown,
        "fused_equals_unfused_chain": chain_equal,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
