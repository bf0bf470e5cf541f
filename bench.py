"""Benchmark: one training step (forward + backward) of a parareal network on one MI355X.

Default workload: Parareal ResNet-1001 with N = 16 fine sub-networks (21 bottleneck units each,
the last 18), batch 128 of 3x32x32 synthetic N(0,1) images, 100 classes, bf16 storage.

Prints ONE JSON line.  ``value`` is the metric's first part: fine-sub-network convolution TFLOP/s,
i.e. 3 x (forward conv FLOPs of all N sub-networks, projections included) / GPU time of
parareal_fine_fwd + parareal_fine_bwd, averaged over the timed steps.  ``images_per_s`` is
batch / whole-step time (preprocessing, fine, combine, coarse, head and all backward parts).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 (vector / MFMA dense)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def conv_flops(seg, batch):
    """Forward multiply-add FLOPs (2 x MACs) of the convolutions of one segment."""
    from pnn_synth.gen import segment_shapes
    sh = segment_shapes(seg)
    f = 0
    for n in seg.nodes:
        if n.op == "conv":
            H, W, C = sh[n.dst]
            f += 2 * batch * H * W * C * n.k * n.k * sh[n.src][2]
    return f


def fine_flops(net):
    return 3 * sum(conv_flops(s, net.batch) for s in net.fine)


def cpu_baseline(idx, batch=24):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload: one full step of the
    same network at a reduced batch.  Reported in the metric's unit (fine conv TFLOP/s)."""
    import pnn_synth as S
    from oracle import prim
    from oracle.net import ParaRealOracle
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    o = ParaRealOracle(net, params)
    t0 = time.perf_counter()
    o.step(x, labels)
    dt = time.perf_counter() - t0
    return {"value": fine_flops(net) / dt / 1e12, "unit": "TFLOP/s", "cores": prim.threads(),
            "kind": "oracle",
            "sample": f"one full fwd+bwd step of {net.name} at batch {batch} (of {S.config(idx).batch}), "
                      f"{dt:.1f} s, fine conv FLOPs / whole-step time"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, help="workload index 0..4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 256 MiB device copy first (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs the whole parareal network on ONE GPU (all N "
                          "fine sub-networks as grouped launches); --gpus must be 1"}))
        sys.exit(2)

    import torch
    import pnn_synth as S
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU

    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    net = S.config(args.config)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    s = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]

    def step(k=None):
        e = ev[k] if k is not None else None
        g.forward(fine_events=(e[0], e[1]) if e else None)
        g.backward(fine_events=(e[2], e[3]) if e else None)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(k)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    fine_ms = sum(e[0].elapsed_time(e[1]) + e[2].elapsed_time(e[3]) for e in ev) / args.steps
    ff = fine_flops(net)
    tflops = ff / (fine_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if net.dtype == "bf16" else PEAK_F32_TFLOPS

    # per-kernel-family GPU time (HIP events around every launch of that family, same stream),
    # over the same number of steps right after the timed region
    fam = {}
    for f, name in ((1, "conv_kernel"), (2, "wgrad_kernel")):
        B.pnn_timing_enable(g.plan, f)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ms, n, fl, by = B.pnn_timing_read(g.plan)
        B.pnn_timing_enable(g.plan, 0)
        fam[name] = {"ms": ms, "launches": n, "flops": fl, "bytes": by}
    dom = max(fam, key=lambda k: fam[k]["ms"])
    d = fam[dom]
    achieved = d["bytes"] / (d["ms"] * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
            "kernel": dom, "avg_launch_us": round(d["ms"] * 1e3 / max(d["launches"], 1), 2),
            "mfma_tflops": round(d["flops"] / (d["ms"] * 1e-3) / 1e12, 2)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config)

    out = {
        "metric": "fine-subnet conv TFLOP/s (fwd+bwd, % bf16 MFMA peak) + images/s per step",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": net.dtype,
        "data": "synthetic N(0,1) images, uniform labels, He-normal init (seeded)",
        "config": {"workload": f"{net.name}: batch {net.batch}, {net.in_shape[0]}x{net.in_shape[1]}x"
                               f"{net.in_shape[2]} input, N={net.n_sub} fine sub-networks, "
                               f"{net.classes} classes",
                   "batch": net.batch, "n_sub": net.n_sub, "parallelism": "single GPU, N sub-networks grouped"},
        "images_per_s": round(net.batch / (ms_step * 1e-3), 1),
        "pct_bf16_mfma_peak": round(100.0 * tflops / peak, 3),
        "fine_ms_per_step": round(fine_ms, 3),
        "fine_gflop_per_step": round(ff / 1e9, 1),
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
