"""Benchmark: one training step (forward + backward) of a parareal network on one MI355X.

Default workload: Parareal ResNet-1001 with N = 16 fine sub-networks (21 bottleneck units each,
the last 18), batch 128 of 3x32x32 synthetic N(0,1) images, 100 classes, bf16 storage.

Prints ONE JSON line.  ``value`` is the metric's first part: fine-sub-network convolution TFLOP/s,
i.e. 3 x (forward conv FLOPs of all N sub-networks, projections included) / GPU time of
parareal_fine_fwd + parareal_fine_bwd, averaged over as many steps as are timed.  ``images_per_s``
is batch / whole-step time (preprocessing, fine, combine, coarse, head and all backward parts).
``--graph`` times replays of the step captured in HIP graphs (one graph per part, so that the
fine and coarse parts are timed between replays) instead of eager library calls.  The timed steps
run the backward as parareal_bwd (coarse chain overlapped with the fine sub-networks; ``--no-overlap``:
the two separate calls); the fine and coarse GPU times (and so ``value``) then come from the same
number of steps with the separate calls, run right after the timed region.
"""
from __future__ import annotations

import argparse
import json
import statistics
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


def cpu_baseline(idx, batch=24, coarse="config"):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload: one full step of the
    same network at a reduced batch.  Reported in the metric's unit (fine conv TFLOP/s)."""
    import pnn_synth as S
    from oracle import prim
    from oracle.net import ParaRealOracle
    net = S.config(idx, batch, coarse=coarse)
    x, labels, params = S.make_all(net)
    o = ParaRealOracle(net, params)
    t0 = time.perf_counter()
    o.step(x, labels)
    dt = time.perf_counter() - t0
    return {"value": fine_flops(net) / dt / 1e12, "unit": "TFLOP/s", "cores": prim.threads(),
            "kind": "oracle",
            "sample": f"one full fwd+bwd step of {net.name} at batch {batch} (of {S.config(idx).batch}), "
                      f"{dt:.1f} s, fine conv FLOPs / whole-step time"}


# sources a kernel family's code and launch shapes come from; a stored traffic figure is void
# once any of them changes
KERNEL_SOURCES = {
    "conv_kernel": ["k_conv.hip", "k_gemm.hip", "conv_epilogue.h", "bn_fuse.h", "device_common.h", "pnn_internal.h",
                    "plan.hip"],
    "wgrad_kernel": ["k_conv.hip", "device_common.h", "pnn_internal.h", "plan.hip"],
}
COPY_BYTES = 256 << 20          # the --copy-calibration copy
# the kernels of a family: the launches the library's timing family covers (conv: every forward
# and data-gradient convolution launch, the GEMM kernel's and its split-K reduce's included)
FAMILY_KERNELS = {"conv_kernel": ("conv_kernel", "gemm_conv_kernel", "gemm_reduce_kernel")}


def _sources_sha(kernel):
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2103_08802_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def stored_traffic(kernel):
    """HBM bytes per launch of ``kernel`` measured with rocprofv3 PMC counters (FETCH_SIZE and
    WRITE_SIZE passes, each scaled by the same counter's reading for a plain copy of known size),
    kept in profiles/ with a hash of the kernel's sources; None once those sources have changed."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}.json")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("sources_sha256") != _sources_sha(kernel):
        return None
    return rec["bytes_per_launch"]


def stored_mfma(kernel):
    """MFMA utilisation of ``kernel`` from a rocprofv3 --pmc run of the derived counters MfmaUtil
    and MfmaFlopsBF16 (profiles/mfma_<kernel>.json, hash-guarded like the traffic record)."""
    path = os.path.join(ROOT, "profiles", f"mfma_{kernel}.json")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("sources_sha256") != _sources_sha(kernel):
        return None
    return {"mfma_util_pct": rec["mfma_util_pct"], "mfma_flops_per_launch": rec["mfma_flops_per_launch"]}


def _short(name):
    return name.split("(")[0].replace("void ", "").split("<")[0].replace("pnn::", "")


def summarize_pmc(fetch_csv, write_csv, kernel, cmd):
    """Reduce two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE; KiB per dispatch) of a
    ``--copy-calibration`` run to HBM bytes per launch of ``kernel`` and store the result."""
    import csv

    def load(p):
        per, copy = {}, None
        for r in csv.DictReader(open(p)):
            v = float(r["Counter_Value"]) * 1024.0
            n = _short(r["Kernel_Name"])
            if n == "__amd_rocclr_copyBuffer":
                copy = max(copy or 0.0, v)        # the largest copy is the calibration copy
            per.setdefault(n, []).append(v)
        return per, copy

    fe, fcopy = load(fetch_csv)
    wr, wcopy = load(write_csv)
    ffac, wfac = COPY_BYTES / fcopy, COPY_BYTES / wcopy
    names = FAMILY_KERNELS.get(kernel, (kernel,))
    fe = {kernel: [v for n in names for v in fe.get(n, [])]}
    wr = {kernel: [v for n in names for v in wr.get(n, [])]}
    fb = sum(fe[kernel]) / len(fe[kernel]) * ffac
    wb = sum(wr[kernel]) / len(wr[kernel]) * wfac
    rec = {"kernel": kernel, "bytes_per_launch": round(fb + wb), "fetch_bytes_per_launch": round(fb),
           "write_bytes_per_launch": round(wb), "dispatches": len(fe[kernel]), "family_kernels": list(names),
           "fetch_scale": round(ffac, 4), "write_scale": round(wfac, 4),
           "calibration": f"one {COPY_BYTES >> 20} MiB device-to-device copy reads and writes "
                          f"{COPY_BYTES} bytes; FETCH_SIZE read {fcopy:.0f}, WRITE_SIZE {wcopy:.0f}",
           "command": cmd, "sources": KERNEL_SOURCES[kernel], "sources_sha256": _sources_sha(kernel)}
    out = os.path.join(ROOT, "profiles", f"traffic_{kernel}.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))


def summarize_families(fetch_csv, write_csv, trace_csv, out_md, cmd):
    """Per kernel family: HBM bytes per launch from the two --pmc runs (each counter scaled by what
    it reads for the calibration copy), average duration from a --kernel-trace run of the same
    build and workload, and the HBM bandwidth they give."""
    import csv

    def inst(name):
        return name.split("(")[0].replace("void ", "").replace("pnn::", "")

    def load(p, key):
        per, copy = {}, None
        for r in csv.DictReader(open(p)):
            v = float(r["Counter_Value"]) * 1024.0
            if _short(r["Kernel_Name"]) == "__amd_rocclr_copyBuffer":
                copy = max(copy or 0.0, v)
            per.setdefault(key(r["Kernel_Name"]), []).append(v)
        return per, copy

    def durations(key):
        dur = {}
        for r in csv.DictReader(open(trace_csv)):
            dur.setdefault(key(r["Kernel_Name"]), []).append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        return dur

    def table(key):
        fe, fcopy = load(fetch_csv, key)
        wr, wcopy = load(write_csv, key)
        ffac, wfac = COPY_BYTES / fcopy, COPY_BYTES / wcopy
        dur = durations(key)
        rows = []
        for n in fe:
            if n not in wr or n not in dur or "__amd" in n or n.startswith("at::"):
                continue
            fb = sum(fe[n]) / len(fe[n]) * ffac
            wb = sum(wr[n]) / len(wr[n]) * wfac
            us = sum(dur[n]) / len(dur[n])
            rows.append((n, len(dur[n]), fb / 1e6, wb / 1e6, us, (fb + wb) / (us * 1e3)))
        rows.sort(key=lambda r: -r[1] * r[4])
        return rows, ffac, wfac

    rows, ffac, wfac = table(_short)
    irows = [r for r in table(inst)[0] if r[0].startswith("conv_kernel<")]
    with open(out_md, "w") as f:
        f.write("# HBM traffic per kernel family: parareal ResNet-1001, N=16, batch 128, bf16 (one "
                "stream)\n\nCommands (from the repository root, on one MI355X):\n\n```\n"
                f"{cmd}\n```\n\n")
        f.write(f"FETCH_SIZE scaled by {ffac:.4f}, WRITE_SIZE by {wfac:.4f} (what each reads for one "
                f"{COPY_BYTES >> 20} MiB device copy).  Bytes per launch are averages over the PMC "
                "runs' dispatches, durations over the kernel-trace run's; both runs use the same "
                "launches per step.\n\n")
        f.write("| family | launches (trace) | fetched MB | written MB | avg us | HBM GB/s |\n"
                "|---|---:|---:|---:|---:|---:|\n")
        for n, c, fm, wm, us, gbs in rows:
            f.write(f"| `{n}` | {c} | {fm:.1f} | {wm:.1f} | {us:.2f} | {gbs:.0f} |\n")
        f.write("\nPer `conv_kernel` instantiation (template arguments: storage type, mode 0 forward / 1 "
                "data gradient, gather kind 0 pointwise / 1 vector / 2 element-wise / 3 3x3 halo tile, "
                "row and column sub-tiles per wave):\n\n")
        f.write("| instantiation | launches (trace) | fetched MB | written MB | avg us | HBM GB/s |\n"
                "|---|---:|---:|---:|---:|---:|\n")
        for n, c, fm, wm, us, gbs in irows:
            f.write(f"| `{n}` | {c} | {fm:.1f} | {wm:.1f} | {us:.2f} | {gbs:.0f} |\n")


def summarize_mfma(csv_path, out_md, algo_flops, cmd, title="parareal ResNet-1001, N=16, batch 128, bf16 (one stream)"):
    """Per kernel family, from one rocprofv3 --pmc run of the derived counters MfmaUtil (MFMA busy
    cycles summed over SIMDs / (GPU active cycles x SIMDs), percent) and MfmaFlopsBF16 (bf16 MFMA
    operations x 512): the launch-weighted MFMA utilisation and the MFMA FLOPs per launch.  For
    conv_kernel the counted FLOPs are set against the algorithmic 2 M N K per launch
    (``algo_flops``, from the bench line's roofline record of the same build): their ratio is the
    work the MFMA tiles do on padding (K rounded up to the instruction's 32, ragged row tiles)."""
    import csv
    util, flops, durs = {}, {}, {}
    for r in csv.DictReader(open(csv_path)):
        n = _short(r["Kernel_Name"])
        v = float(r["Counter_Value"])
        key = (n, r["Dispatch_Id"])
        if r["Counter_Name"] == "MfmaUtil":
            util[key] = v
        elif r["Counter_Name"] == "MfmaFlopsBF16":
            flops[key] = v
        durs[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    fams = {}
    for (n, d), u in util.items():
        f = fams.setdefault(n, [0, 0.0, 0.0, 0.0])
        f[0] += 1
        f[1] += u * durs[(n, d)]
        f[2] += durs[(n, d)]
        f[3] += flops.get((n, d), 0.0)
    rows = sorted(fams.items(), key=lambda kv: -kv[1][2])
    rec = None
    with open(out_md, "w") as fh:
        fh.write(f"# MFMA utilisation per kernel family: {title}\n\nCommand (from the repository root, "
                 "on one MI355X):\n\n```\n"
                 f"{cmd}\n```\n\nMfmaUtil = SQ_VALU_MFMA_BUSY_CYCLES summed over SIMDs / "
                 "(GRBM_GUI_ACTIVE x SIMD count), per dispatch, averaged weighted by dispatch "
                 "duration; MFMA GFLOP = MfmaFlopsBF16 (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) per "
                 "dispatch; TFLOP/s = that over the dispatch's duration.\n\n")
        fh.write("| family | dispatches | MfmaUtil % | MFMA GFLOP / dispatch | MFMA TFLOP/s |\n"
                 "|---|---:|---:|---:|---:|\n")
        for n, (c, uw, t, fl) in rows:
            fh.write(f"| `{n}` | {c} | {uw / t:.2f} | {fl / c / 1e9:.3f} | {fl / (t * 1e-6) / 1e12:.1f} |\n")
        members = [fams[n] for n in FAMILY_KERNELS["conv_kernel"] if n in fams]
        if members and algo_flops:      # the record: the workload whose algorithmic FLOPs are given
            c, uw, t, fl = (sum(m[i] for m in members) for i in range(4))
            fh.write(f"| conv family ({' + '.join(FAMILY_KERNELS['conv_kernel'])}) | {c} | {uw / t:.2f} | "
                     f"{fl / c / 1e9:.3f} | {fl / (t * 1e-6) / 1e12:.1f} |\n")
            rec = {"kernel": "conv_kernel", "mfma_util_pct": round(uw / t, 3),
                   "mfma_flops_per_launch": round(fl / c), "dispatches": c}
            if algo_flops:
                rec["algorithmic_flops_per_launch"] = algo_flops
                rec["mfma_over_algorithmic"] = round(fl / c / algo_flops, 4)
                fh.write(f"\nconv family: {fl / c / 1e9:.3f} GFLOP of bf16 MFMA work per launch against "
                         f"{algo_flops / 1e9:.3f} GFLOP algorithmic (2 M N K of the launch's problems, "
                         f"bench line): ratio {fl / c / algo_flops:.3f} (padding of K to the "
                         "instruction's 32 and of ragged row tiles).\n")
    if rec is not None:
        rec.update({"command": cmd, "sources": KERNEL_SOURCES["conv_kernel"],
                    "sources_sha256": _sources_sha("conv_kernel")})
        with open(os.path.join(ROOT, "profiles", "mfma_conv_kernel.json"), "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        print(json.dumps(rec))


def summarize_sq(csv_path, out_md, cmd):
    """Per kernel instantiation, ratios of one rocprofv3 --pmc run of SQ counters (SQ_WAVES,
    SQ_WAVE_CYCLES, SQ_BUSY_CYCLES, SQ_WAIT_ANY, SQ_WAIT_INST_LDS, SQ_ACTIVE_INST_LDS,
    SQ_VALU_MFMA_BUSY_CYCLES, SQ_LDS_BANK_CONFLICT), summed over its dispatches."""
    import csv
    tot, disp = {}, {}
    for r in csv.DictReader(open(csv_path)):
        n = r["Kernel_Name"].split("(")[0].replace("void ", "")
        tot.setdefault(n, {}).setdefault(r["Counter_Name"], 0.0)
        tot[n][r["Counter_Name"]] += float(r["Counter_Value"])
        disp.setdefault(n, set()).add(r["Dispatch_Id"])
    rows = sorted(tot.items(), key=lambda kv: -kv[1].get("SQ_WAVE_CYCLES", 0.0))
    with open(out_md, "w") as f:
        f.write("# SQ counters per conv_kernel instantiation: parareal ResNet-1001, N=16, batch 128, "
                "bf16 (one stream)\n\nCommand (from the repository root, on one MI355X):\n\n```\n"
                f"{cmd}\n```\n\nwave cycles = SQ_WAVE_CYCLES / SQ_WAVES; the waits and LDS activity as "
                "fractions of SQ_WAVE_CYCLES; LDS bank-conflict cycles per LDS-active cycle (MFMA "
                "utilisation: the MfmaUtil summary).\n\n")
        f.write("| kernel | dispatches | waves / dispatch | cycles / wave | wait any | wait LDS | "
                "LDS active | bank conflicts / LDS active |\n"
                "|---|---:|---:|---:|---:|---:|---:|---:|\n")
        for n, c in rows:
            w, wc = c.get("SQ_WAVES", 0.0), c.get("SQ_WAVE_CYCLES", 0.0)
            if w <= 0 or wc <= 0:
                continue
            lds = max(c.get("SQ_ACTIVE_INST_LDS", 0.0), 1.0)
            f.write(f"| `{n}` | {len(disp[n])} | {w / len(disp[n]):.0f} | {wc / w:.0f} | "
                    f"{c.get('SQ_WAIT_ANY', 0.0) / wc:.2f} | {c.get('SQ_WAIT_INST_LDS', 0.0) / wc:.2f} | "
                    f"{c.get('SQ_ACTIVE_INST_LDS', 0.0) / wc:.2f} | "
                    f"{c.get('SQ_LDS_BANK_CONFLICT', 0.0) / lds:.2f} |\n")


def summarize_trace(stats_csv, trace_csv, out_md, title, cmd):
    """Markdown summary of a rocprofv3 --kernel-trace --stats run: the per-instantiation statistics
    and, per kernel family, the average duration over all its dispatches."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    fam = {}
    for r in csv.DictReader(open(trace_csv)):
        n = _short(r["Kernel_Name"])
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        t = fam.setdefault(n, [0, 0.0])
        t[0] += 1
        t[1] += d
    # every step runs the head once: its dispatch count is the number of steps in the run
    steps = fam.get("head_sample_kernel", [0, 0.0])[0]
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\nCommand (from the repository root, on one MI355X):\n\n```\n{cmd}\n```\n\n")
        f.write("Per kernel family, all dispatches of the run (warm-up, timed and instrumented steps):\n\n")
        f.write("| family | dispatches | per step | avg us | total ms |\n|---|---:|---:|---:|---:|\n")
        lib = 0
        for n, (c, t) in sorted(fam.items(), key=lambda kv: -kv[1][1]):
            per = f"{c / steps:.1f}" if steps else "-"
            f.write(f"| `{n}` | {c} | {per} | {t / c:.2f} | {t / 1e3:.1f} |\n")
            if not n.startswith(("at::", "__amd")):
                lib += c
        if steps:
            f.write(f"\n{steps} steps in the run (one head launch each): {lib / steps:.0f} library kernel "
                    "launches per step (torch fills and copies excluded).\n")
        cf = [fam[n] for n in FAMILY_KERNELS["conv_kernel"] if n in fam]
        if cf:
            c, t = sum(x[0] for x in cf), sum(x[1] for x in cf)
            f.write(f"\nconv family ({' + '.join(FAMILY_KERNELS['conv_kernel'])}: the launches the bench's "
                    f"conv timing covers): {c} dispatches, {t / c:.2f} us on average.\n")
        f.write("\nPer instantiation (rocprofv3 --stats):\n\n")
        f.write("| kernel | calls | avg us | min us | max us | total % |\n|---|---:|---:|---:|---:|---:|\n")
        for r in rows[:24]:
            name = r["Name"].split("(")[0].replace("void ", "")
            f.write(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                    f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                    f"{float(r['Percentage']):.2f} |\n")


def time_config(idx, streams, steps, warmup):
    """ms per step (4 streams, overlapped backward), images/s, and the fine sub-networks' conv
    TFLOP/s and share of the bf16 MFMA peak (from as many steps with the separate calls) of
    workload ``idx``."""
    import torch
    import pnn_synth as S
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    B.pnn_set_streams(g.plan, streams)
    g.load_input(x, labels)
    g.overlap_bwd = True
    for _ in range(warmup):
        g.forward()
        g.backward()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.forward()
        g.backward()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    g.overlap_bwd = False
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for e in ev:
        g.forward(fine_events=(e[0], e[1]))
        g.backward(fine_events=(e[2], e[3]))
    torch.cuda.synchronize()
    fine_ms = statistics.median(e[0].elapsed_time(e[1]) + e[2].elapsed_time(e[3]) for e in ev)
    tf = fine_flops(net) / (fine_ms * 1e-3) / 1e12
    del g
    torch.cuda.empty_cache()
    return {"workload": f"{net.name}: batch {net.batch}, {net.in_shape[0]}x{net.in_shape[1]}x"
                        f"{net.in_shape[2]} input, N={net.n_sub}",
            "steps": steps, "ms_per_step": round(ms, 3), "images_per_s": round(net.batch / (ms * 1e-3), 1),
            "fine_ms_per_step": round(fine_ms, 3), "fine_tflops": round(tf, 2),
            "pct_bf16_mfma_peak": round(100.0 * tf / PEAK_BF16_TFLOPS, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3, help="workload index 0..4")
    ap.add_argument("--partition", default="contiguous",
                    choices=("contiguous", "per_stage", "balanced", "balanced_flops"),
                    help="split of the ResNet units into sub-networks")
    ap.add_argument("--coarse", default="config", choices=("config", "paper"),
                    help="coarse blocks F^j: the workload's (one unit) or the paper's own networks")
    ap.add_argument("--streams", type=int, default=4,
                    help="streams the fine forward / backward may spread its sub-network groups over "
                         "(1: everything on one stream, as the per-kernel timing passes run)")
    ap.add_argument("--no-overlap", action="store_true",
                    help="timed steps call coarse_bwd_all and parareal_fine_bwd one after the other "
                         "instead of parareal_bwd (the coarse chain overlapped with the fine backward)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured in HIP graphs instead of eager library calls")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 256 MiB device copy first (reference for HBM byte counters)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU work: store HBM bytes per launch of --kernel from two PMC runs")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("STATS_CSV", "TRACE_CSV", "OUT_MD"),
                    help="no GPU work: write a markdown summary of a kernel-trace run")
    ap.add_argument("--summarize-families", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "TRACE_CSV", "OUT_MD"),
                    help="no GPU work: HBM bytes, duration and bandwidth per kernel family")
    ap.add_argument("--summarize-mfma", nargs=2, metavar=("PMC_CSV", "OUT_MD"),
                    help="MfmaUtil / MfmaFlopsBF16 summary of a rocprofv3 --pmc run (and profiles/mfma_conv_kernel.json)")
    ap.add_argument("--algo-flops", type=float, default=0.0,
                    help="algorithmic FLOPs per conv_kernel launch of the same build (bench line)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the timing of the other workloads (the line's 'configs' record)")
    ap.add_argument("--summarize-sq", nargs=2, metavar=("PMC_CSV", "OUT_MD"),
                    help="no GPU work: SQ counter ratios per kernel instantiation")
    ap.add_argument("--kernel", default="conv_kernel")
    ap.add_argument("--title", default="")
    ap.add_argument("--cmd", default="", help="command that produced the CSVs (recorded)")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.kernel, args.cmd)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace, args.title, args.cmd)
        return
    if args.summarize_families:
        summarize_families(*args.summarize_families, args.cmd)
        return
    if args.summarize_sq:
        summarize_sq(*args.summarize_sq, args.cmd)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma, args.algo_flops, args.cmd,
                       args.title or "parareal ResNet-1001, N=16, batch 128, bf16 (one stream)")
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this library runs the whole parareal network on ONE GPU (all N "
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
    net = S.config(args.config, coarse=args.coarse, partition=args.partition)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    B.pnn_set_streams(g.plan, args.streams)
    g.load_input(x, labels)
    s = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(args.steps)]

    def step(k=None, graph=False):
        e = ev[k] if k is not None else None
        fwd, bwd = (g.replay_forward, g.replay_backward) if graph else (g.forward, g.backward)
        fwd(fine_events=(e[0], e[1]) if e else None, coarse_events=(e[4], e[5]) if e else None)
        bwd(fine_events=(e[2], e[3]) if e else None, coarse_events=(e[6], e[7]) if e else None)

    use_graph = args.graph
    g.overlap_bwd = not args.no_overlap and not args.graph    # the graphs capture the separate calls
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if use_graph:
        g.capture()             # the timed steps replay the captured step (all its launches)
        for _ in range(args.warmup):
            step(graph=True)
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(k, graph=use_graph)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    overlapped = g.overlap_bwd and net.n_sub > 1
    # backward of the timed steps: coarse chain + fine sub-networks (one span when overlapped)
    bwd_ms = sum(e[2].elapsed_time(e[3]) + (0.0 if overlapped else e[6].elapsed_time(e[7]))
                 for e in ev) / args.steps
    if overlapped:
        # the fine and coarse parts of the overlapped backward are not separable: time them from
        # the same number of steps with the separate calls, right after the timed region
        g.overlap_bwd = False
        for _ in range(args.warmup):
            step()
        for k in range(args.steps):
            step(k)
        torch.cuda.synchronize()
        g.overlap_bwd = True
    # per-step GPU times of the fine calls and of the coarse chain: the median over the timed steps
    fine_ms = statistics.median(e[0].elapsed_time(e[1]) + e[2].elapsed_time(e[3]) for e in ev)
    coarse_ms = (statistics.median(e[4].elapsed_time(e[5]) + e[6].elapsed_time(e[7]) for e in ev)
                 if net.n_sub > 1 else 0.0)
    ff = fine_flops(net)
    tflops = ff / (fine_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if net.dtype == "bf16" else PEAK_F32_TFLOPS

    # per-kernel-family GPU time (HIP events around every launch of that family, same stream),
    # over the same number of steps right after the timed region; these passes run every launch on
    # one stream, so that each launch is timed alone
    fam = {}
    for f, name in ((1, "conv_kernel"), (2, "wgrad_kernel"), (3, "pw_kernel")):
        B.pnn_timing_enable(g.plan, f)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ms, n, fl, by = B.pnn_timing_read(g.plan)
        B.pnn_timing_enable(g.plan, 0)
        fam[name] = {"ms": ms, "launches": n, "flops": fl, "bytes": by}
    dom = max(fam, key=lambda k: fam[k]["ms"])
    default_cfg = (args.config, args.coarse, args.partition) == (3, "config", "contiguous")
    d = fam[dom]
    # the family's bound: MFMA when its algorithmic intensity is above the ridge point
    # (peak FLOP/s / peak bytes/s), else HBM
    peak_f = PEAK_BF16_TFLOPS if net.dtype == "bf16" else PEAK_F32_TFLOPS
    mfma = d["flops"] / max(d["bytes"], 1.0) > peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    tflops_dom = d["flops"] / (d["ms"] * 1e-3) / 1e12
    achieved = d["bytes"] / (d["ms"] * 1e-3) / 1e9
    roof = {"bound": "mfma" if mfma else "hbm",
            "achieved": round(tflops_dom if mfma else achieved, 2 if mfma else 1),
            "peak": peak_f if mfma else PEAK_HBM_GBS, "unit": "TFLOP/s" if mfma else "GB/s",
            "frac": round((tflops_dom / peak_f) if mfma else (achieved / PEAK_HBM_GBS), 4),
            "traffic": (stored_traffic(dom) if default_cfg else None),
            "algorithmic_bytes_per_launch": round(d["bytes"] / max(d["launches"], 1)),
            "algorithmic_flops_per_launch": round(d["flops"] / max(d["launches"], 1)),
            "kernel": dom, "kernels": list(FAMILY_KERNELS.get(dom, (dom,))),
            "avg_launch_us": round(d["ms"] * 1e3 / max(d["launches"], 1), 2),
            "hbm_gbs": round(achieved, 1), "mfma_tflops": round(tflops_dom, 2)}
    mf = stored_mfma(dom) if default_cfg else None
    if mf is not None:
        roof.update(mf)

    # the parameter update (SGD, Nesterov momentum; not part of the step the metric times)
    g.sgd_init()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g.sgd_step(0.01, 0.9, 1e-4, True)
    e0.record()
    for _ in range(args.steps):
        g.sgd_step(0.01, 0.9, 1e-4, True)
    e1.record()
    torch.cuda.synchronize()
    sgd_ms = e0.elapsed_time(e1) / args.steps

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config, coarse=args.coarse)

    # the other workloads the throughput target names, timed the same way (fewer steps)
    configs = None
    if default_cfg and not args.no_configs:
        del g
        torch.cuda.empty_cache()
        configs = {}
        for idx, key in ((1, "vgg16-n4-b128"), (2, "resnet1001-n4-b64"), (4, "resnet1001-64px-n8-b128")):
            configs[key] = time_config(idx, args.streams, max(3, args.steps // 2), 2)

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
                   "batch": net.batch, "n_sub": net.n_sub,
                   "parallelism": f"single GPU, N sub-networks grouped, {args.streams} stream(s), "
                                  f"{'HIP graph replay' if args.graph else 'eager launches'}"},
        "images_per_s": round(net.batch / (ms_step * 1e-3), 1),
        "pct_bf16_mfma_peak": round(100.0 * tflops / peak, 3),
        "fine_ms_per_step": round(fine_ms, 3),
        "fine_gflop_per_step": round(ff / 1e9, 1),
        "coarse_ms_per_step": round(coarse_ms, 3),
        "bwd_ms_per_step": round(bwd_ms, 3),
        "bwd_overlapped": overlapped,
        "sgd_ms_per_step": round(sgd_ms, 3),
        "roofline": roof,
        "cpu_baseline": cpu,
        "configs": configs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
