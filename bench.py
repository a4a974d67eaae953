"""Benchmark: mixed-precision convolution fwd + dgrad + wgrad throughput on
ResNet-50 shapes, one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload sweep]

One step = one pass of the whole path over one batch: for every one of
ResNet-50 v1.5's 53 convolution layers at batch 256 (channel-last fp16,
loss scale 1024): the stem's 3->8 channel padding, forward, backward-data
(not for the stem: no gradient to the image), backward-weight split-K with
its reduction / loss-scale epilogue into fp32 dw, and the shared overflow
flag.  Every layer has its own activation, weight and gradient buffers;
inputs are seeded synthetic draws already resident in HBM.  Prints one
JSON line.

value = sum of algorithmic FLOPs (2*N*K*P*Q*Cg*R*S per pass, stem with its
3 logical channels) / time of the timed steps, cold: before every timed step
a 1 GiB scratch buffer is written (outside the timed region), so no operand
starts in the 256 MB last-level cache.  The same K steps back to back (warm)
are reported beside it.  The GPU clock is sampled during the timed steps.
The timed steps carry no markers; per-pass, per-layer and per-launch figures
come from the same number of steps run again afterwards with HIP events
around every pass.
"""
from __future__ import annotations

import argparse
import re
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_F16_TFLOPS = 2516.6     # 256 CU x 4096 flop/clk x 2.4 GHz, dense fp16/bf16 MFMA
PEAK_HBM_GBS = 8000.0
METRIC = "conv fwd+dgrad+wgrad TFLOP/s on ResNet-50 shapes; % of fp16 MFMA peak"
METRIC_DW = ("depthwise conv fwd+dgrad+wgrad compulsory HBM GB/s on EfficientNet-B0 shapes; "
             "% of 8 TB/s")
METRIC_RNXT = ("grouped conv fwd+dgrad+wgrad algorithmic TFLOP/s on ResNeXt-50 32x4d shapes; "
               "% of fp16 MFMA peak")
METRIC_LAT = "conv fwd+dgrad+wgrad latency of one 3x3 16->16 NCHW convolution at batch 2; us"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="sweep",
                    choices=["sweep", "cfg1", "cfg2", "cfg3", "cfg4", "effdw", "rnxt"],
                    help="sweep: the 53 ResNet-50 layers at batch 256 (the headline metric); "
                         "cfg1: one 3x3 16->16 NCHW convolution at batch 2 (latency, us per "
                         "step); cfg2: the stage-1 bottleneck at batch 64; cfg3: the stage "
                         "transitions at batch 128; cfg4: the stem at batch 128 (fwd + wgrad); "
                         "effdw: the 16 depthwise layers of EfficientNet-B0 at batch 128 (one "
                         "channel per group, reported as HBM GB/s); rnxt: the 16 grouped 3x3 "
                         "layers of ResNeXt-50 32x4d at batch 128 (algorithmic TFLOP/s)")
    ap.add_argument("--dtype", default="f16", choices=["f16", "bf16"])
    ap.add_argument("--batch", type=int, default=0, help="override the batch size")
    ap.add_argument("--cpu-seconds", type=float, default=30.0,
                    help="upper bound on the oracle CPU-baseline sample (0 disables it)")
    ap.add_argument("--flush-mib", type=int, default=1024,
                    help="scratch written before every cold timed step (0: warm only)")
    ap.add_argument("--schedule", default="train2", choices=["serial", "train1", "train2"],
                    help="order of the timed steps: serial = fwd, dgrad, wgrad layer by layer "
                         "on one stream; train1 = the training order (forward over the layers, "
                         "then backward in reverse) on one stream; train2 (the headline) = the "
                         "training order with each backward-weight pass on a second stream, "
                         "started once the backward-data pass that yields its dy is queued; "
                         "any other schedule's cold time is reported beside it as 'serial'")
    ap.add_argument("--no-events", action="store_true",
                    help="skip the event-instrumented steps (per-pass times, roofline)")
    ap.add_argument("--layers", default="",
                    help="comma-separated layer names: run only these layers of the workload "
                         "(for profiling one shape; the reported value then covers only them)")
    ap.add_argument("--per-layer", default="",
                    help="write a per-layer / per-pass roofline table to this file")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the steps, run one plain device copy of this many MiB "
                         "(nnconv_pad_channels with no padding) as the reference dispatch "
                         "for scaling FETCH_SIZE / WRITE_SIZE counters")
    ap.add_argument("--summarize-profile", default="",
                    help="no GPU work: summarise rocprofv3 CSV output under this directory "
                         "(kernel trace and/or FETCH_SIZE / WRITE_SIZE counter runs of this "
                         "script) and exit")
    return ap.parse_args()


def layers_for(args):
    from paper_2102_06725_amd import inputs as I
    if args.workload in ("sweep", "effdw", "rnxt"):
        cfg = {"sweep": 5, "effdw": 6, "rnxt": 7}[args.workload]
        wl = I.workload(cfg, args.dtype, batch=args.batch or None)
        shapes = {5: I.resnet50_layers, 6: I.efficientnet_b0_depthwise,
                  7: I.resnext50_grouped}[cfg]
        expanded = []
        for l, c in shapes(wl.layers[0].n):
            expanded += [l] * c
        if args.layers:
            keep = set(args.layers.split(","))
            expanded = [l for l in expanded if l.name in keep]
        return wl, expanded
    cfg = {"cfg1": 1, "cfg2": 2, "cfg3": 3, "cfg4": 4}[args.workload]
    wl = I.workload(cfg, args.dtype, batch=args.batch or None)
    return wl, list(wl.layers)


class LayerBuffers:
    def __init__(self, L, wl, seed, dev, torch, nc):
        self.L = L
        self.torch = torch
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        tdt = torch.float16 if wl.dtype == "f16" else torch.bfloat16
        cl = L.c_alg
        # x: ReLU-like |N(0,1)| activations (the stem: N(0,1) pixels), channel-last
        x = torch.randn((L.n, L.h, L.w, cl), generator=g, device=dev, dtype=torch.float32)
        if wl.x_kind == "absnormal":
            x.abs_()
        self.x_raw = x.to(tdt)
        if cl != L.c:
            self.x = torch.empty((L.n, L.h, L.w, L.c), device=dev, dtype=tdt)
        else:
            self.x = self.x_raw
        # He-normal weights: fan-in is the group's logical channels times R*S
        cg, cgl = L.c // L.groups, cl // L.groups
        std = math.sqrt(2.0 / (cgl * L.r * L.s))
        w = torch.zeros((L.k, L.r, L.s, cg), device=dev, dtype=torch.float32)
        w[..., :cgl] = torch.randn((L.k, L.r, L.s, cgl), generator=g, device=dev) * std
        self.w = w.to(tdt)
        dy = torch.randn((L.n, L.p, L.q, L.k), generator=g, device=dev) * (wl.loss_scale * wl.dy_std)
        self.dy = dy.to(tdt)
        del x, w, dy
        self.y = torch.empty((L.n, L.p, L.q, L.k), device=dev, dtype=tdt)
        self.dx = torch.empty((L.n, L.h, L.w, L.c), device=dev, dtype=tdt) if L.dgrad else None
        self.dw = torch.empty((L.k, L.r, L.s, cg), device=dev, dtype=torch.float32)
        self.desc = nc.make_desc(L.n, L.c, L.h, L.w, L.k, L.r, L.s, (L.stride, L.stride),
                                 (L.pad, L.pad), (L.dil, L.dil), L.groups,
                                 nc.NNCONV_NCHW if wl.layout == "nchw" else nc.NNCONV_NHWC,
                                 nc.NNCONV_F16 if wl.dtype == "f16" else nc.NNCONV_BF16)
        self.ws_need = {}
        for p in (nc.NNCONV_FWD, nc.NNCONV_DGRAD, nc.NNCONV_WGRAD):
            st, nb = nc.nnconv_workspace_size(self.desc, p)
            nc.check(st, "workspace_size")
            self.ws_need[p] = nb


def compulsory_bytes(L, pass_):
    """Bytes a pass must move at least once: its operands and its output
    (2-byte elements, fp32 dw).  For strided 1x1 layers only the sampled
    pixels of x are read."""
    e = 2
    x_full = L.n * L.h * L.w * L.c * e
    if L.r == 1 and L.s == 1 and L.pad == 0:
        x_read = L.n * L.p * L.q * L.c * e
    else:
        x_read = x_full
    y = L.n * L.p * L.q * L.k * e
    w = L.k * L.r * L.s * (L.c // L.groups) * e
    if pass_ == "fwd":
        return x_read + w + y
    if pass_ == "dgrad":
        return y + w + x_full
    return x_read + y + 2 * w


def roofline_us(L, pass_):
    t_mfma = L.flops(executed=True) / (PEAK_F16_TFLOPS * 1e12)
    t_hbm = compulsory_bytes(L, pass_) / (PEAK_HBM_GBS * 1e9)
    return max(t_mfma, t_hbm) * 1e6, ("mfma" if t_mfma >= t_hbm else "hbm")


def write_per_layer(path, layers, ev_steps, steps):
    rows = []
    for i, L in enumerate(layers):
        for pi, pname in enumerate(("fwd", "dgrad", "wgrad")):
            if pname == "dgrad" and not L.dgrad:
                continue
            us = sum(ev[i][pi].elapsed_time(ev[i][pi + 1]) for ev in ev_steps) / steps * 1e3
            bound_us, bound = roofline_us(L, pname)
            rows.append((i, L.name, pname, us, L.flops() / (us * 1e-6) / 1e12, bound,
                         bound_us, 100.0 * bound_us / us))
    with open(path, "w") as f:
        f.write("%-3s %-10s %-6s %9s %8s %5s %9s %7s\n" % ("i", "layer", "pass", "us", "TFLOP/s",
                                                          "bound", "roof_us", "%roof"))
        for r in rows:
            f.write("%-3d %-10s %-6s %9.1f %8.1f %5s %9.1f %7.1f\n" % r)
        tot = sum(r[3] for r in rows)
        roof = sum(r[6] for r in rows)
        f.write("total %.1f us, roofline %.1f us (%.1f%%)\n" % (tot, roof, 100 * roof / tot))


# Sources that determine the forward launches (dispatch plans and kernels);
# stored HBM-traffic counters are reported only while these are unchanged.
FWD_SOURCES = ("api.hip", "common.hpp", "igemm_c8.hip", "igemm_c64.hip", "igemm_halo.hip",
               "igemm_hring.hip", "igemm_store.hpp", "launch.hpp", "stem.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "igemm_fwd_traffic_resnet50_b256.txt")
COPY_ROW_BYTES = 128    # calibration copy: rows of 64 fp16 channels


def fwd_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in FWD_SOURCES:
        with open(os.path.join(ROOT, "paper_2102_06725_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def stored_traffic(kind="mfma"):
    """HBM bytes per forward launch of the MFMA-bound (kind "mfma") or
    HBM-bound ("hbm") sweep layers from the committed FETCH_SIZE / WRITE_SIZE
    counter summary, or None when it is missing or was taken on other kernel
    sources."""
    try:
        kv = {}
        with open(TRAFFIC_FILE) as f:
            for line in f:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("source_sha256") != fwd_source_hash():
            return None
        return float(kv["%s_fetch_bytes_per_launch" % kind]) + \
            float(kv["%s_write_bytes_per_launch" % kind])
    except (OSError, KeyError, ValueError):
        return None


FWD_KERNEL = re.compile(r"nnconv::(igemm|stem_fwd|dw_fwd|dwt_fwd|pack_hring)")


def _main_fwd_kernel(n):
    return "nnconv::" in n and ("igemm" in n or "stem_fwd" in n or "dw_fwd" in n or
                                "dwt_fwd" in n)


def _opens_call(prev):
    """A dispatch after which the next library call starts: a non-library
    dispatch, a split reduction (end of a backward-weight call) or a padding
    copy (the stem's channel padding)."""
    return "nnconv::" not in prev or "wgrad_reduce" in prev or "pad_channels" in prev


def forward_calls(names):
    """Dispatch indices of each forward call in a trace of the serial schedule
    (flag clear, then per layer: optional stem channel padding, forward,
    backward-data kernels, backward-weight kernel and its reduction).  A
    forward call is an implicit-GEMM, stem or depthwise-forward dispatch that
    opens a call, with the weight-packing dispatch of the register-weight halo
    tiles in front of it when there is one."""
    calls = []
    for i, n in enumerate(names):
        if not _main_fwd_kernel(n):
            continue
        j, pre = i - 1, []
        if j >= 0 and "pack_hring" in names[j]:
            pre, j = [j], j - 1
        if j < 0 or _opens_call(names[j]):
            calls.append(pre + [i])
    return calls


def summarize_profile(args):
    """Prints per-kernel totals and the forward-launch figures from rocprofv3
    CSV output of `bench.py --calib-copy-mib M --steps K --warmup W`: a
    kernel trace, FETCH_SIZE and WRITE_SIZE counter runs (bytes per forward
    launch, for the MFMA-bound and the HBM-bound layers of the workload), and
    any other counter run (per-kernel averages per dispatch, with the MFMA
    utilisation and LDS bank-conflict rate derived where their counters are
    present)."""
    import csv
    import glob
    import collections
    layers = layers_for(args)[1]
    nl = len(layers)
    skip = args.warmup * nl
    mf, hb = fwd_sets(layers)
    sets = (("mfma", set(mf)), ("hbm", set(hb)))
    out = []

    def fwd_launches(names):
        """Forward calls (dispatch index lists) after the warm-up steps, with
        their layer index."""
        f = forward_calls(names)[skip:]
        return [(c, j % nl) for j, c in enumerate(f)]

    def family(n):
        return n.split("(")[0].replace("void ", "") if "nnconv::" in n else "(torch / runtime)"

    for path in sorted(glob.glob(os.path.join(args.summarize_profile, "**", "*kernel_trace.csv"),
                                 recursive=True)):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        names = [r["Kernel_Name"] for r in rows]
        dur = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in rows]
        fam = collections.defaultdict(lambda: [0, 0])
        for n, d in zip(names, dur):
            fam[family(n)][0] += 1
            fam[family(n)][1] += d
        tot = sum(v[1] for v in fam.values())
        out.append("kernel trace: %s" % os.path.relpath(path, args.summarize_profile))
        out.append("%-72s %7s %12s %10s %6s" % ("kernel", "calls", "total_us", "avg_us", "%"))
        for k, v in sorted(fam.items(), key=lambda kv: -kv[1][1]):
            out.append("%-72s %7d %12.1f %10.2f %6.2f" % (k[:72], v[0], v[1] / 1e3,
                                                          v[1] / v[0] / 1e3, 100.0 * v[1] / tot))
        fwd = fwd_launches(names)
        cdur = [sum(dur[i] for i in c) for c, _ in fwd]
        out.append("forward calls (after %d warm-up ones): %d, average %.2f us, total %.1f us"
                   % (skip, len(fwd), sum(cdur) / max(1, len(fwd)) / 1e3, sum(cdur) / 1e3))
        for kind, members in sets:
            sel = [d for d, (_, li) in zip(cdur, fwd) if li in members]
            if sel:
                out.append("forward calls of the %s-bound layers: %d, average %.2f us"
                           % (kind, len(sel), sum(sel) / len(sel) / 1e3))
        # the roofline launches of a run without --no-events: the runs of
        # forward kernels right after each loss-scaler initialisation (the
        # MFMA-bound set first, then the HBM-bound one)
        runs = []
        for i, n in enumerate(names):
            if "loss_scaler_init" in n:
                j = i + 1
                while j < len(names) and FWD_KERNEL.search(names[j]):
                    j += 1
                if j > i + 1:
                    runs.append(range(i + 1, j))
        for kind, run in zip([k for k, m in sets if m], runs):
            ncalls = sum(1 for i in run if "pack_hring" not in names[i])
            out.append("roofline calls (%s-bound set, back to back): %d, average %.2f us"
                       % (kind, ncalls, sum(dur[i] for i in run) / ncalls / 1e3))
    for path in sorted(glob.glob(os.path.join(args.summarize_profile, "**",
                                              "*counter_collection.csv"), recursive=True)):
        allrows = list(csv.DictReader(open(path)))
        counters = sorted({r["Counter_Name"] for r in allrows})
        for counter in counters:
            rows = sorted((r for r in allrows if r["Counter_Name"] == counter),
                          key=lambda r: int(r["Dispatch_Id"]))
            names = [r["Kernel_Name"] for r in rows]
            vals = [float(r["Counter_Value"]) for r in rows]
            if counter not in ("FETCH_SIZE", "WRITE_SIZE"):
                continue
            line = "%s (%s):" % (counter, os.path.relpath(path, args.summarize_profile))
            factor = None
            if args.calib_copy_mib:
                copy = [i for i, n in enumerate(names) if "pad_channels" in n][0]
                factor = args.calib_copy_mib * 1024.0 / vals[copy]
                line += " copy of %d MiB reads as %.1f KiB (factor %.4f);" % (
                    args.calib_copy_mib, vals[copy], factor)
            fwd = fwd_launches(names)
            out.append(line)
            for kind, members in sets:
                sel = [c for c, li in fwd if li in members]
                if not sel:
                    continue
                per = sum(vals[i] for c in sel for i in c) / len(sel) * 1024.0
                out.append("  forward launches of the %s-bound layers: %d, %.1f MB per launch as "
                           "counted%s" % (kind, len(sel), per / 1e6, "" if factor is None else
                                          ", %.1f MB scaled" % (per * factor / 1e6)))
                if factor is not None:
                    out.append("%s_%s_bytes_per_launch: %.0f" % (
                        kind, "fetch" if counter == "FETCH_SIZE" else "write", per * factor))
        others = [c for c in counters if c not in ("FETCH_SIZE", "WRITE_SIZE")]
        if not others:
            continue
        # per dispatch: counter values, duration and resources; then averages
        # per kernel and per (layer, kernel)
        disp = collections.defaultdict(dict)
        for r in allrows:
            d = disp[int(r["Dispatch_Id"])]
            d["name"] = r["Kernel_Name"]
            d["dur"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            d["res"] = (int(r["VGPR_Count"]), int(r["Accum_VGPR_Count"]),
                        int(r["LDS_Block_Size"]), int(r["Workgroup_Size"]))
            d[r["Counter_Name"]] = float(r["Counter_Value"])
        ids = sorted(disp)
        names = [disp[k]["name"] for k in ids]
        # layer of each dispatch: that of the latest forward launch (none
        # during the warm-up steps); pass: forward for that launch, then
        # backward-weight for the split-K kernels and their reduction,
        # backward-data for the rest
        layer_of, li = {}, None
        calls = forward_calls(names)
        call_of = {i: j for j, c in enumerate(calls) for i in c}
        for pos, k in enumerate(ids):
            fwd = pos in call_of
            if fwd and pos == calls[call_of[pos]][0]:
                j = call_of[pos] - skip
                li = layers[j % nl].name if j >= 0 else None
            nm = names[pos]
            ps = "fwd" if fwd else ("wgrad" if "wgrad" in nm else "dgrad")
            layer_of[k] = None if li is None else (li, ps)
        fam = collections.OrderedDict()
        per_layer = collections.OrderedDict()
        for k in ids:
            if "nnconv::" not in disp[k]["name"]:
                continue
            fam.setdefault(family(disp[k]["name"]), []).append(disp[k])
            if layer_of[k] is not None:
                per_layer.setdefault(layer_of[k] + (family(disp[k]["name"]),), []).append(disp[k])

        def derived(avg, dur):
            """MFMA utilisation, LDS bank-conflict rate, L2 hit rate, wait share."""
            f = []
            ga = avg.get("GRBM_GUI_ACTIVE")
            if ga and "SQ_VALU_MFMA_BUSY_CYCLES" in avg:
                # GRBM_GUI_ACTIVE sums the 8 XCDs; 1024 SIMDs
                f.append(("mfma_util", avg["SQ_VALU_MFMA_BUSY_CYCLES"] / (1024 * ga / 8)))
            if ga:
                f.append(("clock_ghz", ga / 8 / dur))
            if avg.get("SQ_LDS_IDX_ACTIVE") and "SQ_LDS_BANK_CONFLICT" in avg:
                f.append(("lds_conflict", avg["SQ_LDS_BANK_CONFLICT"] / avg["SQ_LDS_IDX_ACTIVE"]))
            if "TCC_HIT_sum" in avg and "TCC_MISS_sum" in avg:
                h, m = avg["TCC_HIT_sum"], avg["TCC_MISS_sum"]
                f.append(("l2_hit", h / max(1.0, h + m)))
            if avg.get("SQ_WAVE_CYCLES"):
                for c, n in (("SQ_WAIT_ANY", "wait_share"), ("SQ_ACTIVE_INST_ANY", "issue_share"),
                             ("SQ_WAIT_INST_LDS", "lds_wait_share")):
                    if c in avg:
                        f.append((n, avg[c] / avg["SQ_WAVE_CYCLES"]))
            return f

        def occupancy(res):
            """Waves per SIMD allowed by registers (512 per lane, granule 8)
            and by LDS (160 KiB per CU, 4 SIMDs).  On gfx950 the trace's
            VGPR_Count is half the registers a wave is given: the kernels
            here, compiled with -Rpass-analysis=kernel-resource-usage, report
            VGPRs + AGPRs (each rounded up to 8) equal to twice the trace's
            count, and the occupancy that gives."""
            vg, ag, lds, wg = res
            regs = ((2 * vg + 7) // 8) * 8 + ((ag + 7) // 8) * 8
            by_regs = min(8, 512 // max(8, regs))
            waves = max(1, wg // 64)
            by_lds = 8 if lds == 0 else (163840 // lds) * waves / 4.0
            return by_regs, by_lds

        out.append("counters per dispatch (%s), averaged per kernel:"
                   % os.path.relpath(path, args.summarize_profile))
        for name, ds in fam.items():
            avg = {c: sum(d.get(c, 0.0) for d in ds) / len(ds) for c in others}
            dur = sum(d["dur"] for d in ds) / len(ds)
            res = ds[0]["res"]
            occ = occupancy(res)
            out.append("%s  n=%d  avg %.2f us  registers %d (trace vgpr %d agpr %d) lds %d wg %d  "
                       "waves/SIMD: regs %d, lds %.1f"
                       % ((name[:100], len(ds), dur / 1e3, 2 * res[0]) + res + occ))
            out.append("    " + "  ".join("%s=%.4g" % kv for kv in sorted(avg.items())))
            f = derived(avg, dur)
            if f:
                out.append("    " + "  ".join("%s %.3f" % kv for kv in f))
        if per_layer:
            out.append("per layer and kernel (%s; layer = that of the latest forward launch):"
                       % os.path.relpath(path, args.summarize_profile))
            keys = None
            for (lname, ps, name), ds in per_layer.items():
                avg = {c: sum(d.get(c, 0.0) for d in ds) / len(ds) for c in others}
                dur = sum(d["dur"] for d in ds) / len(ds)
                f = derived(avg, dur)
                if keys is None:
                    keys = [k for k, _ in f]
                    out.append("  %-9s %-5s %-58s %4s %8s " % ("layer", "pass", "kernel", "n", "us") +
                               " ".join("%13s" % k for k in keys))
                short = name.replace("nnconv::", "")
                out.append("  %-9s %-5s %-58s %4d %8.1f " % (lname, ps, short[:58], len(ds),
                                                             dur / 1e3) +
                           " ".join("%13.3f" % v for _, v in f))
    out.append("source_sha256: %s" % fwd_source_hash())
    print("\n".join(out))


CPU_SAMPLE_BATCH = 16  # about 10-15 s of oracle work for the ResNet-50 shapes


def cpu_baseline(args, wl):
    """The fp64 oracle as it stands, timed on this host's cores over a bounded
    sample: every distinct layer shape of the workload at batch
    CPU_SAMPLE_BATCH, all its passes, stopping once the time bound is
    reached."""
    import numpy as np
    import oracle.oracle as orc
    from paper_2102_06725_amd import inputs as I
    orc.build(force=False)
    cores = len(os.sched_getaffinity(0))
    orc.set_threads(cores)
    seen = []
    for L in wl.layers:
        if L not in seen:
            seen.append(L)
    flops = 0
    t_total = 0.0
    done = 0
    passes_done = 0
    for li, L in enumerate(seen):
        Ls = L.with_batch(CPU_SAMPLE_BATCH)
        cl = Ls.c_alg
        cv = orc.Conv(Ls.n, cl, Ls.h, Ls.w, Ls.k, Ls.r, Ls.s, (Ls.stride,) * 2, (Ls.pad,) * 2,
                      (Ls.dil,) * 2, Ls.groups)
        rng = np.random.default_rng(7000 + li)
        x = np.abs(rng.standard_normal(cv.x_shape))
        w = rng.standard_normal(cv.w_shape) * math.sqrt(2.0 / (cl * Ls.r * Ls.s))
        dy = rng.standard_normal(cv.y_shape) * 1.024
        t0 = time.perf_counter()
        cv.fwd(x, w)
        n_pass = 1
        if Ls.dgrad:
            cv.dgrad(dy, w)
            n_pass += 1
        cv.wgrad(x, dy, 1.0 / 1024)
        n_pass += 1
        t_total += time.perf_counter() - t0
        flops += Ls.flops() * n_pass
        passes_done += n_pass
        done += 1
        if t_total > args.cpu_seconds:
            break
    return {
        "value": flops / t_total / 1e12,
        "unit": "TFLOP/s",
        "cores": orc.get_threads(),
        "kind": "oracle",
        "sample": "fp64 direct-loop oracle, %d of %d distinct layer shapes at batch %d "
                  "(%d passes, %.1f GFLOP) in %.1f s" % (done, len(seen), CPU_SAMPLE_BATCH,
                                                        passes_done, flops / 1e9, t_total),
    }


UPDATE_BYTES_PER_PARAM = 22  # read master, momentum, grad (fp32); write master, momentum, w16


def measure_update(args, layers, torch, nc, dev, sptr, stream, flush, reps=20):
    """Times the fused fp32 master-weight update (momentum SGD, loss-scale
    division, 16-bit copy) over every weight of the workload's layers held in
    one flat buffer -- outside the convolution metric, reported beside it.
    Cold: each launch follows a scratch write that evicts its operands from
    the last-level cache (back-to-back launches would find the 516 MB of
    operands partly cached); the warm back-to-back figure is reported too."""
    count = sum(L.k * (L.c_alg // L.groups) * L.r * L.s for L in layers)
    count = (count + 3) // 4 * 4
    g = torch.Generator(device="cpu").manual_seed(5)
    master = (torch.randn(count, generator=g) * 0.05).to(dev)
    mom = torch.zeros(count, dtype=torch.float32, device=dev)
    grad = (torch.randn(count, generator=g) * 20.0).to(dev)
    w16 = torch.empty(count, dtype=torch.int16, device=dev)
    state = torch.zeros(6, dtype=torch.int32, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    nc.check(nc.nnconv_loss_scaler_init(state.data_ptr(), 1024.0, 2.0, 2000, sptr), "scaler")
    w16_dtype = nc.NNCONV_F16 if args.dtype == "f16" else nc.NNCONV_BF16

    def call():
        nc.check(nc.nnconv_sgd_update(count, master.data_ptr(), mom.data_ptr(), w16.data_ptr(),
                                      w16_dtype, grad.data_ptr(), state.data_ptr(),
                                      flag.data_ptr(), 0.1, 0.9, 1e-4, sptr), "sgd_update")

    for _ in range(3):
        call()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    warm_us = e0.elapsed_time(e1) * 1e3 / reps
    us = warm_us
    if flush is not None:
        tot = 0.0
        for k in range(reps):
            flush.fill_(k & 0xFF)
            e0.record(stream)
            call()
            e1.record(stream)
            torch.cuda.synchronize()
            tot += e0.elapsed_time(e1) * 1e3
        us = tot / reps
    gbps = count * UPDATE_BYTES_PER_PARAM / (us * 1e-6) / 1e9
    return {"kernel": "sgd_update_kernel (one launch over all %d conv weights)" % count,
            "params": count, "us_per_launch": us, "bound": "hbm",
            "achieved": gbps, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": gbps / PEAK_HBM_GBS, "cache": "cold" if flush is not None else "warm",
            "warm_us_per_launch": warm_us,
            "warm_achieved": count * UPDATE_BYTES_PER_PARAM / (warm_us * 1e-6) / 1e9}


class ClockSampler:
    """Samples the GPU shader clock (the current level of the card's
    pp_dpm_sclk in sysfs, else amd-smi) on a host thread while armed; only
    samples taken inside armed intervals count."""

    def __init__(self, period_s=0.002):
        import glob
        import threading
        self.period = period_s
        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if paths else None
        self.source = "sysfs pp_dpm_sclk" if self.path else "amd-smi metric -c"
        self.samples = []
        self.armed = False
        self.stop = False
        self.t = threading.Thread(target=self._run, daemon=True)
        self.t.start()

    def _read(self):
        import re
        import subprocess
        try:
            if self.path:
                with open(self.path) as f:
                    for line in f:
                        if line.rstrip().endswith("*"):
                            m = re.search(r"(\d+)\s*[Mm]hz", line)
                            return float(m.group(1)) if m else None
                return None
            out = subprocess.run(["amd-smi", "metric", "-c", "--json"], capture_output=True,
                                 text=True, timeout=5).stdout
            vals = [float(v) for v in re.findall(r'"clk":\s*\{\s*"value":\s*(\d+)', out)]
            return sum(vals) / len(vals) if vals else None
        except Exception:
            return None

    def _run(self):
        while not self.stop:
            if self.armed:
                v = self._read()
                if v is not None and self.armed:
                    self.samples.append(v)
            time.sleep(self.period if self.path else 0.05)

    def close(self):
        self.stop = True
        self.t.join(timeout=2)

    def summary(self):
        busy = [v for v in self.samples if v >= 500.0]  # deep-sleep readings excluded
        if not busy:
            return None
        mean = sum(busy) / len(busy)
        return {"source": self.source, "samples": len(busy), "mean_mhz": mean,
                "min_mhz": min(busy), "max_mhz": max(busy),
                "peak_tflops_at_mean": 256 * 4096 * mean * 1e6 / 1e12}


def fwd_sets(layers):
    """Indices of the layers whose forward pass is MFMA-bound / HBM-bound by
    the compulsory-byte roofline."""
    mf = [i for i, L in enumerate(layers) if roofline_us(L, "fwd")[1] == "mfma"]
    hb = [i for i, L in enumerate(layers) if roofline_us(L, "fwd")[1] == "hbm"]
    return mf, hb


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(args)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only (libnnconv has no multi-GPU path); "
              "got --gpus %d" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2102_06725_amd import nnconv as nc

    nc.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    wl, layers = layers_for(args)
    bufs = [LayerBuffers(L, wl, 1_000_000 * 5 + 1000 * i + 1, dev, torch, nc)
            for i, L in enumerate(layers)]
    ws_bytes = max(max(b.ws_need.values()) for b in bufs)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    inv_s = 1.0 / wl.loss_scale
    flush = (torch.empty(args.flush_mib * 1024 * 1024, dtype=torch.uint8, device=dev)
             if args.flush_mib > 0 else None)
    if args.calib_copy_mib:
        rows = args.calib_copy_mib * 1024 * 1024 // COPY_ROW_BYTES
        src = torch.ones((rows, COPY_ROW_BYTES // 2), device=dev, dtype=torch.float16)
        dst = torch.empty_like(src)
        nc.check(nc.nnconv_pad_channels(src.data_ptr(), dst.data_ptr(), rows,
                                        COPY_ROW_BYTES // 2, COPY_ROW_BYTES // 2, sptr), "copy")
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()

    def one_step(ev):
        flag.zero_()
        for i, b in enumerate(bufs):
            L = b.L
            if b.x is not b.x_raw:
                nc.check(nc.nnconv_pad_channels(b.x_raw.data_ptr(), b.x.data_ptr(),
                                                L.n * L.h * L.w, L.c_alg, L.c, sptr), "pad")
            if ev is not None:
                ev[i][0].record(stream)
            nc.check(nc.nnconv_fwd(b.desc, b.x.data_ptr(), b.w.data_ptr(), b.y.data_ptr(), 1.0,
                                   ws.data_ptr(), ws_bytes, sptr), "fwd")
            if ev is not None:
                ev[i][1].record(stream)
            if L.dgrad:
                nc.check(nc.nnconv_dgrad(b.desc, b.dy.data_ptr(), b.w.data_ptr(), b.dx.data_ptr(),
                                         1.0, ws.data_ptr(), ws_bytes, sptr), "dgrad")
            if ev is not None:
                ev[i][2].record(stream)
            nc.check(nc.nnconv_wgrad(b.desc, b.x.data_ptr(), b.dy.data_ptr(), b.dw.data_ptr(),
                                     nc.NNCONV_F32, inv_s, 0, flag.data_ptr(), ws.data_ptr(),
                                     ws_bytes, sptr), "wgrad")
            if ev is not None:
                ev[i][3].record(stream)

    side = torch.cuda.Stream(device=dev) if args.schedule == "train2" else None
    ws_side = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev) if side else None
    ready = [torch.cuda.Event() for _ in bufs]
    joined = torch.cuda.Event()

    def train_step():
        """Forward over the layers in network order, then backward in reverse
        order.  A layer's dy exists once the backward-data pass of the layer
        after it has run, so its backward-weight pass may start there; with a
        side stream it runs next to the rest of the backward-data chain."""
        flag.zero_()
        for b in bufs:
            L = b.L
            if b.x is not b.x_raw:
                nc.check(nc.nnconv_pad_channels(b.x_raw.data_ptr(), b.x.data_ptr(),
                                                L.n * L.h * L.w, L.c_alg, L.c, sptr), "pad")
            nc.check(nc.nnconv_fwd(b.desc, b.x.data_ptr(), b.w.data_ptr(), b.y.data_ptr(), 1.0,
                                   ws.data_ptr(), ws_bytes, sptr), "fwd")
        for i in reversed(range(len(bufs))):
            b = bufs[i]
            if side is not None:
                ready[i].record(stream)
                side.wait_event(ready[i])
                nc.check(nc.nnconv_wgrad(b.desc, b.x.data_ptr(), b.dy.data_ptr(),
                                         b.dw.data_ptr(), nc.NNCONV_F32, inv_s, 0,
                                         flag.data_ptr(), ws_side.data_ptr(), ws_bytes,
                                         side.cuda_stream), "wgrad")
            else:
                nc.check(nc.nnconv_wgrad(b.desc, b.x.data_ptr(), b.dy.data_ptr(),
                                         b.dw.data_ptr(), nc.NNCONV_F32, inv_s, 0,
                                         flag.data_ptr(), ws.data_ptr(), ws_bytes, sptr),
                         "wgrad")
            if b.L.dgrad:
                nc.check(nc.nnconv_dgrad(b.desc, b.dy.data_ptr(), b.w.data_ptr(),
                                         b.dx.data_ptr(), 1.0, ws.data_ptr(), ws_bytes, sptr),
                         "dgrad")
        if side is not None:
            joined.record(side)
            stream.wait_event(joined)

    timed_step = (lambda: one_step(None)) if args.schedule == "serial" else train_step

    for _ in range(args.warmup):
        timed_step()
    torch.cuda.synchronize()

    clock = ClockSampler()
    # Warm: the K steps back to back (the last-level cache keeps what the
    # previous step left in it).  The timed steps carry no markers: an event
    # record between every two launches costs about 0.7 ms per sweep step.
    torch.cuda.synchronize()
    clock.armed = True
    t0 = time.perf_counter()
    for _ in range(args.steps):
        timed_step()
    torch.cuda.synchronize()
    warm_s = time.perf_counter() - t0
    clock.armed = False
    # Cold (the headline): every timed step starts after a scratch write of
    # flush_mib MiB, which leaves no operand in the 256 MB last-level cache;
    # the writes and their synchronisation are outside the timed region.
    cold_s = None
    if flush is not None:
        cold_s = 0.0
        for k in range(args.steps):
            flush.fill_(k & 0xFF)
            torch.cuda.synchronize()
            clock.armed = True
            t0 = time.perf_counter()
            timed_step()
            torch.cuda.synchronize()
            cold_s += time.perf_counter() - t0
            clock.armed = False
    # The serial schedule's cold time beside the headline (one stream, layer
    # by layer: the sum of the passes' kernel times with no overlap).
    serial_s = None
    if flush is not None and args.schedule != "serial":
        serial_s = 0.0
        for k in range(args.steps):
            flush.fill_(k & 0xFF)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            one_step(None)
            torch.cuda.synchronize()
            serial_s += time.perf_counter() - t0
    clock.close()
    elapsed = cold_s if cold_s is not None else warm_s
    if int(flag.item()) != 0:
        print("warning: overflow flag set during the benchmark", file=sys.stderr)

    # Per-pass, per-layer and per-launch figures: the same number of steps
    # again, warm, with HIP events around every pass (not part of `value`).
    use_ev = not args.no_events
    ev_steps = []
    if use_ev:
        for _ in range(args.steps):
            ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in bufs]
            one_step(ev)
            ev_steps.append(ev)
        torch.cuda.synchronize()

    # Roofline launches: the forward launches of the MFMA-bound and of the
    # HBM-bound layers, each set back to back `steps` times between two
    # events (an event pair around every launch would add the dispatch gap
    # to each one).  A loss-scaler initialisation before each set marks it
    # in a kernel trace.
    mf, hb = fwd_sets(layers)
    roof_launch_ms = {}
    if use_ev:
        mark = torch.empty(64, dtype=torch.uint8, device=dev)
        for kind, members in (("mfma", mf), ("hbm", hb)):
            if not members:
                continue
            nc.check(nc.nnconv_loss_scaler_init(mark.data_ptr(), 1.0, 2.0, 1, sptr), "mark")
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(args.steps):
                for i in members:
                    b = bufs[i]
                    nc.check(nc.nnconv_fwd(b.desc, b.x.data_ptr(), b.w.data_ptr(),
                                           b.y.data_ptr(), 1.0, ws.data_ptr(), ws_bytes, sptr),
                             "fwd")
            e1.record(stream)
            torch.cuda.synchronize()
            roof_launch_ms[kind] = e0.elapsed_time(e1) / (args.steps * len(members))

    step_flops = sum(L.flops() * (3 if L.dgrad else 2) for L in layers)
    depthwise = args.workload == "effdw"
    latency = args.workload == "cfg1"
    step_bytes = sum(compulsory_bytes(L, p) for L in layers
                     for p in (("fwd", "dgrad", "wgrad") if L.dgrad else ("fwd", "wgrad")))

    def rate(seconds):
        if latency:     # microseconds per step
            return seconds / args.steps * 1e6
        if depthwise:   # bound by HBM: compulsory bytes moved per second
            return step_bytes * args.steps / seconds / 1e9
        return step_flops * args.steps / seconds / 1e12

    value = rate(elapsed)

    per_pass, roofline, roofline_hbm, attainable = {}, None, None, None
    if use_ev:
        # event time of layer i, pass index pi, averaged over the steps (ms)
        def ev_ms(i, pi):
            return sum(ev[i][pi].elapsed_time(ev[i][pi + 1]) for ev in ev_steps) / args.steps

        for pi, pname in enumerate(("fwd", "dgrad", "wgrad")):
            ls = [i for i, L in enumerate(layers) if pname != "dgrad" or L.dgrad]
            ms = sum(ev_ms(i, pi) for i in ls)
            if ms > 0:
                per_pass[pname] = {"ms_per_step": ms,
                                   "tflops": sum(layers[i].flops() for i in ls) / ms / 1e9}
        # compulsory-byte roofline over every layer-pass of the step
        roof_ms = meas_ms = 0.0
        for i, L in enumerate(layers):
            for pi, pname in enumerate(("fwd", "dgrad", "wgrad")):
                if pname == "dgrad" and not L.dgrad:
                    continue
                roof_ms += roofline_us(L, pname)[0] / 1e3
                meas_ms += ev_ms(i, pi)
        attainable = {"roofline_ms_per_step": roof_ms, "measured_ms_per_step": meas_ms,
                      "frac": roof_ms / meas_ms,
                      "note": "sum over every layer-pass of max(executed flop / MFMA peak, "
                              "compulsory bytes / HBM peak) over the sum of their event times"}
        # The forward pass is one kernel launch per call; its average
        # duration comes from the back-to-back roofline launches above.
        # MFMA-bound and HBM-bound layers (by the compulsory-byte roofline)
        # are reported against their own peaks.
        if mf:
            ms = roof_launch_ms["mfma"]
            fl = sum(layers[i].flops() for i in mf) / len(mf)
            ach = fl / (ms * 1e-3) / 1e12
            traffic = stored_traffic("mfma") if args.workload == "sweep" and not args.layers \
                and not args.batch and args.dtype == "f16" else None
            roofline = {"kernel": "forward implicit GEMM (igemm_c64_kernel), the %d layers of "
                                  "the workload whose forward pass is MFMA-bound" % len(mf),
                        "bound": "mfma", "achieved": ach, "peak": PEAK_F16_TFLOPS,
                        "unit": "TFLOP/s", "frac": ach / PEAK_F16_TFLOPS, "traffic": traffic,
                        "avg_launch_us": ms * 1e3, "avg_flops_per_launch": fl,
                        "launch_timing": "the set's forward launches back to back, %d times, "
                                         "between two HIP events" % args.steps,
                        "frac_of_attainable": sum(roofline_us(layers[i], "fwd")[0] for i in mf)
                        / 1e3 / len(mf) / ms}
        if hb:
            ms = roof_launch_ms["hbm"]
            by = sum(compulsory_bytes(layers[i], "fwd") for i in hb) / len(hb)
            gbs = by / (ms * 1e-3) / 1e9
            traffic = stored_traffic("hbm") if args.workload == "sweep" and not args.layers \
                and not args.batch and args.dtype == "f16" else None
            kern = "depthwise forward (dwt_fwd_kernel)" if depthwise else \
                "forward implicit GEMM (igemm_c64_kernel; stem_fwd4_kernel for the stem)"
            roofline_hbm = {"kernel": "%s, the %d layers of the workload whose forward pass is "
                                      "HBM-bound" % (kern, len(hb)),
                            "bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS,
                            "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "traffic": traffic,
                            "avg_launch_us": ms * 1e3, "avg_bytes_per_launch": by,
                            "launch_timing": "the set's forward launches back to back, %d "
                                             "times, between two HIP events" % args.steps}
        if roofline is None:
            roofline, roofline_hbm = roofline_hbm, None

    update = measure_update(args, layers, torch, nc, dev, sptr, stream, flush) if use_ev \
        else None

    if args.per_layer and use_ev:
        write_per_layer(args.per_layer, layers, ev_steps, args.steps)

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(args, wl)

    sclk = clock.summary()
    L0 = layers[0]
    metric = (METRIC_DW if depthwise else METRIC_RNXT if args.workload == "rnxt" else
              METRIC_LAT if latency else METRIC)
    unit = "us" if latency else "GB/s" if depthwise else "TFLOP/s"
    out = {
        "metric": metric,
        "value": value,
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": not latency,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic (seeded; no dataset)",
        "config": {"workload": wl.name + ", %s %s, fwd+dgrad+wgrad%s, loss scale %g, "
                               "fp32 dw" % (
                                   "NCHW" if wl.layout == "nchw" else "channel-last", args.dtype,
                                   " (stem fwd+wgrad)" if not all(L.dgrad for L in layers)
                                   else "", wl.loss_scale),
                   "batch": L0.n, "layers": len(layers),
                   "layer_passes": sum(3 if L.dgrad else 2 for L in layers),
                   "tflop_per_step": step_flops / 1e12,
                   "compulsory_gb_per_step": step_bytes / 1e9},
        "schedule": {"headline": args.schedule,
                     "note": "train2: forward over the layers in network order, then backward in "
                             "reverse order with each backward-weight pass on a second stream "
                             "(default priority), queued once the backward-data pass that yields "
                             "its dy is queued, as a training step can run them",
                     "serial_cold": None if serial_s is None else {
                         "ms_per_step": serial_s / args.steps * 1e3, "value": rate(serial_s)}},
        "cache": {"headline": "cold" if cold_s is not None else "warm",
                  "flush_bytes": args.flush_mib * 1024 * 1024,
                  "cold": None if cold_s is None else {
                      "ms_per_step": cold_s / args.steps * 1e3, "value": rate(cold_s)},
                  "warm": {"ms_per_step": warm_s / args.steps * 1e3, "value": rate(warm_s)}},
        "sclk": sclk,
        "per_pass": per_pass,
        "attainable": attainable,
        "roofline": roofline,
        "roofline_hbm": roofline_hbm,
        "cpu_baseline": cpu,
        "update": update,
    }
    if not latency:
        peak = PEAK_HBM_GBS if depthwise else PEAK_F16_TFLOPS
        out["pct_of_peak"] = 100.0 * value / peak
        if sclk and not depthwise:
            out["pct_of_peak_at_sclk"] = 100.0 * value / sclk["peak_tflops_at_mean"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
