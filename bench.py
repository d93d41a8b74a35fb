"""Benchmark: pattern/connectivity-pruned VGG-16 conv stack, batch 1, fp32,
224x224 input, on one MI355X.

One step = one full forward frame through pp_net_fwd (13 conv layers -- the
first dense, twelve pattern-pruned 4-of-9 keeping 1/3 of the kernels -- each
fused with bias + ReLU, and five 2x2 max pools), inputs resident in HBM.

Prints ONE JSON line:
  value        effective GMAC/s over the frame, counting surviving MACs only
  ms_per_step  ms per frame
  roofline     the pruned-conv kernel's rate against the MI355X fp32 vector
               peak (157.3 TFLOP/s), timed live with HIP events per layer
               (bf16 frames whose time goes mostly to the matrix-core form:
               that form's contraction against the bf16 matrix peak)
  cpu_baseline the fp64 CPU oracle on the same frame (reported baseline)
  dense        the same masked model run as dense convs (torch conv2d on the
               same GPU) for the speedup

    python bench.py [--steps K] [--warmup W] [--config 2] [--dtype f32]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_VECTOR_TFLOPS = 157.3     # MI355X: 256 CU x 2.4 GHz x 256 FLOP/clk.  gfx950 retires a plain
                                    # (non-packed) wave64 v_fmac_f32 in about 2 cycles per SIMD with enough
                                    # waves, so this is the FMA peak of the kernels here (built without packed
                                    # FP32); the measured ceiling (libppceil.so) is reported beside it
PEAK_HBM_GBS = 8000.0
PEAK_BF16_MFMA_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak
MFMA_RECIPE = 64                    # pp_conv2d_recipe id of the bf16 matrix-core form

WORKLOADS = {2: "vgg16_conv_stack_224x224_b1", 3: "style_transfer_512x512_b1", 4: "super_resolution_270x480_x4_b1",
             5: "colorization_256x256_b8", 1: "pruned_layer_16x16_32x32_b1"}


def layer_shapes(spec):
    """(op index, op, input (c,h,w), output (c,h,w)) for every op."""
    c, h, w = spec["c"], spec["h"], spec["w"]
    slots = {0: (c, h, w)}
    out = []
    for i, op in enumerate(spec["ops"]):
        c, h, w = slots[op["src"]]
        k = op["op"]
        if k == "conv3":
            s, p, d = op["stride"], op["pad"], op["dil"]
            o = (op["c_out"], (h + 2 * p - 2 * d - 1) // s + 1, (w + 2 * p - 2 * d - 1) // s + 1)
        elif k == "conv":
            o = (op["c_out"], h + 2 * op["pad"] - op["k"] + 1, w + 2 * op["pad"] - op["k"] + 1)
        elif k == "deconv":
            o = (op["c_out"], 2 * h, 2 * w)
        elif k == "maxpool2":
            o = (c, h // 2, w // 2)
        elif k == "up2":
            o = (c, 2 * h, 2 * w)
        elif k == "pshuf2":
            o = (c // 4, 2 * h, 2 * w)
        else:
            o = (c, h, w)
        out.append((i, op, (c, h, w), o))
        slots[op["dst"]] = o
    return out


def surviving_macs(op, prm, oshape, batch):
    """MACs that survive pruning: output pixels x kept taps (padded taps counted)."""
    k = op["op"]
    _, ho, wo = oshape
    if k == "conv3":
        taps = np.array([bin(int(m)).count("1") for m in prm["lib"]])
        kept = taps[np.where(prm["conn"] != 0, prm["pid"], 0)] * (prm["conn"] != 0)
        return batch * ho * wo * int(kept.sum())
    if k == "conv":
        return batch * ho * wo * op["c_out"] * op["c_in"] * op["k"] ** 2
    if k == "deconv":
        return batch * ho * wo * op["c_out"] * op["c_in"] * 4   # 2x2 of the 4x4 taps per output
    return 0


KERNEL_SOURCES = ("conv_pp_kernel.hpp", "conv_pp_inst.hpp", "conv_pp.hpp", "conv_plan.cpp", "conv_pp_c8_s1d1.hip",
                  "conv_pp_wave.hpp", "conv_pp_wave_inst.hpp", "conv_pp_wave_s1d1.hip", "conv_pp_wave_d9_s1d1.hip",
                  "conv_pp_lean.hpp", "conv_pp_lean.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pp_conv3x3_vgg16_224x224_b1_traffic.json")


def kernel_source_hash():
    """sha256 over the sources of the pruned-conv kernel and its planner: a
    stored byte count is valid only for the code it was measured on."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2004_11250_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _kernel_label(name):
    """Kernel name(s) without 'void ' and without the parameter lists."""
    out = []
    for part in name.split(" + "):
        part = part.replace("void ", "")
        out.append(part[:part.rfind("(")] if part.endswith(")") else part)
    return " + ".join(out)


def summarize_profile(root, cfg=2):
    """Summarise rocprofv3 CSV output under ``root`` (kt/: --kernel-trace
    --stats; fetch/, write/: --pmc FETCH_SIZE / WRITE_SIZE of a run with
    --copy-mib; sq*/: other --pmc passes) for one frame of the network: the
    dispatches of the first frame are the len(ops) dispatches starting at the
    first pruned-conv launch (an op fused into the conv before it has no
    dispatch of its own).  Writes the traffic JSON read by the benchmark and
    prints a markdown summary."""
    import csv
    import glob

    import paper_2004_11250_amd as pp
    import workloads
    spec = workloads.net_spec(cfg)
    fused = pp.net_plan(spec["ops"], workloads.net_params(cfg), spec["batch"], spec["c"], spec["h"],
                        spec["w"])["fused"]
    n_disp = len(spec["ops"]) - len(fused)
    shapes = layer_shapes(spec)

    def rows(sub):
        f = glob.glob(os.path.join(root, sub, "*_counter_collection.csv")) or \
            glob.glob(os.path.join(root, sub, "*_kernel_trace.csv"))
        return list(csv.DictReader(open(f[0]))) if f else []

    def by_dispatch(rs):
        d = {}
        for r in rs:
            e = d.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "grid": r.get("Grid_Size") or
                                                     r.get("Grid_Size_X"), "c": {}})
            e["dur_ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            if "Counter_Name" in r:
                e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        return [d[k] for k in sorted(d)]

    def frames(ds):
        # a frame is one dispatch per unfused op, starting at the first
        # pruned-conv launch; a channel-split conv is followed by its
        # reduction dispatch, which is merged into the conv's entry
        def is_conv(e):
            return "pp_conv3x3" in e["name"]

        first = next(i for i, e in enumerate(ds) if is_conv(e))
        out = []
        while len(out) < 400 and first < len(ds) and is_conv(ds[first]):
            fr, j = [], first
            for _ in range(n_disp):
                if j >= len(ds):
                    return out
                e = dict(ds[j], c=dict(ds[j]["c"]))
                j += 1
                if j < len(ds) and ("pp_split_reduce" in ds[j]["name"] or "pp_lean_reduce" in ds[j]["name"]):
                    e["dur_ns"] += ds[j]["dur_ns"]
                    for k, v in ds[j]["c"].items():
                        e["c"][k] = e["c"].get(k, 0.0) + v
                    e["name"] += " + " + ds[j]["name"]
                    j += 1
                fr.append(e)
            out.append(fr)
            first = j
        return out

    def calib(ds, counter, mib):
        # the elementwise copy: the largest grid among the non-library kernels
        # before the first frame, reads and writes exactly mib MiB
        first = next(i for i, e in enumerate(ds) if "pp_conv3x3" in e["name"])
        cands = [e for e in ds[:first] if "mul" in e["name"].lower() or "elementwise" in e["name"].lower()]
        e = max(cands, key=lambda e: int(e["grid"]))
        return mib * 1024.0 / e["c"][counter], e["c"][counter]

    kt = by_dispatch(rows("kt"))
    fe = by_dispatch(rows("fetch"))
    wr = by_dispatch(rows("write"))
    kt_fr, fe_fr, wr_fr = frames(kt), frames(fe), frames(wr)
    ff, f_raw = calib(fe, "FETCH_SIZE", 256)
    wf, w_raw = calib(wr, "WRITE_SIZE", 256)
    sq = {}
    for sub in sorted(os.listdir(root)):
        if sub.startswith("sq") and os.path.isdir(os.path.join(root, sub)):
            for fr in frames(by_dispatch(rows(sub)))[:1]:
                for di, e in enumerate(fr):
                    sq.setdefault(di, {}).update(e["c"])
    lay = []
    di = -1   # dispatch index within a frame
    for i, (k, op, ish, osh) in enumerate(shapes):
        if i in fused:
            into = i + 1 if fused[i] == "up2" else i - 1
            lay.append(dict(op=i, kind=op["op"], lib="", c_in=ish[0], c_out=osh[0], hw=f"{osh[1]}x{osh[2]}",
                            kernel=f"(fused into op {into})", us=0.0, fetch_mb=0.0, write_mb=0.0, sq={}))
            continue
        di += 1
        # steady state: the median over every frame of the run (the first,
        # warm-up frames of a trace run several times slower)
        dur = float(np.median([f[di]["dur_ns"] for f in kt_fr])) / 1e3
        fetch = float(np.median([f[di]["c"]["FETCH_SIZE"] for f in fe_fr])) * ff * 1024
        write = float(np.median([f[di]["c"]["WRITE_SIZE"] for f in wr_fr])) * wf * 1024
        kind = ("up2+" if fused.get(i - 1) == "up2" else "") + op["op"] + \
            ("+" + fused[i + 1] if i + 1 in fused and fused[i + 1] != "up2" else "")
        lay.append(dict(op=i, kind=kind, lib=op.get("lib", ""), c_in=ish[0], c_out=osh[0], hw=f"{osh[1]}x{osh[2]}",
                        kernel=_kernel_label(kt_fr[0][di]["name"]), us=round(dur, 3),
                        fetch_mb=round(fetch / 1e6, 3), write_mb=round(write / 1e6, 3), sq=sq.get(di, {})))
    pr = [l for l in lay if l["kind"].startswith("conv3") and l["lib"] == "canon8"]
    traffic = dict(kernel_source_sha256=kernel_source_hash(), fetch_factor=round(ff, 4), write_factor=round(wf, 4),
                   launches=len(pr), bytes_per_frame=int(sum((l["fetch_mb"] + l["write_mb"]) * 1e6 for l in pr)),
                   us_per_frame=round(sum(l["us"] for l in pr), 3), frames_traced=len(kt_fr),
                   layers=[{k: v for k, v in l.items() if k != "sq"} for l in pr])
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(traffic, fh, indent=1)
    print(f"calibration: 256 MiB elementwise copy reads FETCH_SIZE={f_raw:.0f} KiB (factor {ff:.4f}), "
          f"WRITE_SIZE={w_raw:.0f} KiB (factor {wf:.4f})\n")
    sqk = sorted({c for l in lay for c in l["sq"]})
    print("| op | kind | lib | c_in->c_out | out | kernel | us (trace) | HBM read MB | HBM write MB | " +
          " | ".join(sqk) + " |")
    print("|" + "---|" * (9 + len(sqk)))
    for l in lay:
        print(f"| {l['op']} | {l['kind']} | {l['lib']} | {l['c_in']}->{l['c_out']} | {l['hw']} | {l['kernel']} | "
              f"{l['us']} | {l['fetch_mb']} | {l['write_mb']} | " +
              " | ".join(f"{l['sq'].get(c, 0):.4g}" for c in sqk) + " |")
    print(f"\npattern-pruned launches per frame: {len(pr)}, {traffic['us_per_frame']} us, "
          f"{traffic['bytes_per_frame'] / 1e6:.2f} MB HBM traffic")


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def measured_ceilings():
    """fp32 FMA throughput (TFLOP/s) and HBM copy bandwidth (GB/s, read +
    write) measured on this GPU by libppceil.so's micro-benchmarks."""
    import ctypes
    path = os.path.join(ROOT, "paper_2004_11250_amd", "libppceil.so")
    if not os.path.exists(path):
        return {}
    lib = ctypes.CDLL(path)
    lib.pp_ceiling_fma.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    lib.pp_ceiling_copy.argtypes = [ctypes.c_size_t, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    f, c = ctypes.c_double(0), ctypes.c_double(0)
    out = {}
    if lib.pp_ceiling_fma(256, ctypes.byref(f)) == 0:
        out["fma_tflops"] = round(f.value, 2)
    if lib.pp_ceiling_copy(1 << 30, 5, ctypes.byref(c)) == 0:
        out["copy_gbs"] = round(c.value, 1)
    return out


def other_workloads(dev, no_dense, steps=10, warmup=3):
    """ms/frame of the other evaluated networks (style transfer, super
    resolution, colourization; fp32 and bf16) and of the VGG-16 stack in
    bf16, and of the same masked models run dense through torch, for the
    speedup."""
    import torch
    import torch.nn.functional as F

    import paper_2004_11250_amd as pp
    import workloads
    stream = torch.cuda.current_stream()
    out = []
    for cfg, dts in ((2, ("bf16",)), (3, ("f32", "bf16")), (4, ("f32", "bf16")), (5, ("f32", "bf16"))):
        spec = workloads.net_spec(cfg)
        params = workloads.net_params(cfg)
        shapes = layer_shapes(spec)
        for dtype in dts:
            tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
            net = pp.Net(spec["ops"], params, dtype, device=dev)
            x = torch.from_numpy(workloads.net_input(cfg)).to(dev).to(tdt)
            nbytes, oshape = net.plan(*x.shape)
            ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
            y = torch.empty(oshape, dtype=tdt, device=dev)

            def timed(fn, min_ms=50.0):
                # at least `steps` frames and about min_ms of them, so that
                # short frames are not timed over a handful of calls
                for _ in range(warmup):
                    fn()
                torch.cuda.synchronize()
                a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a0.record(stream)
                fn()
                a1.record(stream)
                torch.cuda.synchronize()
                k = max(steps, min(1000, int(min_ms / max(a0.elapsed_time(a1), 1e-3)) + 1))
                a0.record(stream)
                for _ in range(k):
                    fn()
                a1.record(stream)
                torch.cuda.synchronize()
                return a0.elapsed_time(a1) / k

            ms = timed(lambda: net.forward(x, y, ws))
            macs = sum(surviving_macs(op, prm, o, spec["batch"]) for (i, op, _, o), prm in zip(shapes, params))
            entry = dict(workload=WORKLOADS[cfg], dtype=dtype, ms_per_frame=round(ms, 4),
                         eff_gmacs=round(macs / (ms * 1e-3) / 1e9, 1))
            if not no_dense:
                dw = []
                for (i, op, _, o), prm in zip(shapes, params):
                    if op["op"] == "conv3":
                        m = np.zeros(prm["conn"].shape + (9,), np.float32)
                        for pi, mask in enumerate(prm["lib"]):
                            bits = np.array([(int(mask) >> t) & 1 for t in range(9)], np.float32)
                            m[(prm["pid"] == pi) & (prm["conn"] != 0)] = bits
                        dw.append((torch.from_numpy(prm["w"] * m.reshape(prm["w"].shape)).to(dev).to(tdt),
                                   torch.from_numpy(prm["b"]).to(dev).to(tdt)))
                    elif op["op"] in ("conv", "deconv"):
                        dw.append((torch.from_numpy(prm["w"]).to(dev).to(tdt), torch.from_numpy(prm["b"]).to(dev).to(tdt)))
                    else:
                        dw.append(None)

                def dense_frame():
                    sl = {0: x}
                    for (i, op, _, o), wb in zip(shapes, dw):
                        src = sl[op["src"]]
                        if op["op"] in ("conv3", "conv"):
                            r = F.conv2d(src, wb[0], wb[1], stride=op["stride"], padding=op["pad"], dilation=op["dil"])
                            r = torch.relu(r) if op["relu"] else r
                        elif op["op"] == "deconv":
                            r = F.conv_transpose2d(src, wb[0], wb[1], stride=op["stride"], padding=op["pad"])
                            r = torch.relu(r) if op["relu"] else r
                        elif op["op"] == "maxpool2":
                            r = F.max_pool2d(src, 2)
                        elif op["op"] == "up2":
                            r = F.interpolate(src, scale_factor=2, mode="nearest")
                        elif op["op"] == "pshuf2":
                            r = F.pixel_shuffle(src, 2)
                        else:
                            r = src + sl[op["src2"]]
                        sl[op["dst"]] = r
                    return sl[1]

                torch.backends.cudnn.benchmark = True
                with torch.no_grad():
                    dms = timed(dense_frame)
                entry.update(dense_ms_per_frame=round(dms, 4), speedup=round(dms / ms, 3))
                del dw
            out.append(entry)
            del net, ws, y, x
            torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense comparator")
    ap.add_argument("--layer-steps", type=int, default=100)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="first run one elementwise fp32 copy of this many MiB (reads and writes exactly that "
                         "much), the reference for scaling hardware byte counters")
    ap.add_argument("--summarize-profile", metavar="DIR", default=None,
                    help="summarise rocprofv3 output under DIR (no GPU needed) and exit")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the other workloads' frame times (configs 3-5, reported beside the headline)")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the measured FMA / HBM ceilings")
    args = ap.parse_args()
    if args.summarize_profile:
        summarize_profile(args.summarize_profile, args.config)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2004_11250_amd as pp
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg, dtype = args.config, args.dtype
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    shapes = layer_shapes(spec)
    batch = spec["batch"]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    t0 = time.time()
    net = pp.Net(spec["ops"], params, dtype, device=dev)
    pack_s = time.time() - t0
    x = torch.from_numpy(workloads.net_input(cfg)).to(dev).to(tdt)
    nbytes, oshape = net.plan(*x.shape)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    y = torch.empty(oshape, dtype=tdt, device=dev)
    stream = torch.cuda.current_stream()

    if args.copy_mib > 0:
        n = args.copy_mib * (1 << 20) // 4
        ca = torch.rand(n, device=dev)
        cb = torch.empty_like(ca)
        torch.mul(ca, 1.0, out=cb)
        torch.cuda.synchronize()
        del ca, cb

    # ---- whole-frame timing: pp_net_fwd launched on the stream (the headline
    # figure), and the same call captured once as a HIP graph and replayed
    # (reported beside it)
    for _ in range(args.warmup):
        net.forward(x, y, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.time()
    e0.record(stream)
    for _ in range(args.steps):
        net.forward(x, y, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.time() - t_wall) * 1e3 / args.steps
    ms = e0.elapsed_time(e1) / args.steps
    # per-frame distribution: the same frames, each between its own events
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for i in range(args.steps):
        net.forward(x, y, ws)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    frame_pct = dict(p10=round(float(np.percentile(per, 10)), 5), p50=round(float(np.percentile(per, 50)), 5),
                     p90=round(float(np.percentile(per, 90)), 5), frames=args.steps)
    graph = net.capture(x, y, ws)
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1) / args.steps
    del graph

    total_macs = sum(surviving_macs(op, prm, o, batch) for (i, op, _, o), prm in zip(shapes, params))
    value = total_macs / (ms * 1e-3) / 1e9

    # ---- per-layer timing of the pruned-conv kernel (same launches as in the
    # frame: a conv whose next op pp_net_fwd fuses runs with that op's flag,
    # and with the prepared weights the net reads; an accumulating conv adds
    # into the same tensor every call)
    layers = []
    li = 0
    esz = 2 if dtype == "bf16" else 4
    pdt = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    fused = net.launch_plan(spec["batch"], spec["c"], spec["h"], spec["w"])["fused"]
    for (i, op, ishape, o), prm in zip(shapes, params):
        if op["op"] != "conv3":
            continue
        L = net.pruned[li]
        li += 1
        f = fused.get(i + 1)
        f = None if f == "up2" else f
        up = fused.get(i - 1) == "up2"
        if f == "maxpool2":
            o = (o[0], o[1] // 2, o[2] // 2)
        elif f == "pshuf2":
            o = (o[0] // 4, 2 * o[1], 2 * o[2])
        if up:
            ishape = (ishape[0], ishape[1] // 2, ishape[2] // 2)   # read as stored, upsampled on load
        # with the layer's prepared weights when the net has them (it passes
        # them to pp_net_fwd), and split scratch behind them
        kw = dict(relu=op["relu"], maxpool2=f == "maxpool2", accumulate=f == "add", pixshuf2=f == "pshuf2",
                  upsample2=up, prepared=L.prepared is not None)
        xin = torch.rand((batch,) + ishape, device=dev).to(tdt)
        yo = torch.zeros((batch,) + o, device=dev, dtype=tdt)
        for _ in range(5):
            pp.conv2d_fwd(L, xin, out=yo, **kw)
        torch.cuda.synchronize()
        # the launches recorded in a graph and replayed: the layer's GPU time
        # (a host loop of calls would be bound by the calls themselves for
        # the shortest layers)
        gr = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            with torch.cuda.graph(gr, stream=side):
                for _ in range(args.layer_steps):
                    pp.conv2d_fwd(L, xin, out=yo, **kw)
        gr.replay()
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        gr.replay()
        a1.record(stream)
        torch.cuda.synchronize()
        del gr
        us = a0.elapsed_time(a1) * 1e3 / args.layer_steps
        macs = surviving_macs(op, prm, shapes[i][3], batch)
        # the form the planner runs: the vector-ALU kernels, or (bf16) the
        # matrix-core form, which does the layer's whole masked dense contraction
        hin, win = (2 * ishape[1], 2 * ishape[2]) if up else (ishape[1], ishape[2])
        mfma = f != "maxpool2" and pp.conv2d_recipe(L.h_blob, batch, hin, win, pdt) == MFMA_RECIPE
        co = shapes[i][3]
        dense_macs = batch * co[1] * co[2] * co[0] * 9 * op["c_in"]
        # the residual of an accumulating conv is read as well as written
        alg_bytes = batch * (int(np.prod(ishape)) + (2 if f == "add" else 1) * int(np.prod(o))) * esz + \
            L.h_blob.nbytes
        layers.append(dict(op=i, c_in=op["c_in"], c_out=op["c_out"], hw=f"{o[1]}x{o[2]}", lib=op["lib"],
                           fused=f, upsample2_in=up,
                           form="mfma" if mfma else "vector", dense_mmac=round(dense_macs / 1e6, 3),
                           surviving_mmac=round(macs / 1e6, 3), us=round(us, 3),
                           eff_tmacs=round(macs / us / 1e6, 3), alg_mb=round(alg_bytes / 1e6, 3),
                           frac_fp32_peak=round(2 * macs / us / 1e6 / PEAK_FP32_VECTOR_TFLOPS, 4)))
        del xin, yo
    pr = [l for l in layers if l["lib"] == "canon8" and l["form"] == "vector"]
    pr_macs = sum(l["surviving_mmac"] for l in pr) * 1e6
    pr_us = sum(l["us"] for l in pr)
    achieved = 2 * pr_macs / (pr_us * 1e-6) / 1e12 if pr_us else 0.0
    mf = [l for l in layers if l["form"] == "mfma"]
    mf_us = sum(l["us"] for l in mf)
    traffic = None
    if cfg == 2 and dtype == "f32" and os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
        if t.get("kernel_source_sha256") == kernel_source_hash():
            traffic = t["bytes_per_frame"]
    ceil = measured_ceilings() if not args.no_ceilings else {}
    roofline = dict(bound="alu", achieved=round(achieved, 3), peak=PEAK_FP32_VECTOR_TFLOPS, unit="TFLOP/s",
                    frac=round(achieved / PEAK_FP32_VECTOR_TFLOPS, 4), traffic=traffic,
                    kernel=f"pattern-pruned 3x3 conv kernels (the {len(pr)} pruned layers on the vector ALUs, "
                           "summed over the frame)")
    if ceil.get("fma_tflops"):
        roofline.update(peak_measured=ceil["fma_tflops"], frac_measured=round(achieved / ceil["fma_tflops"], 4),
                        hbm_measured_gbs=ceil.get("copy_gbs"))
    if mf_us > pr_us:
        # the bf16 matrix-core form dominates: its contraction (the masked
        # dense conv) against the bf16 dense matrix peak
        mf_achieved = 2 * sum(l["dense_mmac"] for l in mf) * 1e6 / (mf_us * 1e-6) / 1e12
        roofline = dict(bound="mfma", achieved=round(mf_achieved, 3), peak=PEAK_BF16_MFMA_TFLOPS, unit="TFLOP/s",
                        frac=round(mf_achieved / PEAK_BF16_MFMA_TFLOPS, 4), traffic=None,
                        kernel=f"bf16 matrix-core form of the pruned 3x3 convs (the {len(mf)} layers the planner "
                               "puts there: weight expansion + implicit GEMM, summed over the frame)")

    # ---- dense comparator: the same masked model as dense convs (torch / MIOpen)
    dense = None
    if not args.no_dense:
        import torch.nn.functional as F
        torch.backends.cudnn.benchmark = True
        dw = []
        for (i, op, _, o), prm in zip(shapes, params):
            if op["op"] == "conv3":
                m = np.zeros(prm["conn"].shape + (9,), np.float32)
                for p, mask in enumerate(prm["lib"]):
                    bits = np.array([(int(mask) >> t) & 1 for t in range(9)], np.float32)
                    m[(prm["pid"] == p) & (prm["conn"] != 0)] = bits
                wm = prm["w"] * m.reshape(prm["w"].shape)
                dw.append((torch.from_numpy(wm).to(dev).to(tdt), torch.from_numpy(prm["b"]).to(dev).to(tdt)))
            elif op["op"] in ("conv", "deconv"):
                dw.append((torch.from_numpy(prm["w"]).to(dev).to(tdt), torch.from_numpy(prm["b"]).to(dev).to(tdt)))
            else:
                dw.append(None)

        def dense_frame(xx):
            sl = {0: xx}
            for (i, op, _, o), wb in zip(shapes, dw):
                src = sl[op["src"]]
                if op["op"] in ("conv3", "conv"):
                    r = F.conv2d(src, wb[0], wb[1], stride=op["stride"], padding=op["pad"], dilation=op["dil"])
                    r = torch.relu(r) if op["relu"] else r
                elif op["op"] == "deconv":
                    r = F.conv_transpose2d(src, wb[0], wb[1], stride=op["stride"], padding=op["pad"])
                    r = torch.relu(r) if op["relu"] else r
                elif op["op"] == "maxpool2":
                    r = F.max_pool2d(src, 2)
                elif op["op"] == "up2":
                    r = F.interpolate(src, scale_factor=2, mode="nearest")
                elif op["op"] == "pshuf2":
                    r = F.pixel_shuffle(src, 2)
                else:
                    r = src + sl[op["src2"]]
                sl[op["dst"]] = r
            return sl[1]

        with torch.no_grad():
            for _ in range(args.warmup):
                dense_frame(x)
            torch.cuda.synchronize()
            d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            d0.record(stream)
            for _ in range(args.steps):
                dense_frame(x)
            d1.record(stream)
            torch.cuda.synchronize()
            # the comparator computes the same function: its output against ours
            yd = dense_frame(x).float()
            net.forward(x, y, ws)
            torch.cuda.synchronize()
            diff = float((yd - y.float()).abs().max() / yd.abs().max().clamp_min(1e-30))
        dms = d0.elapsed_time(d1) / args.steps
        dense = dict(ms_per_frame=round(dms, 4), speedup=round(dms / ms, 3), max_rel_diff=float(f"{diff:.3e}"),
                     impl="torch.nn.functional (MIOpen) on the masked dense weights, same dtype")

    # ---- CPU oracle baseline (rank 0, N=1)
    cpu = None
    if not args.no_cpu:
        from threadpoolctl import threadpool_info, threadpool_limits

        from oracle import net as onet
        x_np = workloads.net_input(cfg)
        affinity = len(os.sched_getaffinity(0))
        reps, t_cpu = 0, 0.0
        while t_cpu < 10.0 and reps < 20:
            t = time.time()
            onet.run_net(spec, params, x_np, dtype)
            t_cpu += time.time() - t
            reps += 1
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        # the same frame on one core (one BLAS thread), one frame
        with threadpool_limits(limits=1):
            t = time.time()
            onet.run_net(spec, params, x_np, dtype)
            t1 = time.time() - t
        cpu = dict(value=round(total_macs * reps / t_cpu / 1e9, 4), unit="GMAC/s", cores=int(min(threads, affinity)),
                   kind="oracle", affinity_cpus=affinity, cpu_model=cpu_model(),
                   one_core=dict(value=round(total_macs / t1 / 1e9, 4), unit="GMAC/s", ms_per_frame=round(t1 * 1e3, 1)),
                   sample=f"{reps} full frame(s) of the same workload through the fp64 oracle on "
                          f"{min(threads, affinity)} BLAS threads ({t_cpu:.1f} s, {t_cpu / reps * 1e3:.0f} ms/frame), "
                          f"and one frame on one thread ({t1:.1f} s)")

    others = None
    if not args.no_others and cfg == 2 and dtype == "f32":
        others = other_workloads(dev, args.no_dense)

    line = dict(metric="effective GMAC/s (surviving MACs) per pruned 3x3 layer; ms/frame VGG-16 batch 1",
                value=round(value, 3), unit="GMAC/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
                ms_per_step=round(ms, 5), higher_is_better=True, scaling="weak", vs_baseline=None,
                dtype=dtype, data="synthetic",
                config=dict(workload=WORKLOADS[cfg], batch=batch, input=[spec["c"], spec["h"], spec["w"]],
                            surviving_gmac_per_frame=round(total_macs / 1e9, 4), library="canon8 4-of-9",
                            parallelism="single GPU"),
                wall_ms_per_step=round(wall_ms, 5), ms_per_frame_pct=frame_pct,
                ms_per_step_graph_replay=round(ms_graph, 5), pack_s=round(pack_s, 3),
                roofline=roofline, cpu_baseline=cpu, dense=dense, other_workloads=others, layers=layers)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
