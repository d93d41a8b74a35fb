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

PEAK_FP32_VECTOR_TFLOPS = 157.3     # MI355X: 256 CU x 2.4 GHz x 256 FLOP/clk (packed fp32)
PEAK_FP32_SCALAR_FMA_TFLOPS = 78.6  # same without packed fp32 (128 FLOP/clk/CU)
PEAK_HBM_GBS = 8000.0

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
    args = ap.parse_args()
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

    # ---- whole-frame timing
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

    total_macs = sum(surviving_macs(op, prm, o, batch) for (i, op, _, o), prm in zip(shapes, params))
    value = total_macs / (ms * 1e-3) / 1e9

    # ---- per-layer timing of the pruned-conv kernel (same launches as in the frame)
    layers = []
    li = 0
    esz = 2 if dtype == "bf16" else 4
    for (i, op, ishape, o), prm in zip(shapes, params):
        if op["op"] != "conv3":
            continue
        L = net.layers[li]
        li += 1
        xin = torch.rand((batch,) + ishape, device=dev).to(tdt)
        yo = torch.empty((batch,) + o, device=dev, dtype=tdt)
        for _ in range(5):
            pp.conv2d_fwd(L, xin, relu=op["relu"], out=yo)
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        for _ in range(args.layer_steps):
            pp.conv2d_fwd(L, xin, relu=op["relu"], out=yo)
        a1.record(stream)
        torch.cuda.synchronize()
        us = a0.elapsed_time(a1) * 1e3 / args.layer_steps
        macs = surviving_macs(op, prm, o, batch)
        alg_bytes = batch * (int(np.prod(ishape)) + int(np.prod(o))) * esz + L.h_blob.nbytes
        layers.append(dict(op=i, c_in=op["c_in"], c_out=op["c_out"], hw=f"{o[1]}x{o[2]}", lib=op["lib"],
                           surviving_mmac=round(macs / 1e6, 3), us=round(us, 3),
                           eff_tmacs=round(macs / us / 1e6, 3), alg_mb=round(alg_bytes / 1e6, 3),
                           frac_fp32_peak=round(2 * macs / us / 1e6 / PEAK_FP32_VECTOR_TFLOPS, 4)))
        del xin, yo
    pr = [l for l in layers if l["lib"] == "canon8"]
    pr_macs = sum(l["surviving_mmac"] for l in pr) * 1e6
    pr_us = sum(l["us"] for l in pr)
    achieved = 2 * pr_macs / (pr_us * 1e-6) / 1e12 if pr_us else 0.0
    roofline = dict(bound="alu", achieved=round(achieved, 3), peak=PEAK_FP32_VECTOR_TFLOPS, unit="TFLOP/s",
                    frac=round(achieved / PEAK_FP32_VECTOR_TFLOPS, 4), traffic=None,
                    kernel="pp_conv3x3_kernel (pattern-pruned layers, summed over the frame)",
                    scalar_fma_peak=PEAK_FP32_SCALAR_FMA_TFLOPS)

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
            else:
                dw.append(None)

        def dense_frame(xx):
            sl = {0: xx}
            for (i, op, _, o), wb in zip(shapes, dw):
                src = sl[op["src"]]
                if op["op"] == "conv3":
                    r = F.conv2d(src, wb[0], wb[1], stride=op["stride"], padding=op["pad"], dilation=op["dil"])
                    r = torch.relu(r) if op["relu"] else r
                elif op["op"] == "maxpool2":
                    r = F.max_pool2d(src, 2)
                else:
                    raise ValueError("dense comparator covers the VGG ops only")
                sl[op["dst"]] = r
            return sl[1]

        if cfg in (1, 2):
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
            dms = d0.elapsed_time(d1) / args.steps
            dense = dict(ms_per_frame=round(dms, 4), speedup=round(dms / ms, 3), impl="torch.nn.functional.conv2d")

    # ---- CPU oracle baseline (rank 0, N=1)
    cpu = None
    if not args.no_cpu:
        from threadpoolctl import threadpool_info

        from oracle import net as onet
        x_np = workloads.net_input(cfg)
        reps, t_cpu = 0, 0.0
        while t_cpu < 10.0 and reps < 20:
            t = time.time()
            onet.run_net(spec, params, x_np, dtype)
            t_cpu += time.time() - t
            reps += 1
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        cpu = dict(value=round(total_macs * reps / t_cpu / 1e9, 4), unit="GMAC/s", cores=int(threads), kind="oracle",
                   sample=f"{reps} full frame(s) of the same workload through the fp64 oracle "
                          f"({t_cpu:.1f} s, {t_cpu / reps * 1e3:.0f} ms/frame)")

    line = dict(metric="effective GMAC/s (surviving MACs) per pruned 3x3 layer; ms/frame VGG-16 batch 1",
                value=round(value, 3), unit="GMAC/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
                ms_per_step=round(ms, 5), higher_is_better=True, scaling="weak", vs_baseline=None,
                dtype=dtype, data="synthetic",
                config=dict(workload=WORKLOADS[cfg], batch=batch, input=[spec["c"], spec["h"], spec["w"]],
                            surviving_gmac_per_frame=round(total_macs / 1e9, 4), library="canon8 4-of-9",
                            parallelism="single GPU"),
                wall_ms_per_step=round(wall_ms, 5), pack_s=round(pack_s, 3),
                roofline=roofline, cpu_baseline=cpu, dense=dense, layers=layers)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
