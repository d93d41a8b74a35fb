"""Seeded synthetic inputs shaped like the paper's workloads.

This module is the only code shared by the CPU oracle (``oracle/``) and the
GPU path (``paper_2004_11250_amd``).  It draws random numbers and lists the
layers of each network; it performs none of the method's arithmetic (no
convolution, no masking, no packing, no shape arithmetic).

The paper evaluates style transfer, colouring and super resolution and cites
VGG-16 as the canonical heavy network (Sec. 1 and Sec. 4); it gives no input
resolutions, pruning rates or precision, so the shapes below are fixed here:

  1. one pruned 3x3 layer 16->16 at 32x32, fp32;
  2. VGG-16 conv stack at 224x224, batch 1, fp32;
  3. a Johnson-style style-transfer net at 512x512, fp32;
  4. an EDSR-like super-resolution body, 270x480 -> 1080x1920, fp32/bf16;
  5. a colourisation encoder-decoder at 256x256, batch 8, fp32/bf16.

Random draws use ``numpy.random.Generator(PCG64(SeedSequence([2004_11250,
cfg, layer])))``; per layer the draw order is W, b, pattern ids, connectivity.
The network input uses layer index 999.
"""
from __future__ import annotations

import numpy as np

SEED_ROOT = 2004_11250
INPUT_LAYER = 999

# Pattern library used for every pattern-pruned layer: eight 4-of-9 patterns,
# each containing the centre tap.  Tap t = 3*ky + kx, bit t of the 9-bit mask.
# Four "T" shapes, then the four 2x2 blocks that contain the centre.
CANON8 = (0x03A, 0x0B2, 0x0B8, 0x09A, 0x01B, 0x036, 0x0D8, 0x1B0)
# Library of a dense 3x3 layer: one pattern with all nine taps.
DENSE9 = (0x1FF,)


def rng_for(cfg: int, layer: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, cfg, layer])))


# --------------------------------------------------------------------------
# network specs: ordered op lists over activation slots.
# slot 0 = network input, slot 1 = network output, slots >= 2 = workspace.
# ops:
#   conv3     3x3 conv through the pattern-pruned path (lib 'canon8' or 'dense9')
#   conv      dense k x k conv (k = 9 or 1 here)
#   deconv    dense transposed conv (k = 4, stride 2, pad 1)
#   maxpool2  2x2 max pool, stride 2
#   up2       nearest-neighbour upsample x2
#   pshuf2    PixelShuffle(2)
#   add       dst = src + src2 (residual; no activation after it)
# --------------------------------------------------------------------------

def _conv3(src, dst, cin, cout, *, stride=1, dil=1, relu=True, lib="canon8", keep=None,
           wscale=1.0):
    return dict(op="conv3", src=src, dst=dst, c_in=cin, c_out=cout, stride=stride,
                pad=dil, dil=dil, relu=relu, lib=lib, keep=keep, wscale=wscale)


def _conv(src, dst, cin, cout, k, *, relu=True):
    return dict(op="conv", src=src, dst=dst, c_in=cin, c_out=cout, k=k, stride=1,
                pad=k // 2, dil=1, relu=relu)


def vgg16_spec():
    keep = 1.0 / 3.0
    ops = [_conv3(0, 2, 3, 64, lib="dense9")]
    chans = [(64, 64), "P", (64, 128), (128, 128), "P", (128, 256), (256, 256), (256, 256), "P",
             (256, 512), (512, 512), (512, 512), "P", (512, 512), (512, 512), (512, 512), "P"]
    cur = 2
    for i, ch in enumerate(chans):
        nxt = 3 if cur == 2 else 2
        last = i == len(chans) - 1
        dst = 1 if last else nxt
        if ch == "P":
            ops.append(dict(op="maxpool2", src=cur, dst=dst))
        else:
            ops.append(_conv3(cur, dst, ch[0], ch[1], keep=keep))
        cur = dst
    return dict(name="vgg16", batch=1, c=3, h=224, w=224, ops=ops)


def layer1_spec():
    return dict(name="layer16", batch=1, c=16, h=32, w=32,
                ops=[_conv3(0, 1, 16, 16, keep=0.5)])


def style_spec():
    keep = 0.5
    ops = [_conv(0, 2, 3, 32, 9),
           _conv3(2, 3, 32, 64, stride=2, keep=keep),
           _conv3(3, 2, 64, 128, stride=2, keep=keep)]
    cur, a, b = 2, 3, 4
    for _ in range(5):
        ops.append(_conv3(cur, a, 128, 128, keep=keep))
        ops.append(_conv3(a, b, 128, 128, keep=keep, relu=False))
        ops.append(dict(op="add", src=cur, src2=b, dst=a))
        cur, a = a, cur
    ops.append(dict(op="up2", src=cur, dst=a))
    ops.append(_conv3(a, b, 128, 64, keep=keep))
    ops.append(dict(op="up2", src=b, dst=a))
    ops.append(_conv3(a, b, 64, 32, keep=keep))
    ops.append(_conv(b, 1, 32, 3, 9, relu=False))
    return dict(name="style", batch=1, c=3, h=512, w=512, ops=ops)


def sr_spec():
    keep = 0.5
    ops = [_conv3(0, 2, 3, 64, lib="dense9")]
    cur, a, b = 2, 3, 4
    for _ in range(16):
        ops.append(_conv3(cur, a, 64, 64, keep=keep, wscale=0.1))
        ops.append(_conv3(a, b, 64, 64, keep=keep, relu=False, wscale=0.1))
        ops.append(dict(op="add", src=cur, src2=b, dst=a))
        cur, a = a, cur
    for _ in range(2):
        ops.append(_conv3(cur, a, 64, 256, keep=keep, relu=False))
        ops.append(dict(op="pshuf2", src=a, dst=b))
        cur, a, b = b, cur, a
    ops.append(_conv3(cur, 1, 64, 3, lib="dense9", relu=False))
    return dict(name="sr", batch=1, c=3, h=270, w=480, ops=ops)


def color_spec():
    keep = 0.3
    ops = [_conv3(0, 2, 1, 64, lib="dense9")]
    layers = [(64, 64, 2, 1), (64, 128, 1, 1), (128, 128, 2, 1), (128, 256, 1, 1), (256, 256, 1, 1),
              (256, 256, 2, 1), (256, 512, 1, 1), (512, 512, 1, 1), (512, 512, 1, 1),
              (512, 512, 1, 2), (512, 512, 1, 2), (512, 512, 1, 2)]
    cur, nxt = 2, 3
    for cin, cout, s, d in layers:
        ops.append(_conv3(cur, nxt, cin, cout, stride=s, dil=d, keep=keep))
        cur, nxt = nxt, cur
    ops.append(dict(op="deconv", src=cur, dst=nxt, c_in=512, c_out=256, k=4, stride=2, pad=1,
                    relu=True))
    cur, nxt = nxt, cur
    for _ in range(2):
        ops.append(_conv3(cur, nxt, 256, 256, keep=keep))
        cur, nxt = nxt, cur
    ops.append(_conv(cur, 1, 256, 313, 1, relu=False))
    return dict(name="color", batch=8, c=1, h=256, w=256, ops=ops)


SPECS = {1: layer1_spec, 2: vgg16_spec, 3: style_spec, 4: sr_spec, 5: color_spec}


def net_spec(cfg: int) -> dict:
    return SPECS[cfg]()


# --------------------------------------------------------------------------
# parameter and input draws
# --------------------------------------------------------------------------

def _kept_exact(rng, c_out, c_in, keep):
    """Connectivity mask keeping exactly round(keep*c_out*c_in) kernels, chosen
    by a seeded permutation."""
    total = c_out * c_in
    n = int(round(keep * total))
    conn = np.zeros(total, dtype=np.uint8)
    conn[rng.permutation(total)[:n]] = 1
    return conn.reshape(c_out, c_in)


def layer_params(cfg: int, index: int, op: dict) -> dict:
    """Weights and pruning structure of op number ``index`` of config ``cfg``."""
    rng = rng_for(cfg, index)
    kind = op["op"]
    if kind == "conv3":
        c_out, c_in = op["c_out"], op["c_in"]
        if cfg == 1:
            w = rng.normal(0.0, 0.1, size=(c_out, c_in, 3, 3)).astype(np.float32)
            b = rng.normal(0.0, 0.01, size=c_out).astype(np.float32)
        else:
            std = np.sqrt(2.0 / (c_in * 9)) * op.get("wscale", 1.0)
            w = rng.normal(0.0, std, size=(c_out, c_in, 3, 3)).astype(np.float32)
            b = np.zeros(c_out, dtype=np.float32)
        if op["lib"] == "dense9":
            lib = DENSE9
            pid = np.zeros((c_out, c_in), dtype=np.uint8)
            conn = np.ones((c_out, c_in), dtype=np.uint8)
        else:
            lib = CANON8
            pid = rng.integers(0, len(lib), size=(c_out, c_in), dtype=np.uint8)
            if cfg == 1:
                conn = (rng.random(size=(c_out, c_in)) >= 0.5).astype(np.uint8)
            else:
                conn = _kept_exact(rng, c_out, c_in, op["keep"])
        return dict(w=w, b=b, pid=pid, conn=conn, lib=np.array(lib, dtype=np.uint16))
    if kind in ("conv", "deconv"):
        c_out, c_in, k = op["c_out"], op["c_in"], op["k"]
        std = np.sqrt(2.0 / (c_in * k * k))
        if kind == "conv":
            w = rng.normal(0.0, std, size=(c_out, c_in, k, k)).astype(np.float32)
        else:  # transposed conv weight layout [c_in][c_out][k][k]
            w = rng.normal(0.0, std, size=(c_in, c_out, k, k)).astype(np.float32)
        b = np.zeros(c_out, dtype=np.float32)
        return dict(w=w, b=b)
    return {}


def net_params(cfg: int) -> list:
    spec = net_spec(cfg)
    return [layer_params(cfg, i, op) for i, op in enumerate(spec["ops"])]


def net_input(cfg: int) -> np.ndarray:
    spec = net_spec(cfg)
    rng = rng_for(cfg, INPUT_LAYER)
    shape = (spec["batch"], spec["c"], spec["h"], spec["w"])
    if cfg == 1:
        return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    return rng.uniform(0.0, 1.0, size=shape).astype(np.float32)


def random_layer(seed: int, c_out: int, c_in: int, *, lib=CANON8, keep=0.5, wstd=0.1,
                 bstd=0.01) -> dict:
    """A free-standing random pruned 3x3 layer (tests and fuzzing)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, 7, seed])))
    w = rng.normal(0.0, wstd, size=(c_out, c_in, 3, 3)).astype(np.float32)
    b = rng.normal(0.0, bstd, size=c_out).astype(np.float32)
    lib = np.array(lib, dtype=np.uint16)
    pid = rng.integers(0, len(lib), size=(c_out, c_in), dtype=np.uint8)
    conn = (rng.random(size=(c_out, c_in)) < keep).astype(np.uint8)
    return dict(w=w, b=b, pid=pid, conn=conn, lib=lib)


def random_input(seed: int, shape, lo=-1.0, hi=1.0) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, 8, seed])))
    return rng.uniform(lo, hi, size=shape).astype(np.float32)
