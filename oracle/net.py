"""Network runner for the oracle (test infrastructure only).

Runs the op lists of ``workloads.py`` with the oracle's own functions.  The
paper fuses each convolution with its activation (Sec. 3, "DSL related
optimization"); here an op is one layer including its ReLU.  Every op is
evaluated in fp64 on inputs stored in the activation dtype; its result is
then rounded to that dtype (fp32, or bf16 round-to-nearest-even) before it
feeds the next op, which is how the activations are stored between layers.
"""
from __future__ import annotations

import numpy as np

from . import bf16 as _bf16
from . import conv as _conv


def store(y, dtype: str) -> np.ndarray:
    """Round an fp64 activation once to its storage dtype (returned as fp32)."""
    y = np.asarray(y, dtype=np.float64)
    if dtype == "bf16":
        return _round_f64_to_bf16(y)
    return y.astype(np.float32)        # round to nearest even


def _round_f64_to_bf16(y: np.ndarray) -> np.ndarray:
    """Round fp64 -> bf16 (nearest, ties to even) in one step.  Rounding via
    fp32 gives the same answer except when the fp32 value lands exactly on a
    bf16 midpoint while the fp64 value does not; that case is decided here by
    the side of the midpoint the exact value lies on."""
    y32 = y.astype(np.float32)
    r = _bf16.round_f32(y32)
    bits = y32.view(np.uint32)
    tie = (bits & np.uint32(0xFFFF)) == np.uint32(0x8000)
    if np.any(tie):
        lo = (bits & np.uint32(0xFFFF0000)).view(np.float32)                     # toward zero
        hi = ((bits & np.uint32(0xFFFF0000)) + np.uint32(0x10000)).view(np.float32)  # away from zero
        mag, mid = np.abs(y), np.abs(y32.astype(np.float64))
        r = np.where(tie & (mag > mid), hi, np.where(tie & (mag < mid), lo, r))
    return r.astype(np.float32)


def weights_for(dtype: str, w) -> np.ndarray:
    w = np.asarray(w, dtype=np.float32)
    return _bf16.round_f32(w) if dtype == "bf16" else w


def run_op(op: dict, prm: dict, src, src2=None, dtype: str = "f32"):
    """One op on stored inputs.  Returns (fp64 result, fp64 bound S or None).
    S is |b| + sum |w||x| over the op's terms (None for ops that do no
    arithmetic beyond a single rounding-free selection)."""
    kind = op["op"]
    if kind == "conv3":
        w = weights_for(dtype, prm["w"])
        args = (src, w, prm["b"], prm["pid"], prm["conn"], prm["lib"])
        kw = dict(stride=op["stride"], pad=op["pad"], dil=op["dil"])
        return (_conv.conv3x3_pruned(*args, relu=op["relu"], **kw),
                _conv.conv3x3_bound(*args, **kw))
    if kind == "conv":
        w = weights_for(dtype, prm["w"])
        kw = dict(stride=op["stride"], pad=op["pad"], dil=op["dil"])
        return (_conv.conv2d(src, w, prm["b"], relu=op["relu"], **kw),
                _conv.conv2d_bound(src, w, prm["b"], **kw))
    if kind == "deconv":
        w = weights_for(dtype, prm["w"])
        return (_conv.conv_transpose2d(src, w, prm["b"], op["stride"], op["pad"], op["relu"]),
                _conv.conv_transpose2d_bound(src, w, prm["b"], op["stride"], op["pad"]))
    if kind == "maxpool2":
        return _conv.maxpool2(np.asarray(src, np.float64)), None
    if kind == "up2":
        return _conv.upsample2(np.asarray(src, np.float64)), None
    if kind == "pshuf2":
        return _conv.pixel_shuffle2(np.asarray(src, np.float64)), None
    if kind == "add":
        a = np.asarray(src, np.float64)
        b = np.asarray(src2, np.float64)
        return a + b, np.abs(a) + np.abs(b)
    raise ValueError(f"unknown op {kind}")


def run_net(spec: dict, params: list, x, dtype: str = "f32", keep_all: bool = False):
    """Run a whole network.  Returns the stored output, and with keep_all the
    list of (stored input(s), fp64 result, bound) per op as well."""
    slots = {0: store(x, dtype)}
    trace = []
    for op, prm in zip(spec["ops"], params):
        src = slots[op["src"]]
        src2 = slots.get(op.get("src2")) if "src2" in op else None
        y, bound = run_op(op, prm, src, src2, dtype)
        slots[op["dst"]] = store(y, dtype)
        if keep_all:
            trace.append(dict(src=src, src2=src2, y=y, bound=bound))
    return (slots[1], trace) if keep_all else slots[1]
