"""Independent writer and interpreter of the PPK1 packed-layer format
(test infrastructure only).

The paper stores the pruned weights in a format more compact than CSR: no
zero weights and no per-weight indices, because the pattern already says which
taps survive (Sec. 3, "sparse model storage").  It then reorders the filters so
that those with the same or similar patterns sit together, and compacts the
weights along the kernel direction (Sec. 3, "matrix reorder").

PPK1 layout (little-endian; every section starts on a 64-byte boundary; all
padding bytes are zero):

  header   24 x u32: magic 'PPK1', version | wdtype<<16, c_out, c_in, stride,
           pad, dilation, n_patterns, group (=8), n_groups, n_kept, n_wt,
           off_masks, off_perm, off_codes, off_woff, off_w, off_bias,
           total_bytes, 0, 0, 0, 0, 0
  masks    u16[n_patterns]               9-bit tap mask of each pattern
  perm     u32[n_groups*8]               packed slot -> original filter
                                         (0xFFFFFFFF for padding slots)
  codes    u8[n_groups][c_in][8]         pattern id of kernel (perm[8g+s], c),
                                         0xFF if the kernel is pruned
  woff     u32[n_groups*c_in + 1]        entry (g, c): bits 0..23 index of its
                                         first weight, bits 24..31 the mask of
                                         its kept slots (bit s = slot s kept);
                                         the last entry is n_wt (< 2^24)
  w        f32 or bf16 [n_wt]            for g, c, s ascending, kept kernels
                                         only: the pattern's taps in ascending
                                         tap order (bf16: padded to an even
                                         count with a zero element)
  bias     f32[n_groups*8]               bias in packed slot order

Filter order (the reorder): filters sorted by number of kept kernels
(descending), then by their pattern histogram (count of pattern 0, 1, ...,
each descending), then by filter index.  Slot group g holds sorted positions
8g .. 8g+7.
"""
from __future__ import annotations

import math
import struct

import numpy as np

from . import bf16 as _bf16

MAGIC = 0x314B5050
VERSION = 2
MAX_WT = (1 << 24) - 1
GROUP = 8
ALIGN = 64
HEADER_WORDS = 24
WD_F32, WD_BF16 = 0, 1
PRUNED = 0xFF
NO_FILTER = 0xFFFFFFFF


def _align(n: int) -> int:
    return (n + ALIGN - 1) // ALIGN * ALIGN


def _popcount(v: int) -> int:
    return bin(int(v)).count("1")


def _validate(w, b, pid, conn, lib, stride, pad, dil, wdtype):
    w = np.asarray(w, dtype=np.float32)
    if w.ndim != 4 or w.shape[2:] != (3, 3):
        raise ValueError("w must be [c_out][c_in][3][3]")
    c_out, c_in = w.shape[:2]
    if c_out < 1 or c_in < 1 or c_out > 65535 or c_in > 65535:
        raise ValueError("c_out/c_in out of range")
    lib = [int(m) for m in np.asarray(lib).ravel()]
    if not 1 <= len(lib) <= 255:
        raise ValueError("n_patterns must be 1..255")
    for m in lib:
        if not 1 <= m <= 0x1FF:
            raise ValueError("pattern mask must be a nonzero 9-bit value")
    pid = np.asarray(pid)
    conn = np.asarray(conn)
    if pid.shape != (c_out, c_in) or conn.shape != (c_out, c_in):
        raise ValueError("pattern_id/conn must be [c_out][c_in]")
    if np.any((conn != 0) & (conn != 1)):
        raise ValueError("conn must be 0/1")
    if np.any((conn == 1) & (pid.astype(np.int64) >= len(lib))):
        raise ValueError("pattern id out of range for a kept kernel")
    if not (1 <= stride <= 16 and 1 <= dil <= 16 and 0 <= pad <= 16):
        raise ValueError("stride/dilation/pad out of range")
    if wdtype not in (WD_F32, WD_BF16):
        raise ValueError("bad weight dtype")
    b = np.zeros(c_out, np.float32) if b is None else np.asarray(b, dtype=np.float32)
    if b.shape != (c_out,):
        raise ValueError("bias must be [c_out]")
    return w, b, pid.astype(np.int64), conn.astype(np.int64), lib


def filter_order(pid, conn, n_patterns) -> list:
    """The matrix reorder: original filter indices in packed order."""
    pid = np.asarray(pid, dtype=np.int64)
    conn = np.asarray(conn, dtype=np.int64)
    c_out = conn.shape[0]
    keys = []
    for o in range(c_out):
        kept = [int(pid[o, c]) for c in range(conn.shape[1]) if conn[o, c]]
        hist = [kept.count(p) for p in range(n_patterns)]
        keys.append((-len(kept), [-h for h in hist], o))
    keys.sort()
    return [k[2] for k in keys]


def pack(w, b, pid, conn, lib, stride=1, pad=1, dil=1, wdtype=WD_F32) -> bytes:
    w, b, pid, conn, lib = _validate(w, b, pid, conn, lib, stride, pad, dil, wdtype)
    c_out, c_in = w.shape[:2]
    n_p = len(lib)
    n_groups = (c_out + GROUP - 1) // GROUP
    slots = n_groups * GROUP
    order = filter_order(pid, conn, n_p)
    perm = order + [NO_FILTER] * (slots - c_out)

    codes = bytearray([PRUNED]) * (n_groups * c_in * GROUP)
    woff = []
    wvals = []           # float32 values (fp32) or uint16 bit patterns (bf16)
    n_kept = 0
    wflat = w.reshape(c_out, c_in, 9)
    for g in range(n_groups):
        for c in range(c_in):
            woff.append(len(wvals))
            kept_mask = 0
            for s in range(GROUP):
                o = perm[GROUP * g + s]
                if o == NO_FILTER or not conn[o, c]:
                    continue
                p = int(pid[o, c])
                codes[(g * c_in + c) * GROUP + s] = p
                kept_mask |= 1 << s
                n_kept += 1
                taps = [t for t in range(9) if (lib[p] >> t) & 1]
                vals = [wflat[o, c, t] for t in taps]
                if wdtype == WD_BF16:
                    bits = [int(v) for v in _bf16.round_bits(np.array(vals, np.float32))]
                    if len(bits) % 2:
                        bits.append(0)
                    wvals.extend(bits)
                else:
                    wvals.extend(float(v) for v in vals)
            woff[-1] |= kept_mask << 24
    woff.append(len(wvals))
    n_wt = len(wvals)
    if n_wt > MAX_WT:
        raise ValueError("layer has too many weights for 24-bit offsets")

    off_masks = _align(HEADER_WORDS * 4)
    off_perm = _align(off_masks + 2 * n_p)
    off_codes = _align(off_perm + 4 * slots)
    off_woff = _align(off_codes + len(codes))
    off_w = _align(off_woff + 4 * len(woff))
    wbytes = (2 if wdtype == WD_BF16 else 4) * n_wt
    off_bias = _align(off_w + wbytes)
    total = _align(off_bias + 4 * slots)

    out = bytearray(total)
    hdr = [MAGIC, VERSION | (wdtype << 16), c_out, c_in, stride, pad, dil, n_p, GROUP, n_groups,
           n_kept, n_wt, off_masks, off_perm, off_codes, off_woff, off_w, off_bias, total, 0, 0, 0,
           0, 0]
    struct.pack_into("<24I", out, 0, *hdr)
    struct.pack_into(f"<{n_p}H", out, off_masks, *lib)
    struct.pack_into(f"<{slots}I", out, off_perm, *perm)
    out[off_codes:off_codes + len(codes)] = codes
    struct.pack_into(f"<{len(woff)}I", out, off_woff, *woff)
    if wdtype == WD_BF16:
        struct.pack_into(f"<{n_wt}H", out, off_w, *wvals)
    else:
        struct.pack_into(f"<{n_wt}f", out, off_w, *wvals)
    pbias = [float(b[o]) if o != NO_FILTER else 0.0 for o in perm]
    struct.pack_into(f"<{slots}f", out, off_bias, *pbias)
    return bytes(out)


def parse(blob: bytes) -> dict:
    """Read a PPK1 blob back into numpy arrays (no validation beyond shape)."""
    hdr = struct.unpack_from("<24I", blob, 0)
    if hdr[0] != MAGIC:
        raise ValueError("bad magic")
    (c_out, c_in, stride, pad, dil, n_p, group, n_groups, n_kept, n_wt, off_masks, off_perm,
     off_codes, off_woff, off_w, off_bias, total) = hdr[2:19]
    wdtype = hdr[1] >> 16
    slots = n_groups * group
    d = dict(c_out=c_out, c_in=c_in, stride=stride, pad=pad, dil=dil, n_patterns=n_p,
             group=group, n_groups=n_groups, n_kept=n_kept, n_wt=n_wt, wdtype=wdtype,
             total_bytes=total, version=hdr[1] & 0xFFFF,
             offsets=dict(masks=off_masks, perm=off_perm, codes=off_codes, woff=off_woff,
                          w=off_w, bias=off_bias))
    d["masks"] = np.frombuffer(blob, "<u2", n_p, off_masks).copy()
    d["perm"] = np.frombuffer(blob, "<u4", slots, off_perm).copy()
    d["codes"] = np.frombuffer(blob, "u1", n_groups * c_in * group, off_codes).reshape(
        n_groups, c_in, group).copy()
    woff = np.frombuffer(blob, "<u4", n_groups * c_in + 1, off_woff).copy()
    d["woff"] = woff & np.uint32(MAX_WT)
    d["kept_mask"] = (woff >> np.uint32(24)).astype(np.uint8)
    if wdtype == WD_BF16:
        d["w"] = _bf16.bits_to_f32(np.frombuffer(blob, "<u2", n_wt, off_w))
    else:
        d["w"] = np.frombuffer(blob, "<f4", n_wt, off_w).copy()
    d["bias"] = np.frombuffer(blob, "<f4", slots, off_bias).copy()
    return d


def _kernel_list(d: dict):
    """Yield (o, c, [(tap, weight), ...]) for every kept kernel, walking the
    blob in packed order."""
    masks, perm, codes, woff, w = d["masks"], d["perm"], d["codes"], d["woff"], d["w"]
    for g in range(d["n_groups"]):
        for c in range(d["c_in"]):
            pos = int(woff[g * d["c_in"] + c])
            for s in range(d["group"]):
                p = int(codes[g, c, s])
                if p == PRUNED:
                    continue
                taps = [t for t in range(9) if (int(masks[p]) >> t) & 1]
                yield int(perm[d["group"] * g + s]), c, list(zip(taps, w[pos:pos + len(taps)]))
                k = len(taps)
                if d["wdtype"] == WD_BF16 and k % 2:
                    k += 1
                pos += k


def interp(blob: bytes, x, relu=False) -> np.ndarray:
    """Evaluate the layer by walking the packed blob; fp64 accumulation."""
    d = parse(blob)
    x = np.asarray(x, dtype=np.float64)
    n, c_in, h, wd = x.shape
    assert c_in == d["c_in"]
    s, p, dl = d["stride"], d["pad"], d["dil"]
    ho = (h + 2 * p - 2 * dl - 1) // s + 1
    wo = (wd + 2 * p - 2 * dl - 1) // s + 1
    xp = np.zeros((n, c_in, h + 2 * p, wd + 2 * p), dtype=np.float64)
    xp[:, :, p:p + h, p:p + wd] = x
    y = np.zeros((n, d["c_out"], ho, wo), dtype=np.float64)
    for o, c, taps in _kernel_list(d):
        for t, wv in taps:
            ky, kx = divmod(t, 3)
            r0, c0 = ky * dl, kx * dl
            y[:, o] += float(wv) * xp[:, c, r0:r0 + s * (ho - 1) + 1:s, c0:c0 + s * (wo - 1) + 1:s]
    for i, o in enumerate(d["perm"]):
        if o != NO_FILTER:
            y[:, o] += float(d["bias"][i])
    if relu:
        y = np.maximum(y, 0.0)
    return y


def interp_fsum(blob: bytes, x, relu=False) -> np.ndarray:
    """As interp, but every output is math.fsum of its exact terms (tiny inputs)."""
    d = parse(blob)
    x = np.asarray(x, dtype=np.float64)
    n, c_in, h, wd = x.shape
    s, p, dl = d["stride"], d["pad"], d["dil"]
    ho = (h + 2 * p - 2 * dl - 1) // s + 1
    wo = (wd + 2 * p - 2 * dl - 1) // s + 1
    terms = {}
    for o, c, taps in _kernel_list(d):
        for t, wv in taps:
            ky, kx = divmod(t, 3)
            for nn in range(n):
                for yy in range(ho):
                    iy = yy * s + ky * dl - p
                    if not 0 <= iy < h:
                        continue
                    for xx in range(wo):
                        ix = xx * s + kx * dl - p
                        if 0 <= ix < wd:
                            terms.setdefault((nn, o, yy, xx), []).append(float(wv) * float(x[nn, c, iy, ix]))
    bias = {int(o): float(d["bias"][i]) for i, o in enumerate(d["perm"]) if o != NO_FILTER}
    y = np.zeros((n, d["c_out"], ho, wo), dtype=np.float64)
    for nn in range(n):
        for o in range(d["c_out"]):
            for yy in range(ho):
                for xx in range(wo):
                    v = math.fsum(terms.get((nn, o, yy, xx), []) + [bias[o]])
                    y[nn, o, yy, xx] = max(v, 0.0) if relu else v
    return y


def unpack_dense(blob: bytes):
    """Recover (w_masked [c_out][c_in][3][3] fp64, bias [c_out]) from a blob."""
    d = parse(blob)
    w = np.zeros((d["c_out"], d["c_in"], 9), dtype=np.float64)
    for o, c, taps in _kernel_list(d):
        for t, wv in taps:
            w[o, c, t] = float(wv)
    b = np.zeros(d["c_out"], dtype=np.float64)
    for i, o in enumerate(d["perm"]):
        if o != NO_FILTER:
            b[o] = float(d["bias"][i])
    return w.reshape(d["c_out"], d["c_in"], 3, 3), b
