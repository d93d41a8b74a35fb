"""Direct-convolution oracle (test infrastructure only).

A pattern- and connectivity-pruned 3x3 layer (Sec. 2 of the paper: pattern
pruning removes fixed locations inside each kernel, connectivity pruning
removes whole kernels) computes exactly what a dense convolution computes with
the pruned taps set to zero.  The oracle is that definition written out:

    M[o,c,t]   = conn[o,c] * bit_t(lib[pid[o,c]])        t = 3*ky + kx
    y[n,o,h,w] = b[o] + sum_{c,ky,kx} M[o,c,t] W[o,c,ky,kx]
                        * x[n, c, h*s + ky*d - p, w*s + kx*d - p]

with x = 0 outside the image (zero padding), cross-correlation (no kernel
flip), and y = max(y, 0) when the layer is followed by ReLU (the paper fuses
conv + activation, Sec. 3, "DSL related optimization").  Everything is
accumulated in fp64; fp32 x fp32 products are exact in fp64.

The per-tap sum over input channels uses a matrix product (numpy.tensordot);
no other blocking or reordering is applied.
"""
from __future__ import annotations

import math

import numpy as np


def out_size(h: int, k: int, stride: int, pad: int, dil: int) -> int:
    return (h + 2 * pad - dil * (k - 1) - 1) // stride + 1


def pattern_mask(pid, conn, lib) -> np.ndarray:
    """M[o,c,ky,kx] in {0,1}: tap kept iff the kernel is kept (conn) and the
    tap belongs to the kernel's pattern (Sec. 2)."""
    pid = np.asarray(pid)
    conn = np.asarray(conn)
    lib = np.asarray(lib, dtype=np.int64)
    safe = np.where(conn != 0, pid, 0).astype(np.int64)   # pid is only read where conn = 1
    masks = lib[safe]                                      # [O, C]
    taps = np.arange(9)
    bits = (masks[..., None] >> taps) & 1                  # [O, C, 9]
    m = bits * (conn[..., None] != 0)
    return m.reshape(conn.shape + (3, 3)).astype(np.float64)


def masked_weights(w, pid, conn, lib) -> np.ndarray:
    """Dense fp64 weights with every pruned tap set to zero."""
    return np.asarray(w, dtype=np.float64) * pattern_mask(pid, conn, lib)


def conv2d(x, w, b=None, stride=1, pad=0, dil=1, relu=False) -> np.ndarray:
    """Dense k x k cross-correlation, NCHW, fp64 accumulation.
    x: [N,C,H,W], w: [O,C,KH,KW], b: [O] or None."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, c, h, wd = x.shape
    o, c2, kh, kw = w.shape
    assert c == c2
    ho = out_size(h, kh, stride, pad, dil)
    wo = out_size(wd, kw, stride, pad, dil)
    xp = np.zeros((n, c, h + 2 * pad, wd + 2 * pad), dtype=np.float64)
    xp[:, :, pad:pad + h, pad:pad + wd] = x
    y = np.zeros((o, n, ho, wo), dtype=np.float64)
    for ky in range(kh):
        for kx in range(kw):
            r0, c0 = ky * dil, kx * dil
            xs = xp[:, :, r0:r0 + stride * (ho - 1) + 1:stride, c0:c0 + stride * (wo - 1) + 1:stride]
            y += np.tensordot(w[:, :, ky, kx], xs, axes=([1], [1]))
    y = y.transpose(1, 0, 2, 3)
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :, None, None]
    if relu:
        y = np.maximum(y, 0.0)
    return np.ascontiguousarray(y)


def conv3x3_pruned(x, w, b, pid, conn, lib, stride=1, pad=1, dil=1, relu=False) -> np.ndarray:
    """Pattern/connectivity-pruned 3x3 layer: the masked-dense definition."""
    return conv2d(x, masked_weights(w, pid, conn, lib), b, stride, pad, dil, relu)


def conv3x3_bound(x, w, b, pid, conn, lib, stride=1, pad=1, dil=1) -> np.ndarray:
    """S[n,o,h,w] = |b[o]| + sum |M W| |x| over the same index set as the layer.
    Used to scale the error tolerance of every output."""
    bb = None if b is None else np.abs(np.asarray(b, dtype=np.float64))
    return conv2d(np.abs(np.asarray(x, dtype=np.float64)),
                  np.abs(masked_weights(w, pid, conn, lib)), bb, stride, pad, dil, False)


def conv2d_bound(x, w, b=None, stride=1, pad=0, dil=1) -> np.ndarray:
    bb = None if b is None else np.abs(np.asarray(b, dtype=np.float64))
    return conv2d(np.abs(np.asarray(x, dtype=np.float64)), np.abs(np.asarray(w, dtype=np.float64)),
                  bb, stride, pad, dil, False)


def conv3x3_pruned_naive(x, w, b, pid, conn, lib, stride=1, pad=1, dil=1, relu=False) -> np.ndarray:
    """Nested loops; each output is math.fsum of its exact fp64 terms, so the
    result is the correctly rounded value of the exact sum.  Tiny inputs only."""
    x = np.asarray(x, dtype=np.float64)
    n, c_in, h, wd = x.shape
    c_out = np.asarray(w).shape[0]
    ho, wo = out_size(h, 3, stride, pad, dil), out_size(wd, 3, stride, pad, dil)
    y = np.zeros((n, c_out, ho, wo), dtype=np.float64)
    for nn in range(n):
        for o in range(c_out):
            for yy in range(ho):
                for xx in range(wo):
                    terms = [0.0 if b is None else float(b[o])]
                    for c in range(c_in):
                        if not conn[o][c]:
                            continue
                        mask = int(lib[int(pid[o][c])])
                        for t in range(9):
                            if not (mask >> t) & 1:
                                continue
                            ky, kx = divmod(t, 3)
                            iy = yy * stride + ky * dil - pad
                            ix = xx * stride + kx * dil - pad
                            if 0 <= iy < h and 0 <= ix < wd:
                                terms.append(float(w[o][c][ky][kx]) * float(x[nn, c, iy, ix]))
                    v = math.fsum(terms)
                    y[nn, o, yy, xx] = max(v, 0.0) if relu else v
    return y


def conv_transpose2d(x, w, b=None, stride=2, pad=1, relu=False) -> np.ndarray:
    """Transposed convolution (the adjoint of a strided conv), fp64.
    x: [N,C,H,W], w: [C,O,K,K].  Each input pixel (i,j) of channel c adds
    x * w[c,o,ky,kx] to output pixel (i*s - p + ky, j*s - p + kx)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, c, h, wd = x.shape
    c2, o, kh, kw = w.shape
    assert c == c2
    full_h, full_w = (h - 1) * stride + kh, (wd - 1) * stride + kw
    full = np.zeros((n, o, full_h, full_w), dtype=np.float64)
    for ky in range(kh):
        for kx in range(kw):
            contrib = np.tensordot(x, w[:, :, ky, kx], axes=([1], [0]))   # [N,H,W,O]
            full[:, :, ky:ky + stride * (h - 1) + 1:stride, kx:kx + stride * (wd - 1) + 1:stride] += \
                contrib.transpose(0, 3, 1, 2)
    ho, wo = full_h - 2 * pad, full_w - 2 * pad
    y = full[:, :, pad:pad + ho, pad:pad + wo]
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :, None, None]
    if relu:
        y = np.maximum(y, 0.0)
    return np.ascontiguousarray(y)


def conv_transpose2d_bound(x, w, b=None, stride=2, pad=1) -> np.ndarray:
    bb = None if b is None else np.abs(np.asarray(b, dtype=np.float64))
    return conv_transpose2d(np.abs(np.asarray(x, dtype=np.float64)),
                            np.abs(np.asarray(w, dtype=np.float64)), bb, stride, pad, False)


def maxpool2(x) -> np.ndarray:
    """2x2 max pooling with stride 2; a trailing odd row/column is dropped."""
    x = np.asarray(x)
    n, c, h, w = x.shape
    h2, w2 = h // 2, w // 2
    v = x[:, :, :2 * h2, :2 * w2].reshape(n, c, h2, 2, w2, 2)
    return v.max(axis=(3, 5))


def upsample2(x) -> np.ndarray:
    """Nearest-neighbour upsampling by 2: out[.., y, x] = in[.., y//2, x//2]."""
    return np.repeat(np.repeat(np.asarray(x), 2, axis=2), 2, axis=3)


def pixel_shuffle2(x) -> np.ndarray:
    """PixelShuffle(2): out[n, c, 2h+i, 2w+j] = in[n, 4c + 2i + j, h, w]."""
    x = np.asarray(x)
    n, c4, h, w = x.shape
    c = c4 // 4
    v = x.reshape(n, c, 2, 2, h, w).transpose(0, 1, 4, 2, 5, 3)
    return v.reshape(n, c, 2 * h, 2 * w)
