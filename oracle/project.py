"""Pruning-structure projections and batch-norm folding, the pack-side
helpers of the method (test infrastructure only; see ``oracle/__init__``).

ADMM-based structured pruning (Sec. 2) alternates a training step with a
Euclidean projection of the weights onto the structure set S_i.  Its
projection steps have closed forms, written out here as plain definitions:

* pattern pruning -- each 3x3 kernel keeps the taps of one library pattern:
  the nearest such kernel keeps the pattern with the largest sum of squared
  weights on its taps (ties: the lowest pattern index);
* connectivity pruning -- a layer keeps n kernels: the nearest such layer
  keeps the n kernels with the largest (projected) energy (ties: the lower
  flat index o * c_in + c);
* column pruning -- a layer keeps n columns, a column being one (input
  channel, tap) position across all filters: keep the n with the largest sum
  over filters of squared weights (ties: the lower 9 c + t).

Energies are fp64 sums over taps (or filters) in ascending order, so that
the integer decisions are taken on the same values as the library's.

Batch-norm folding (Sec. 3, the conv + BatchNorm fusion of the graph
rewrite): an inference-mode batch norm after a conv is an affine map per
output channel, s = gamma / sqrt(var + eps): w' = s w, b' = s (b - mean) +
beta, evaluated in fp64 and rounded once to fp32.
"""
from __future__ import annotations

import numpy as np


def _mask_bits(lib) -> np.ndarray:
    """[n_p][9] 0/1 table of the library's tap masks."""
    lib = np.asarray(lib, dtype=np.int64)
    return ((lib[:, None] >> np.arange(9)[None, :]) & 1).astype(np.float64)


def pattern_energy(w, lib) -> np.ndarray:
    """[c_out][c_in][n_p]: sum over the taps of each pattern of w^2 (fp64,
    taps ascending)."""
    w = np.asarray(w, dtype=np.float32).reshape(w.shape[0], w.shape[1], 9).astype(np.float64)
    bits = _mask_bits(lib)
    e = np.zeros(w.shape[:2] + (len(bits),))
    for t in range(9):
        e = e + (w[:, :, t:t + 1] * w[:, :, t:t + 1]) * bits[None, None, :, t]
    return e


def project_patterns(w, lib):
    """(pattern_id u8 [c_out][c_in], kept energy fp64 [c_out][c_in])."""
    e = pattern_energy(w, lib)
    pid = np.argmax(e, axis=2)                       # first maximum: the lowest index
    return pid.astype(np.uint8), np.take_along_axis(e, pid[:, :, None], axis=2)[:, :, 0]


def project_connectivity(energy, n_keep: int) -> np.ndarray:
    """conn u8 [c_out][c_in]: the n_keep kernels of largest energy."""
    energy = np.asarray(energy, dtype=np.float64)
    flat = energy.reshape(-1)
    if not 0 <= n_keep <= flat.size:
        raise ValueError("n_keep out of range")
    order = np.lexsort((np.arange(flat.size), -flat))   # energy descending, then index ascending
    conn = np.zeros(flat.size, dtype=np.uint8)
    conn[order[:n_keep]] = 1
    return conn.reshape(energy.shape)


def column_energy(w) -> np.ndarray:
    """[c_in][9]: sum over filters (ascending) of w^2."""
    w = np.asarray(w, dtype=np.float32).reshape(w.shape[0], w.shape[1], 9).astype(np.float64)
    e = np.zeros(w.shape[1:])
    for o in range(w.shape[0]):
        e = e + w[o] * w[o]
    return e


def project_columns(w, n_keep: int) -> np.ndarray:
    """u16 [c_in]: 9-bit mask of the kept taps of each input channel."""
    e = column_energy(w).reshape(-1)
    if not 0 <= n_keep <= e.size:
        raise ValueError("n_keep out of range")
    order = np.lexsort((np.arange(e.size), -e))
    keep = np.zeros(e.size, dtype=np.int64)
    keep[order[:n_keep]] = 1
    keep = keep.reshape(-1, 9)
    return (keep << np.arange(9)[None, :]).sum(axis=1).astype(np.uint16)


def column_library(col_mask, c_out: int):
    """A column-pruned layer as a pattern library: (lib u16[n_p] = the
    distinct nonzero channel masks ascending, pattern_id u8 [c_out][c_in],
    conn u8 [c_out][c_in]); every filter uses its channel's mask."""
    col_mask = np.asarray(col_mask, dtype=np.uint16)
    lib = np.unique(col_mask[col_mask != 0])
    if len(lib) == 0:
        lib = np.array([1], dtype=np.uint16)
    if len(lib) > 255:
        raise ValueError("more than 255 distinct column masks")
    pid = np.searchsorted(lib, col_mask).clip(0, len(lib) - 1).astype(np.uint8)
    conn = (col_mask != 0).astype(np.uint8)
    return lib.astype(np.uint16), np.broadcast_to(pid, (c_out, len(col_mask))).copy(), \
        np.broadcast_to(conn, (c_out, len(col_mask))).copy()


def fold_bn(w, b, gamma, beta, mean, var, eps: float):
    """(w', b') fp32 of a conv followed by an inference-mode batch norm."""
    w = np.asarray(w, dtype=np.float32)
    c_out = w.shape[0]
    b = np.zeros(c_out, np.float32) if b is None else np.asarray(b, np.float32)
    s = np.asarray(gamma, np.float32).astype(np.float64) / \
        np.sqrt(np.asarray(var, np.float32).astype(np.float64) + np.float64(np.float32(eps)))
    wf = (w.reshape(c_out, -1).astype(np.float64) * s[:, None]).astype(np.float32).reshape(w.shape)
    bf = ((b.astype(np.float64) - np.asarray(mean, np.float32).astype(np.float64)) * s +
          np.asarray(beta, np.float32).astype(np.float64)).astype(np.float32)
    return wf, bf
