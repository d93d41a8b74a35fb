"""Error bars for comparing the GPU path with the oracle.

For an output y with exact (oracle, fp64) value y_ref and magnitude sum
S = |b| + sum |w||x| over its terms, the fp32 path must satisfy
|y - y_ref| <= 1e-4 * S and the bf16 path |y - y_ref| <= 2e-2 * S.
Why 1e-4 holds for fp32: any order of n fp32 additions of exact products
has error <= gamma_n * S with gamma_n ~ n * 2^-24; the longest sum on the
pruned path (512 channels x 1/3 kept x 4 taps ~ 683 terms) gives 4.1e-5.
bf16 adds the rounding of the inputs (already in the oracle's inputs) and of
the output (2^-9 relative).  When S = 0 the output must be exact.
"""
import numpy as np

TOL = {"f32": 1e-4, "bf16": 2e-2}


def check(y, y_ref, bound, dtype="f32", what=""):
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    bound = np.asarray(bound, dtype=np.float64)
    assert y.shape == y_ref.shape == bound.shape, (what, y.shape, y_ref.shape, bound.shape)
    err = np.abs(y - y_ref)
    lim = TOL[dtype] * bound
    bad = err > lim
    if np.any(bad):
        i = np.unravel_index(np.argmax(np.where(bad, err / np.maximum(lim, 1e-300), 0)), y.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {y.size} outputs out of tolerance; worst at {i}: "
                             f"y={y[i]!r} ref={y_ref[i]!r} S={bound[i]!r}")
    return float(np.max(err / np.maximum(bound, 1e-300))) if y.size else 0.0


def relu_ref(y, relu):
    return np.maximum(y, 0.0) if relu else y
