"""Pins of the CPU oracle against values fixed by the paper or by mathematics.

None of these compares the oracle with itself: the references are a
hand-computed example, torch's CPU float64 convolution routines (an
independent library implementation), closed forms (stride-2 subsampling,
transposed conv of a single pixel), exact brute force with math.fsum, and
invariants that hold for any correct implementation.
"""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads
from oracle import bf16, conv, net, ppk1
from tests.golden_io import appendix_cases, ppk1_small

CANON8 = np.array(workloads.CANON8, dtype=np.uint16)
X5 = np.arange(1, 26, dtype=np.float64).reshape(1, 1, 5, 5)
W5 = np.arange(1, 10, dtype=np.float32).reshape(1, 1, 3, 3)


def _torch_conv(x, w, b, stride, pad, dil):
    return F.conv2d(torch.from_numpy(np.asarray(x, np.float64)), torch.from_numpy(np.asarray(w, np.float64)),
                    None if b is None else torch.from_numpy(np.asarray(b, np.float64)),
                    stride=stride, padding=pad, dilation=dil).numpy()


def _mask_by_loop(pid, conn, lib):
    o, c = conn.shape
    m = np.zeros((o, c, 3, 3))
    for i in range(o):
        for j in range(c):
            if conn[i, j]:
                for t in range(9):
                    if (int(lib[pid[i, j]]) >> t) & 1:
                        m[i, j, t // 3, t % 3] = 1.0
    return m


# ----------------------------------------------------------------------------
# pin functions (also used by the planted-mistake test at the bottom)
# ----------------------------------------------------------------------------

def pin_appendix(mod=conv):
    for prm, expect in appendix_cases():
        lib = np.array([prm["mask"]], dtype=np.uint16)
        y = mod.conv3x3_pruned(X5, W5, np.array([prm["bias"]], np.float32), np.zeros((1, 1), np.uint8),
                               np.ones((1, 1), np.uint8), lib, prm["stride"], prm["pad"], prm["dil"],
                               bool(prm["relu"]))
        if y.shape[2:] != expect.shape or not np.array_equal(y[0, 0], expect):
            return False
    return True


def pin_torch_masked(mod=conv, seeds=range(6)):
    for seed in seeds:
        rng = np.random.default_rng(seed)
        c_out, c_in = int(rng.integers(1, 7)), int(rng.integers(1, 7))
        stride, dil = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        pad = int(rng.integers(0, 2 * dil + 1))
        h, w = int(rng.integers(5, 12)), int(rng.integers(5, 12))
        L = workloads.random_layer(100 + seed, c_out, c_in, keep=0.6)
        x = workloads.random_input(100 + seed, (2, c_in, h, w))
        y = mod.conv3x3_pruned(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil)
        wm = L["w"].astype(np.float64) * _mask_by_loop(L["pid"], L["conn"], L["lib"])
        ref = _torch_conv(x, wm, L["b"], stride, pad, dil)
        s = conv.conv2d_bound(x, wm, L["b"], stride, pad, dil)
        if y.shape != ref.shape or np.any(np.abs(y - ref) > 1e-12 * s + 1e-300):
            return False
    return True


# ----------------------------------------------------------------------------
# pattern-pruned conv
# ----------------------------------------------------------------------------

def test_appendix_hand_example():
    assert pin_appendix()


def test_appendix_naive_and_packed():
    for prm, expect in appendix_cases():
        lib = np.array([prm["mask"]], dtype=np.uint16)
        args = (X5, W5, np.array([prm["bias"]], np.float32), np.zeros((1, 1), np.uint8),
                np.ones((1, 1), np.uint8), lib)
        kw = dict(stride=prm["stride"], pad=prm["pad"], dil=prm["dil"])
        y = conv.conv3x3_pruned_naive(*args, relu=bool(prm["relu"]), **kw)
        assert np.array_equal(y[0, 0], expect), prm["name"]
        blob = ppk1.pack(W5, args[2], args[3], args[4], lib, **{"stride": prm["stride"], "pad": prm["pad"],
                                                                   "dil": prm["dil"]})
        assert np.array_equal(ppk1.interp(blob, X5, relu=bool(prm["relu"]))[0, 0], expect)


def test_connectivity_pruned_kernel_gives_relu_bias():
    y = conv.conv3x3_pruned(X5, W5, np.array([-2.5], np.float32), np.zeros((1, 1), np.uint8),
                            np.zeros((1, 1), np.uint8), CANON8, relu=True)
    assert np.all(y == 0.0)
    y = conv.conv3x3_pruned(X5, W5, np.array([2.5], np.float32), np.zeros((1, 1), np.uint8),
                            np.zeros((1, 1), np.uint8), CANON8, relu=True)
    assert np.all(y == 2.5)


def test_dense_library_equals_torch_conv2d():
    # the all-ones pattern with no connectivity pruning is a dense conv
    for seed, (stride, pad, dil) in enumerate([(1, 1, 1), (2, 1, 1), (1, 2, 2), (2, 0, 1), (1, 0, 2)]):
        rng = np.random.default_rng(seed)
        c_out, c_in = 5, 3
        w = rng.normal(size=(c_out, c_in, 3, 3)).astype(np.float32)
        b = rng.normal(size=c_out).astype(np.float32)
        x = rng.uniform(-1, 1, size=(2, c_in, 9, 11)).astype(np.float32)
        pid = np.zeros((c_out, c_in), np.uint8)
        conn = np.ones((c_out, c_in), np.uint8)
        y = conv.conv3x3_pruned(x, w, b, pid, conn, np.array([0x1FF], np.uint16), stride, pad, dil)
        ref = _torch_conv(x, w, b, stride, pad, dil)
        s = conv.conv2d_bound(x, w, b, stride, pad, dil)
        assert y.shape == ref.shape
        assert np.all(np.abs(y - ref) <= 1e-12 * s)


def test_masked_layer_equals_torch_conv2d():
    assert pin_torch_masked()


def test_stride2_is_subsampled_stride1():
    L = workloads.random_layer(3, 6, 4)
    x = workloads.random_input(3, (1, 4, 13, 10))
    for dil in (1, 2):
        y1 = conv.conv3x3_pruned(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, dil, dil)
        y2 = conv.conv3x3_pruned(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, dil, dil)
        assert np.array_equal(y2, y1[:, :, ::2, ::2])


def test_naive_fsum_equals_packed_fsum_bitwise():
    rng = np.random.default_rng(11)
    for trial in range(25):
        c_out, c_in = int(rng.integers(1, 10)), int(rng.integers(1, 5))
        stride, dil = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        pad = int(rng.integers(0, 2 * dil + 1))
        h, w = int(rng.integers(3, 7)), int(rng.integers(3, 7))
        if (h + 2 * pad - 2 * dil - 1) < 0 or (w + 2 * pad - 2 * dil - 1) < 0:
            continue
        L = workloads.random_layer(200 + trial, c_out, c_in, keep=float(rng.uniform(0.2, 1.0)))
        x = workloads.random_input(200 + trial, (1, c_in, h, w))
        relu = bool(trial % 2)
        a = conv.conv3x3_pruned_naive(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil, relu)
        blob = ppk1.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil)
        b = ppk1.interp_fsum(blob, x, relu)
        assert np.array_equal(a, b)
        c = conv.conv3x3_pruned(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil, relu)
        s = conv.conv3x3_bound(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil)
        assert np.all(np.abs(a - c) <= 1e-14 * s)


def test_exhaustive_2x2_kernels():
    # every assignment of {8 patterns, pruned} to the four kernels of a 2->2 layer
    rng = np.random.default_rng(5)
    w = rng.normal(size=(2, 2, 3, 3)).astype(np.float32)
    b = rng.normal(size=2).astype(np.float32)
    x = rng.uniform(-1, 1, size=(1, 2, 4, 4)).astype(np.float32)
    for combo in itertools.product(range(9), repeat=4):
        pid = np.array([[c % 8 for c in combo[:2]], [c % 8 for c in combo[2:]]], np.uint8)
        conn = np.array([[c < 8 for c in combo[:2]], [c < 8 for c in combo[2:]]], np.uint8)
        y = conv.conv3x3_pruned(x, w, b, pid, conn, CANON8)
        wm = w.astype(np.float64) * _mask_by_loop(pid, conn, CANON8)
        ref = _torch_conv(x, wm, b, 1, 1, 1)
        assert np.all(np.abs(y - ref) <= 1e-13 * conv.conv2d_bound(x, wm, b, 1, 1, 1))


def test_invariants():
    L = workloads.random_layer(9, 8, 6, keep=0.5)
    x = workloads.random_input(9, (1, 6, 9, 9))
    args = (L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    # zero input -> relu(bias), exactly
    y0 = conv.conv3x3_pruned(np.zeros_like(x), *args, relu=True)
    assert np.array_equal(y0, np.broadcast_to(np.maximum(L["b"], 0).astype(np.float64)[None, :, None, None], y0.shape))
    # perturbing an input channel changes no filter that pruned it
    y = conv.conv3x3_pruned(x, *args)
    x2 = x.copy()
    x2[:, 2] += 7.0
    y2 = conv.conv3x3_pruned(x2, *args)
    for o in range(8):
        if not L["conn"][o, 2]:
            assert np.array_equal(y[:, o], y2[:, o])
        else:
            assert not np.array_equal(y[:, o], y2[:, o])
    # positive homogeneity with power-of-two scale (exact), zero bias
    args0 = (L["w"], None, L["pid"], L["conn"], L["lib"])
    assert np.array_equal(conv.conv3x3_pruned(x * 8.0, *args0), 8.0 * conv.conv3x3_pruned(x, *args0))


# ----------------------------------------------------------------------------
# the tolerance scale S = |b| + sum |M W| |x| (the bound every GPU parity check
# scales by), pinned two ways: exactly on the hand example, where x and W are
# positive so S is the pre-activation output with |b| in place of b; and
# against torch float64 convolutions of |x| and |W M| (M built by loops here)
# plus |b|, for the pruned, dense and transposed bounds.  The planted-mistake
# test below checks that an S over the unmasked weights, or without |b|,
# fails these pins.
# ----------------------------------------------------------------------------

def pin_bound_appendix(mod=conv):
    cases = {prm["name"]: (prm, e) for prm, e in appendix_cases()}
    pre = cases["P0_b0"][1]                           # pattern 0x03A, b = 0: y_pre
    for name, (prm, expect) in cases.items():
        lib = np.array([prm["mask"]], dtype=np.uint16)
        b = np.array([prm["bias"]], np.float32)
        s_ = mod.conv3x3_bound(X5, W5, b, np.zeros((1, 1), np.uint8), np.ones((1, 1), np.uint8), lib,
                               prm["stride"], prm["pad"], prm["dil"])[0, 0]
        if name == "P0_relu":
            want = pre + 150.0                        # b = -150
        elif name == "P0_s2":
            want = pre[::2, ::2] + 150.0
        else:
            want = expect                             # b = 0, no ReLU: S is the output itself
        if s_.shape != want.shape or not np.array_equal(s_, want):
            return False
    return True


def pin_bound_torch(mod=conv, seeds=range(4)):
    for seed in seeds:
        rng = np.random.default_rng(300 + seed)
        c_out, c_in = int(rng.integers(2, 7)), int(rng.integers(2, 7))
        stride, dil = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        pad = int(rng.integers(0, 2 * dil + 1))
        h, w = int(rng.integers(5, 12)), int(rng.integers(5, 12))
        L = workloads.random_layer(300 + seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(300 + seed, (2, c_in, h, w))
        wm = np.abs(L["w"].astype(np.float64) * _mask_by_loop(L["pid"], L["conn"], L["lib"]))
        ref = _torch_conv(np.abs(x), wm, np.abs(L["b"]), stride, pad, dil)
        s_ = mod.conv3x3_bound(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil)
        if s_.shape != ref.shape or np.any(np.abs(s_ - ref) > 1e-12 * ref):
            return False
        # dense k x k and transposed bounds (mixed-sign weights and biases)
        wd = rng.normal(size=(c_out, c_in, 3, 3))
        bd = rng.normal(size=c_out)
        ref = _torch_conv(np.abs(x), np.abs(wd), np.abs(bd), 1, 1, 1)
        if np.any(np.abs(mod.conv2d_bound(x, wd, bd, 1, 1, 1) - ref) > 1e-12 * ref):
            return False
        wt = rng.normal(size=(c_in, c_out, 4, 4))
        ref = F.conv_transpose2d(torch.from_numpy(np.abs(x).astype(np.float64)), torch.from_numpy(np.abs(wt)),
                                 torch.from_numpy(np.abs(bd)), stride=2, padding=1).numpy()
        if np.any(np.abs(mod.conv_transpose2d_bound(x, wt, bd, 2, 1) - ref) > 1e-12 * ref):
            return False
    return True


def test_bound_exact_on_hand_example():
    assert pin_bound_appendix()


def test_bound_equals_abs_conv_torch():
    assert pin_bound_torch()


class _BoundMutant:
    """The oracle's conv module with a planted mistake in the tolerance scale."""

    def __init__(self, kind):
        self.kind = kind

    def conv3x3_bound(self, x, w, b, pid, conn, lib, stride=1, pad=1, dil=1):
        if self.kind == "unmasked":                 # S over the dense |W|
            return conv.conv2d_bound(x, w, b, stride, pad, dil)
        if self.kind == "no_bias":                  # S without |b|
            return conv.conv3x3_bound(x, w, None, pid, conn, lib, stride, pad, dil)
        return conv.conv3x3_bound(x, w, b, pid, conn, lib, stride, pad, dil)

    def conv2d_bound(self, x, w, b=None, stride=1, pad=0, dil=1):
        return conv.conv2d_bound(x, w, None if self.kind == "no_bias" else b, stride, pad, dil)

    def conv_transpose2d_bound(self, x, w, b=None, stride=2, pad=1):
        return conv.conv_transpose2d_bound(x, w, None if self.kind == "no_bias" else b, stride, pad)


@pytest.mark.parametrize("kind", ["unmasked", "no_bias"])
def test_planted_bound_mistake_is_caught(kind):
    mut = _BoundMutant(kind)
    assert not pin_bound_appendix(mut)
    assert not pin_bound_torch(mut)


def test_bound_dominates_result():
    L = workloads.random_layer(12, 6, 5)
    x = workloads.random_input(12, (2, 5, 8, 8))
    y = conv.conv3x3_pruned(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    s = conv.conv3x3_bound(x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    assert np.all(np.abs(y) <= s * (1 + 1e-15))


# ----------------------------------------------------------------------------
# dense ops of the networks
# ----------------------------------------------------------------------------

def test_dense_kxk_conv_vs_torch():
    rng = np.random.default_rng(1)
    for k, pad in ((9, 4), (1, 0), (3, 1)):
        x = rng.uniform(0, 1, size=(2, 3, 12, 10))
        w = rng.normal(size=(4, 3, k, k))
        b = rng.normal(size=4)
        y = conv.conv2d(x, w, b, 1, pad, 1)
        ref = _torch_conv(x, w, b, 1, pad, 1)
        assert np.all(np.abs(y - ref) <= 1e-12 * conv.conv2d_bound(x, w, b, 1, pad, 1))


def test_conv_transpose_single_pixel_closed_form():
    # one input pixel of value 1: the output is the kernel cropped by the padding
    w = np.arange(16, dtype=np.float64).reshape(1, 1, 4, 4)
    y = conv.conv_transpose2d(np.ones((1, 1, 1, 1)), w, None, stride=2, pad=1)
    assert np.array_equal(y[0, 0], w[0, 0, 1:3, 1:3])


def test_conv_transpose_vs_torch():
    rng = np.random.default_rng(2)
    x = rng.uniform(0, 1, size=(2, 5, 6, 7))
    w = rng.normal(size=(5, 3, 4, 4))
    b = rng.normal(size=3)
    y = conv.conv_transpose2d(x, w, b, 2, 1, relu=False)
    ref = F.conv_transpose2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b), stride=2,
                             padding=1).numpy()
    assert y.shape == ref.shape == (2, 3, 12, 14)
    assert np.all(np.abs(y - ref) <= 1e-12 * conv.conv_transpose2d_bound(x, w, b, 2, 1))


def test_pool_upsample_shuffle_hand_examples():
    x = np.array([[1, 5, 2, 0, 9], [3, 4, 8, 7, 9], [0, 0, 1, 1, 9]], dtype=np.float64).reshape(1, 1, 3, 5)
    assert np.array_equal(conv.maxpool2(x)[0, 0], [[5, 8]])
    u = conv.upsample2(np.array([[1.0, 2.0], [3.0, 4.0]]).reshape(1, 1, 2, 2))[0, 0]
    assert np.array_equal(u, [[1, 1, 2, 2], [1, 1, 2, 2], [3, 3, 4, 4], [3, 3, 4, 4]])
    p = conv.pixel_shuffle2(np.array([1.0, 2.0, 3.0, 4.0]).reshape(1, 4, 1, 1))[0, 0]
    assert np.array_equal(p, [[1, 2], [3, 4]])


def test_pool_upsample_shuffle_vs_torch():
    rng = np.random.default_rng(4)
    x = rng.normal(size=(2, 8, 7, 9))
    t = torch.from_numpy(x)
    assert np.array_equal(conv.maxpool2(x), F.max_pool2d(t, 2).numpy())
    assert np.array_equal(conv.upsample2(x), F.interpolate(t, scale_factor=2, mode="nearest").numpy())
    assert np.array_equal(conv.pixel_shuffle2(x), F.pixel_shuffle(t, 2).numpy())


# ----------------------------------------------------------------------------
# bf16 rounding
# ----------------------------------------------------------------------------

def test_bf16_hand_values():
    one_ulp = 2.0 ** -7          # bf16 spacing at 1.0
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -(1.0 + 3 * 2 ** -8)],
                    dtype=np.float32)
    got = bf16.round_f32(vals)
    assert list(got) == [1.0, 1.0, 1.0 + 2 * one_ulp, 1.0 + one_ulp, -(1.0 + 2 * one_ulp)]
    assert int(bf16.round_bits(np.float32(1.0)).reshape(-1)[0]) == 0x3F80


def test_bf16_matches_torch():
    rng = np.random.default_rng(8)
    v = rng.normal(size=20000).astype(np.float32)
    bits = v.view(np.uint32)
    v2 = ((bits & np.uint32(0xFFFF0000)) | np.uint32(0x8000)).view(np.float32)   # exact ties
    for a in (v, v2):
        ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
        assert np.array_equal(bf16.round_f32(a), ref)


def test_store_bf16_single_rounding():
    # fp64 value just above a bf16 midpoint whose fp32 rounding lands on the midpoint
    y = np.array([1.0 + 2 ** -8 + 2 ** -40, 1.0 + 2 ** -8 - 2 ** -40, 1.0 + 2 ** -8])
    assert list(net.store(y, "bf16")) == [1.0 + 2 ** -7, 1.0, 1.0]


# ----------------------------------------------------------------------------
# packed format
# ----------------------------------------------------------------------------

def _small_layer():
    w = np.zeros((4, 3, 9), np.float32)
    for o in range(4):
        for c in range(3):
            for t in range(9):
                w[o, c, t] = 100 * o + 10 * c + t
    pid = np.array([[0, 4, 4], [2, 2, 7], [1, 0, 3], [4, 4, 0]], np.uint8)
    conn = np.array([[1, 0, 1], [1, 1, 1], [0, 0, 0], [1, 1, 0]], np.uint8)
    bias = np.array([0.5, 1.5, 2.5, 3.5], np.float32)
    return w.reshape(4, 3, 3, 3), bias, pid, conn


def test_pack_golden_small():
    g = ppk1_small()
    w, b, pid, conn = _small_layer()
    d = ppk1.parse(ppk1.pack(w, b, pid, conn, CANON8))
    assert list(d["perm"]) == g["perm"]
    assert list(d["codes"].ravel()) == g["codes"]
    assert list(d["woff"]) == g["woff"]
    assert list(d["kept_mask"]) == g["kept_mask"]
    assert list(d["w"]) == g["w"]
    assert list(d["bias"]) == g["bias"]
    assert d["n_kept"] == g["n_kept"][0] and d["n_wt"] == g["n_wt"][0]
    o = d["offsets"]
    assert [o["masks"], o["perm"], o["codes"], o["woff"], o["w"], o["bias"]] == g["offsets"]
    assert d["total_bytes"] == g["total_bytes"][0]


def test_pack_roundtrip_and_structure():
    for seed, (c_out, c_in, wd) in enumerate([(13, 7, 0), (16, 16, 1), (1, 1, 0), (9, 3, 1), (24, 5, 0)]):
        L = workloads.random_layer(300 + seed, c_out, c_in, keep=0.4)
        blob = ppk1.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], wdtype=wd)
        assert len(blob) % 64 == 0
        d = ppk1.parse(blob)
        assert d["n_kept"] == int(L["conn"].sum())
        assert d["n_wt"] == 4 * d["n_kept"]
        wr = bf16.round_f32(L["w"]) if wd else L["w"]
        wm, bm = ppk1.unpack_dense(blob)
        assert np.array_equal(wm, wr.astype(np.float64) * _mask_by_loop(L["pid"], L["conn"], L["lib"]))
        assert np.array_equal(bm, L["b"].astype(np.float64))
        perm = [int(p) for p in d["perm"] if p != ppk1.NO_FILTER]
        assert sorted(perm) == list(range(c_out))
        kept = L["conn"].sum(axis=1)
        assert all(kept[perm[i]] >= kept[perm[i + 1]] for i in range(c_out - 1))
        assert np.all(np.diff(d["woff"].astype(np.int64)) >= 0)
        for g in range(d["n_groups"]):
            for c in range(c_in):
                m = [s for s in range(8) if d["codes"][g, c, s] != ppk1.PRUNED]
                assert d["kept_mask"][g * c_in + c] == sum(1 << s for s in m)


def test_pack_bf16_odd_tap_padding():
    # a 9-tap (dense) kernel in bf16 is padded to an even element count
    w = np.arange(2 * 2 * 9, dtype=np.float32).reshape(2, 2, 3, 3)
    blob = ppk1.pack(w, None, np.zeros((2, 2), np.uint8), np.ones((2, 2), np.uint8),
                     np.array([0x1FF], np.uint16), wdtype=ppk1.WD_BF16)
    d = ppk1.parse(blob)
    assert d["n_wt"] == 4 * 10
    assert list(d["woff"]) == [0, 20, 40]
    raw = np.frombuffer(blob, "<u2", d["n_wt"], d["offsets"]["w"])
    assert raw[9] == 0 and raw[19] == 0


@pytest.mark.parametrize("bad", ["npat0", "npat256", "mask0", "mask512", "pid", "conn2", "stride0"])
def test_pack_rejects_invalid(bad):
    w, b, pid, conn = _small_layer()
    lib = CANON8.copy()
    kw = {}
    if bad == "npat0":
        lib = np.zeros(0, np.uint16)
    elif bad == "npat256":
        lib = np.full(256, 0x10, np.uint16)
    elif bad == "mask0":
        lib[3] = 0
    elif bad == "mask512":
        lib[3] = 0x200
    elif bad == "pid":
        pid = pid.copy()
        pid[1, 1] = 8
    elif bad == "conn2":
        conn = conn.copy()
        conn[0, 0] = 2
    elif bad == "stride0":
        kw["stride"] = 0
    with pytest.raises(ValueError):
        ppk1.pack(w, b, pid, conn, lib, **kw)


def test_pack_ignores_pattern_id_of_pruned_kernels():
    w, b, pid, conn = _small_layer()
    pid2 = pid.copy()
    pid2[2, :] = 200        # filter 2 is fully pruned; its ids are never read
    assert ppk1.pack(w, b, pid, conn, CANON8) == ppk1.pack(w, b, pid2, conn, CANON8)


# ----------------------------------------------------------------------------
# network runner
# ----------------------------------------------------------------------------

def _torch_op(op, prm, t, t2):
    if op["op"] == "conv3":
        wm = prm["w"].astype(np.float64) * _mask_by_loop(prm["pid"], prm["conn"], prm["lib"])
        y = F.conv2d(t, torch.from_numpy(wm), torch.from_numpy(prm["b"].astype(np.float64)),
                     stride=op["stride"], padding=op["pad"], dilation=op["dil"])
    elif op["op"] == "conv":
        y = F.conv2d(t, torch.from_numpy(prm["w"].astype(np.float64)),
                     torch.from_numpy(prm["b"].astype(np.float64)), padding=op["pad"])
    elif op["op"] == "deconv":
        y = F.conv_transpose2d(t, torch.from_numpy(prm["w"].astype(np.float64)),
                               torch.from_numpy(prm["b"].astype(np.float64)), stride=2, padding=1)
    elif op["op"] == "maxpool2":
        return F.max_pool2d(t, 2)
    elif op["op"] == "up2":
        return F.interpolate(t, scale_factor=2, mode="nearest")
    elif op["op"] == "pshuf2":
        return F.pixel_shuffle(t, 2)
    elif op["op"] == "add":
        return t + t2
    return torch.relu(y) if op.get("relu") else y


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_net_runner_matches_torch_on_shrunk_networks(cfg):
    # the config's op list with every channel count divided down and a tiny input
    spec = workloads.net_spec(cfg)
    div = 16 if cfg != 1 else 4
    ops = []
    for op in spec["ops"]:
        op = dict(op)
        for key in ("c_in", "c_out"):
            if key in op and op[key] > 4:
                op[key] = max(2, op[key] // div)
        ops.append(op)
    # keep channel counts consistent after shrinking (pixel shuffle needs 4x)
    for i, op in enumerate(ops):
        if op["op"] == "pshuf2":
            ops[i - 1]["c_out"] = 4 * ops[i + 1]["c_in"]
    spec = dict(spec, ops=ops, batch=min(spec["batch"], 2), c=ops[0]["c_in"], h=32 if cfg == 2 else 16,
                w=32 if cfg == 2 else (12 if cfg == 4 else 16))
    params = []
    for i, op in enumerate(ops):
        p = workloads.layer_params(cfg, i, op)
        params.append(p)
    x = workloads.random_input(cfg, (spec["batch"], spec["c"], spec["h"], spec["w"]), 0, 1)
    y = net.run_net(spec, params, x, "f32")
    slots = {0: torch.from_numpy(x.astype(np.float64))}
    for op, prm in zip(ops, params):
        slots[op["dst"]] = _torch_op(op, prm, slots[op["src"]], slots.get(op.get("src2")))
    ref = slots[1].numpy()
    assert y.shape == ref.shape
    # the oracle rounds activations to fp32 between layers; torch stays in fp64
    assert np.allclose(y, ref, rtol=1e-4, atol=1e-5 * np.abs(ref).max())


def test_workload_keep_counts():
    for cfg in (2, 3, 4, 5):
        spec = workloads.net_spec(cfg)
        for i, op in enumerate(spec["ops"]):
            if op["op"] == "conv3" and op["lib"] == "canon8":
                p = workloads.layer_params(cfg, i, op)
                assert int(p["conn"].sum()) == int(round(op["keep"] * op["c_in"] * op["c_out"]))
                assert p["pid"].max() < 8


# ----------------------------------------------------------------------------
# planted mistakes: each plausible bug in the oracle must fail a pin
# ----------------------------------------------------------------------------

class _Mutant:
    """The oracle's conv module with one planted mistake."""

    def __init__(self, kind):
        self.kind = kind

    def conv3x3_pruned(self, x, w, b, pid, conn, lib, stride=1, pad=1, dil=1, relu=False):
        w = np.asarray(w, np.float64)
        m = conv.pattern_mask(pid, conn, lib)
        if self.kind == "transpose_kernel":
            w = w.transpose(0, 1, 3, 2)
        elif self.kind == "flip_kernel":          # convolution instead of correlation
            w = w[:, :, ::-1, ::-1]
        elif self.kind == "tap_order":
            m = m.reshape(m.shape[:2] + (9,))[..., ::-1].reshape(m.shape)
        elif self.kind == "drop_bias":
            b = None
        elif self.kind == "pad_off_by_one":
            pad = pad + 1
        elif self.kind == "swap_oc":
            w = w.transpose(1, 0, 2, 3) if w.shape[0] == w.shape[1] else w[:, ::-1]
        elif self.kind == "ignore_conn":
            m = conv.pattern_mask(pid, np.ones_like(conn), lib)
        return conv.conv2d(x, w * m, b, stride, pad, dil, relu)


@pytest.mark.parametrize("kind", ["transpose_kernel", "flip_kernel", "tap_order", "drop_bias", "pad_off_by_one",
                                  "swap_oc", "ignore_conn"])
def test_planted_mistake_is_caught(kind):
    mut = _Mutant(kind)
    assert not (pin_appendix(mut) and pin_torch_masked(mut))
