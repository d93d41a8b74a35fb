"""C-ABI checks that need no GPU: the library loads, exports every function
include/pp.h declares, validates blobs, and rejects bad calls on the host
before any device work is enqueued."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads

pp = pytest.importorskip("paper_2004_11250_amd")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return pp.load_library()


def _declared():
    src = open(os.path.join(ROOT, "include", "pp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pp_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(pp.SYMBOLS)
    for name in names:
        assert hasattr(lib, name), name


def test_host_only_library_exports_packer():
    from paper_2004_11250_amd import build
    path = build.build_host()
    h = ctypes.CDLL(path)
    for name in ("pp_pack", "pp_blob_info", "pp_status_str", "pp_last_error", "pp_project_patterns",
                 "pp_project_connectivity", "pp_project_columns", "pp_column_library", "pp_fold_bn"):
        assert hasattr(h, name)


def test_status_strings(lib):
    for s in (0, -1, -2, -3, -4, -5):
        assert lib.pp_status_str(s)
    assert lib.pp_status_str(-99) == b"unknown status"


def _blob(c_out=12, c_in=5, stride=1, pad=1, dil=1, wd=0):
    L = workloads.random_layer(5, c_out, c_in)
    return pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil, wd)


def _info_status(lib, blob, n=None):
    b = np.ascontiguousarray(blob, np.uint8)
    return lib.pp_blob_info(b.ctypes.data, b.nbytes if n is None else n, None, None, None)


def test_blob_info_rejects_corruption(lib):
    blob = _blob()
    assert _info_status(lib, blob) == pp.PP_OK
    assert lib.pp_blob_info(None, 100, None, None, None) == pp.PP_EINVAL
    assert _info_status(lib, blob, 64) == pp.PP_EBLOB                 # truncated
    assert _info_status(lib, blob, len(blob) - 64) == pp.PP_EBLOB     # size != total_bytes
    hdr = blob.view(np.uint32)
    for word, val in ((0, 0x12345678), (1, 7), (2, 0), (7, 0), (8, 4), (9, 99), (13, 3), (16, 1 << 30),
                      (19, 1)):
        bad = blob.copy()
        bad.view(np.uint32)[word] = val
        assert _info_status(lib, bad) == pp.PP_EBLOB, word
    d = pp.blob_info(blob)
    off_codes, off_woff, off_perm = hdr[14], hdr[15], hdr[13]
    bad = blob.copy()
    bad[off_codes] = 200                      # pattern id beyond the library
    assert _info_status(lib, bad) == pp.PP_EBLOB
    bad = blob.copy()
    bad.view(np.uint32)[off_woff // 4 + 1] += 4   # woff out of step with codes
    assert _info_status(lib, bad) == pp.PP_EBLOB
    bad = blob.copy()
    bad.view(np.uint32)[off_perm // 4 + 1] = bad.view(np.uint32)[off_perm // 4]   # perm not a permutation
    assert _info_status(lib, bad) == pp.PP_EBLOB
    assert d["c_out"] == 12


def test_pack_rejects_bad_arguments(lib):
    L = workloads.random_layer(6, 4, 3)
    masks = np.array(workloads.CANON8, np.uint16)
    n = ctypes.c_size_t(0)
    ok = pp.LayerDesc(4, 3, 1, 1, 1, 0)
    base = [L["w"].ctypes.data, None, L["pid"].ctypes.data, L["conn"].ctypes.data, masks.ctypes.data, 8]
    assert lib.pp_pack(ctypes.byref(ok), *base, None, ctypes.byref(n)) == pp.PP_OK
    for desc in (pp.LayerDesc(0, 3, 1, 1, 1, 0), pp.LayerDesc(4, 3, 0, 1, 1, 0), pp.LayerDesc(4, 3, 1, -1, 1, 0),
                 pp.LayerDesc(4, 3, 1, 1, 1, 2)):
        assert lib.pp_pack(ctypes.byref(desc), *base, None, ctypes.byref(n)) == pp.PP_EINVAL
    assert lib.pp_pack(ctypes.byref(ok), None, *base[1:], None, ctypes.byref(n)) == pp.PP_EINVAL
    for n_p in (0, 256):
        args = base[:5] + [n_p]
        assert lib.pp_pack(ctypes.byref(ok), *args, None, ctypes.byref(n)) == pp.PP_EINVAL
    conn = L["conn"].copy()
    conn[0, 0] = 3
    args = base[:3] + [conn.ctypes.data] + base[4:]
    assert lib.pp_pack(ctypes.byref(ok), *args, None, ctypes.byref(n)) == pp.PP_EINVAL
    assert b"conn" in lib.pp_last_error()


def _conv(lib, blob, x=0x100000, y=0x200000, n=1, h=16, w=16, dt=0, flags=0, dblob=0x300000):
    b = np.ascontiguousarray(blob, np.uint8)
    return lib.pp_conv2d_fwd(b.ctypes.data, b.nbytes, dblob, x, y, n, h, w, dt, flags, None, 0, None)


def test_conv_validation_happens_before_any_launch(lib):
    # every call below fails on the host; the fake device addresses are never touched
    blob = _blob()
    assert _conv(lib, blob, x=0) == pp.PP_EINVAL
    assert _conv(lib, blob, dblob=0) == pp.PP_EINVAL
    assert _conv(lib, blob, dblob=0x300010) == pp.PP_EINVAL           # blob not 256-byte aligned
    assert _conv(lib, blob, n=0) == pp.PP_EINVAL
    assert _conv(lib, blob, dt=1) == pp.PP_EUNSUPPORTED               # weight dtype != activation dtype
    assert _conv(lib, blob, dt=5) == pp.PP_EINVAL
    assert _conv(lib, blob, flags=32) == pp.PP_EINVAL                  # unknown flag
    for f in (pp.PP_MAXPOOL2 | pp.PP_ACCUMULATE, pp.PP_ACCUMULATE | pp.PP_PIXSHUF2, 14):
        assert _conv(lib, blob, flags=f) == pp.PP_EINVAL               # more than one fused op
    assert _conv(lib, _blob(c_out=10), flags=pp.PP_PIXSHUF2) == pp.PP_EINVAL   # c_out % 4 != 0
    assert _conv(lib, blob, x=0x100000, y=0x100000 + 64) == pp.PP_EINVAL   # overlapping x / y
    assert _conv(lib, _blob(stride=3)) == pp.PP_EUNSUPPORTED
    assert _conv(lib, _blob(dil=3, pad=3)) == pp.PP_EUNSUPPORTED
    assert _conv(lib, _blob(pad=3)) == pp.PP_EUNSUPPORTED
    bad = blob.copy()
    bad[:4] = 0
    assert _conv(lib, bad) == pp.PP_EBLOB
    assert _conv(lib, _blob(pad=0, dil=2), h=4, w=4) == pp.PP_EUNSUPPORTED   # smaller than the dilated kernel


def test_out_size(lib):
    for (s, p, d, h, w) in ((1, 1, 1, 32, 32), (2, 1, 1, 33, 20), (1, 2, 2, 10, 7), (2, 0, 1, 9, 9)):
        ho, wo = pp.out_size(_blob(stride=s, pad=p, dil=d), h, w)
        assert ho == (h + 2 * p - 2 * d - 1) // s + 1 and wo == (w + 2 * p - 2 * d - 1) // s + 1


def _net_for(cfg, shrink=True):
    spec = workloads.net_spec(cfg)
    params = [workloads.layer_params(cfg, i, op) for i, op in enumerate(spec["ops"])]
    return spec, params


class _HostNet:
    """Op array with host blobs and fake device addresses (never launched)."""

    def __init__(self, spec, params, dtype=0):
        self.keep = []
        self.arr = (pp.NetOp * len(spec["ops"]))()
        for i, (op, prm) in enumerate(zip(spec["ops"], params)):
            e = self.arr[i]
            e.kind = pp.Net._KIND[op["op"]]
            e.src, e.dst, e.src2 = op["src"], op["dst"], op.get("src2", 0)
            e.flags = 1 if op.get("relu") else 0
            if op["op"] == "conv3":
                blob = pp.pack(prm["w"], prm["b"], prm["pid"], prm["conn"], prm["lib"], op["stride"], op["pad"],
                               op["dil"], dtype)
                self.keep.append(blob)
                e.h_blob, e.blob_bytes, e.d_blob = blob.ctypes.data, blob.nbytes, 0x4000000
            elif op["op"] in ("conv", "deconv"):
                e.k, e.stride, e.pad, e.dilation = op["k"], op["stride"], op["pad"], 1
                e.c_in, e.c_out, e.d_w = op["c_in"], op["c_out"], 0x5000000


@pytest.mark.parametrize("cfg,out_shape", [(1, (16, 32, 32)), (2, (512, 7, 7)), (3, (3, 512, 512)),
                                           (4, (3, 1080, 1920)), (5, (313, 64, 64))])
def test_net_workspace_shapes(lib, cfg, out_shape):
    spec, params = _net_for(cfg)
    hn = _HostNet(spec, params)
    nb = ctypes.c_size_t(0)
    oc, oh, ow = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    st = lib.pp_net_workspace(hn.arr, len(spec["ops"]), spec["batch"], spec["c"], spec["h"], spec["w"], 0,
                              ctypes.byref(nb), ctypes.byref(oc), ctypes.byref(oh), ctypes.byref(ow))
    assert st == pp.PP_OK, lib.pp_last_error()
    assert (oc.value, oh.value, ow.value) == out_shape
    # workspace too small -> PP_ESIZE, before anything is launched
    if nb.value:
        st = lib.pp_net_fwd(hn.arr, len(spec["ops"]), 0x100000, 0x200000, spec["batch"], spec["c"], spec["h"],
                            spec["w"], 0, 0x300000, nb.value - 1, None)
        assert st == pp.PP_ESIZE


def test_net_rejects_bad_op_lists(lib):
    spec, params = _net_for(2)
    hn = _HostNet(spec, params)
    nb = ctypes.c_size_t(0)

    def status(n_ops=len(spec["ops"]), c=3, h=224, w=224):
        return lib.pp_net_workspace(hn.arr, n_ops, 1, c, h, w, 0, ctypes.byref(nb), None, None, None)

    assert status() == pp.PP_OK
    assert status(c=4) == pp.PP_EINVAL                 # channel mismatch with the first blob
    assert status(n_ops=0) == pp.PP_EINVAL
    assert status(h=16, w=16) == pp.PP_EINVAL           # pooled below 2x2
    hn.arr[1].src = 9                                   # reads a slot nobody wrote
    assert status() == pp.PP_EINVAL
    hn.arr[1].src = 2
    hn.arr[1].dst = 2                                   # dst == src
    assert status() == pp.PP_EINVAL
    hn.arr[1].dst = 3
    hn.arr[0].kind = 42
    assert status() == pp.PP_EINVAL


def test_round_bf16_matches_the_oracle_rounding(lib):
    from oracle import bf16 as obf16
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(4096).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 4096),
                        np.array([0.0, -0.0, 1e-40, -1e-40], np.float32)]).astype(np.float32)
    assert np.array_equal(pp.round_bf16(x), obf16.round_bits(x))
    # ties to even, carry into the exponent, overflow to infinity, infinities
    u = np.array([0x3F808000, 0x3F818000, 0x3F80FFFF, 0x3FFF8000, 0x7F7FFFFF, 0x7F800000, 0xFF800000],
                 np.uint32)
    want = np.array([0x3F80, 0x3F82, 0x3F81, 0x4000, 0x7F80, 0x7F80, 0xFF80], np.uint16)
    assert np.array_equal(pp.round_bf16(u.view(np.float32)), want)
    # a NaN stays a NaN, also one whose payload sits in the dropped bits
    nan = np.array([0x7FC00000, 0x7F800001, 0xFFFFFFFF], np.uint32).view(np.float32)
    r = pp.round_bf16(nan)
    assert np.all((r & 0x7F80) == 0x7F80) and np.all(r & 0x007F)
    assert lib.pp_round_bf16(None, None, 1) == pp.PP_EINVAL
    assert lib.pp_round_bf16(None, None, 0) == pp.PP_OK


def test_prepare_host_checks(lib):
    # host-side outcomes of pp_conv2d_prepare: the size query, a layer the
    # matrix-core form cannot run, a short buffer, NULL and misaligned
    # pointers -- all before any device work
    L = workloads.random_layer(31, 40, 64, keep=0.5)
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    nb = ctypes.c_size_t(0)
    assert lib.pp_conv2d_prepare(blob.ctypes.data, blob.nbytes, None, None, ctypes.byref(nb), None) == pp.PP_OK
    # bf16, canonical library, stride 1: the matrix-core part (bf16 weights,
    # then the bias), then from the next 256-byte boundary the lean part
    mfma = -(-40 * 9 * 64 * 2 // 256) * 256 + 40 * 4
    assert nb.value == -(-mfma // 256) * 256 + 5 * 64 * 32 * 4
    small = ctypes.c_size_t(nb.value - 1)
    assert lib.pp_conv2d_prepare(blob.ctypes.data, blob.nbytes, 0x100000, 0x200000, ctypes.byref(small),
                                 None) == pp.PP_ESIZE
    assert small.value == nb.value
    assert lib.pp_conv2d_prepare(blob.ctypes.data, blob.nbytes, 0x100000, 0x200010, ctypes.byref(nb),
                                 None) == pp.PP_EINVAL
    assert lib.pp_conv2d_prepare(blob.ctypes.data, blob.nbytes, None, None, None, None) == pp.PP_EINVAL
    L2 = workloads.random_layer(32, 40, 48, keep=0.5)   # c_in not a multiple of 32: the lean part only
    blob2 = pp.pack(L2["w"], L2["b"], L2["pid"], L2["conn"], L2["lib"], 1, 1, 1, pp.PP_BF16)
    assert lib.pp_conv2d_prepare(blob2.ctypes.data, blob2.nbytes, None, None, ctypes.byref(nb),
                                 None) == pp.PP_OK
    assert nb.value == 5 * 48 * 32 * 4
    # the matrix-core part only (stride 2)
    b2s = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 1, 1, pp.PP_BF16)
    assert lib.pp_conv2d_prepare(b2s.ctypes.data, b2s.nbytes, None, None, ctypes.byref(nb), None) == pp.PP_OK
    assert nb.value == mfma
    # neither part: c_in 48 at stride 2
    blob3 = pp.pack(L2["w"], L2["b"], L2["pid"], L2["conn"], L2["lib"], 2, 1, 1, pp.PP_BF16)
    assert lib.pp_conv2d_prepare(blob3.ctypes.data, blob3.nbytes, None, None, ctypes.byref(nb),
                                 None) == pp.PP_EUNSUPPORTED
    # fp32: the lean kernel's expanded weights, [ceil(c_out / 8)][c_in][32]
    # floats, for the canonical library (pad = dilation; stride and dilation
    # not both 2)
    b32 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    assert lib.pp_conv2d_prepare(b32.ctypes.data, b32.nbytes, None, None, ctypes.byref(nb), None) == pp.PP_OK
    assert nb.value == 5 * 64 * 32 * 4
    s2 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 1, 1, pp.PP_F32)     # stride 2: the lean part
    assert lib.pp_conv2d_prepare(s2.ctypes.data, s2.nbytes, None, None, ctypes.byref(nb), None) == pp.PP_OK
    assert nb.value == 5 * 64 * 32 * 4
    s2d2 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 2, 2, pp.PP_F32)   # stride and dilation 2
    assert lib.pp_conv2d_prepare(s2d2.ctypes.data, s2d2.nbytes, None, None, ctypes.byref(nb),
                                 None) == pp.PP_EUNSUPPORTED
    d9 = pp.pack(L["w"], L["b"], np.zeros_like(L["pid"]), L["conn"], np.array(workloads.DENSE9, np.uint16),
                 1, 1, 1, pp.PP_F32)
    assert lib.pp_conv2d_prepare(d9.ctypes.data, d9.nbytes, None, None, ctypes.byref(nb), None) == pp.PP_EUNSUPPORTED
    # the allocation-free call has no prepared buffer to read
    assert lib.pp_conv2d_fwd_noalloc(blob.ctypes.data, blob.nbytes, 0x100000, 0x200000, 0x300000, 1, 8, 8,
                                     pp.PP_BF16, pp.PP_PREPARED, None) == pp.PP_EINVAL
