"""Pattern/connectivity-pruned 3x3 convolution on AMD Instinct MI355X.

Thin ctypes binding over ``libppconv.so`` (C ABI declared in
``include/pp.h``).  Every step of the computation runs in the library's HIP
kernels; this module only marshals arguments.  PyTorch provides device memory
and the current HIP stream.

The library is loaded on first use; if it has not been built the call raises
``RuntimeError`` (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libppconv.so")

PP_OK, PP_EINVAL, PP_ESIZE, PP_EBLOB, PP_EUNSUPPORTED, PP_EHIP = 0, -1, -2, -3, -4, -5
PP_F32, PP_BF16 = 0, 1
PP_RELU = 1
PP_MAXPOOL2 = 2
PP_ACCUMULATE = 4
PP_PIXSHUF2 = 8
PP_UPSAMPLE2 = 16
PP_PREPARED = 32
PP_NET_TAKEN = 0x80000000
(OP_CONV_PP, OP_CONV_DENSE, OP_DECONV, OP_MAXPOOL2, OP_UPSAMPLE2, OP_PIXSHUF2, OP_ADD) = range(7)

# exported symbols declared in include/pp.h
SYMBOLS = ("pp_pack", "pp_blob_info", "pp_conv2d_fwd", "pp_conv2d_workspace", "pp_conv2d_recipe",
           "pp_conv2d_out_size", "pp_net_workspace", "pp_net_fwd", "pp_status_str", "pp_last_error",
           "pp_project_patterns", "pp_project_connectivity", "pp_project_columns", "pp_column_library",
           "pp_fold_bn", "pp_jit_library", "pp_conv2d_fwd_noalloc", "pp_net_plan", "pp_round_bf16",
           "pp_conv2d_prepare")


class PPError(RuntimeError):
    def __init__(self, status, where, detail):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [("c_out", ctypes.c_int32), ("c_in", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("dilation", ctypes.c_int32), ("wdtype", ctypes.c_int32)]


class NetOp(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("src", ctypes.c_int32), ("src2", ctypes.c_int32),
                ("dst", ctypes.c_int32), ("flags", ctypes.c_uint32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("dilation", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32), ("h_blob", ctypes.c_void_p),
                ("blob_bytes", ctypes.c_size_t), ("d_blob", ctypes.c_void_p), ("d_w", ctypes.c_void_p),
                ("d_b", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load (once) and return the ctypes handle of libppconv.so."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2004_11250_amd.build` "
                           "(or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    vp, sz, i32, u32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_uint32
    argtypes = {
        "pp_pack": [ctypes.POINTER(LayerDesc), vp, vp, vp, vp, vp, i32, vp, ctypes.POINTER(sz)],
        "pp_blob_info": [vp, sz, ctypes.POINTER(LayerDesc), ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_int64)],
        "pp_conv2d_fwd": [vp, sz, vp, vp, vp, i32, i32, i32, i32, u32, vp, sz, vp],
        "pp_conv2d_fwd_noalloc": [vp, sz, vp, vp, vp, i32, i32, i32, i32, u32, vp],
        "pp_conv2d_workspace": [vp, sz, i32, i32, i32, i32, ctypes.POINTER(sz)],
        "pp_conv2d_prepare": [vp, sz, vp, vp, ctypes.POINTER(sz), vp],
        "pp_conv2d_out_size": [vp, sz, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "pp_conv2d_recipe": [vp, sz, i32, i32, i32, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "pp_net_workspace": [ctypes.POINTER(NetOp), i32, i32, i32, i32, i32, i32, ctypes.POINTER(sz),
                             ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "pp_net_fwd": [ctypes.POINTER(NetOp), i32, vp, vp, i32, i32, i32, i32, i32, vp, sz, vp],
        "pp_net_plan": [ctypes.POINTER(NetOp), i32, i32, i32, i32, i32, i32, vp, vp],
        "pp_round_bf16": [vp, vp, sz],
        "pp_jit_library": [vp, sz, i32, i32, i32, i32, i32],
        "pp_project_patterns": [vp, i32, i32, vp, i32, vp, vp],
        "pp_project_connectivity": [vp, i32, i32, ctypes.c_int64, vp],
        "pp_project_columns": [vp, i32, i32, ctypes.c_int64, vp],
        "pp_column_library": [vp, i32, i32, vp, ctypes.POINTER(i32), vp, vp],
        "pp_fold_bn": [vp, vp, i32, i32, vp, vp, vp, vp, ctypes.c_float],
        "pp_status_str": [i32],
        "pp_last_error": [],
    }
    # (the host-only packer library, libppconv_host.so, has the host entry
    # points only)
    for name, at in argtypes.items():
        if hasattr(lib, name):
            fn = getattr(lib, name)
            fn.argtypes = at
            fn.restype = ctypes.c_char_p if name in ("pp_status_str", "pp_last_error") else i32
    _lib = lib
    return lib


def _check(status, where):
    if status != PP_OK:
        lib = load_library()
        raise PPError(status, where, lib.pp_last_error().decode())


def _ptr(a) -> int:
    return a.ctypes.data if isinstance(a, np.ndarray) else int(a)


# ---------------------------------------------------------------------------
# packing (host only)
# ---------------------------------------------------------------------------

def pack(w, b, pattern_id, conn, lib_masks, stride=1, pad=1, dilation=1, wdtype=PP_F32) -> np.ndarray:
    """pp_pack: dense fp32 weights + pattern ids + connectivity -> PPK1 blob (uint8 array)."""
    lib = load_library()
    w = np.ascontiguousarray(w, dtype=np.float32)
    c_out, c_in = w.shape[:2]
    pid = np.ascontiguousarray(pattern_id, dtype=np.uint8)
    conn = np.ascontiguousarray(conn, dtype=np.uint8)
    masks = np.ascontiguousarray(lib_masks, dtype=np.uint16)
    bias = None if b is None else np.ascontiguousarray(b, dtype=np.float32)
    d = LayerDesc(c_out, c_in, stride, pad, dilation, wdtype)
    n = ctypes.c_size_t(0)
    args = (ctypes.byref(d), _ptr(w), None if bias is None else _ptr(bias), _ptr(pid), _ptr(conn), _ptr(masks),
            len(masks))
    _check(lib.pp_pack(*args, None, ctypes.byref(n)), "pp_pack(size)")
    out = np.zeros(n.value, dtype=np.uint8)
    _check(lib.pp_pack(*args, _ptr(out), ctypes.byref(n)), "pp_pack")
    return out


# ---------------------------------------------------------------------------
# pruning-structure helpers (host only)
# ---------------------------------------------------------------------------

def project_patterns(w, lib_masks):
    """pp_project_patterns: (pattern_id u8 [c_out][c_in], kept energy float64
    [c_out][c_in]) of dense 3x3 weights w [c_out][c_in][3][3]."""
    lib = load_library()
    w = np.ascontiguousarray(w, dtype=np.float32)
    masks = np.ascontiguousarray(lib_masks, dtype=np.uint16)
    c_out, c_in = w.shape[:2]
    pid = np.zeros((c_out, c_in), np.uint8)
    e = np.zeros((c_out, c_in), np.float64)
    _check(lib.pp_project_patterns(_ptr(w), c_out, c_in, _ptr(masks), len(masks), _ptr(pid), _ptr(e)),
           "pp_project_patterns")
    return pid, e


def project_connectivity(energy, n_keep):
    """pp_project_connectivity: conn u8 keeping the n_keep largest energies."""
    lib = load_library()
    e = np.ascontiguousarray(energy, dtype=np.float64)
    conn = np.zeros(e.shape, np.uint8)
    _check(lib.pp_project_connectivity(_ptr(e), e.shape[0], e.shape[1], int(n_keep), _ptr(conn)),
           "pp_project_connectivity")
    return conn


def project_columns(w, n_keep):
    """pp_project_columns: u16 [c_in] kept-tap masks of column pruning."""
    lib = load_library()
    w = np.ascontiguousarray(w, dtype=np.float32)
    m = np.zeros(w.shape[1], np.uint16)
    _check(lib.pp_project_columns(_ptr(w), w.shape[0], w.shape[1], int(n_keep), _ptr(m)), "pp_project_columns")
    return m


def column_library(col_mask, c_out):
    """pp_column_library: (lib_masks u16[n_p], pattern_id, conn) of a
    column-pruned layer, ready for pack()."""
    lib = load_library()
    m = np.ascontiguousarray(col_mask, dtype=np.uint16)
    masks = np.zeros(255, np.uint16)
    n = ctypes.c_int32(0)
    pid = np.zeros((c_out, len(m)), np.uint8)
    conn = np.zeros((c_out, len(m)), np.uint8)
    _check(lib.pp_column_library(_ptr(m), c_out, len(m), _ptr(masks), ctypes.byref(n), _ptr(pid), _ptr(conn)),
           "pp_column_library")
    return masks[:n.value].copy(), pid, conn


def fold_bn(w, b, gamma, beta, mean, var, eps=1e-5):
    """pp_fold_bn on copies: (w', b') of a conv followed by an inference-mode
    batch norm (b None: no conv bias)."""
    lib = load_library()
    w = np.array(w, dtype=np.float32, order="C", copy=True)
    b = np.zeros(w.shape[0], np.float32) if b is None else np.array(b, dtype=np.float32, copy=True)
    g, bt, mu, v = (np.ascontiguousarray(a, dtype=np.float32) for a in (gamma, beta, mean, var))
    _check(lib.pp_fold_bn(_ptr(w), _ptr(b), w.shape[0], w[0].size, _ptr(g), _ptr(bt), _ptr(mu), _ptr(v),
                          float(eps)), "pp_fold_bn")
    return w, b


def blob_info(blob) -> dict:
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    d = LayerDesc()
    nk = ctypes.c_int32(0)
    nw = ctypes.c_int64(0)
    _check(lib.pp_blob_info(_ptr(blob), blob.nbytes, ctypes.byref(d), ctypes.byref(nk), ctypes.byref(nw)),
           "pp_blob_info")
    return dict(c_out=d.c_out, c_in=d.c_in, stride=d.stride, pad=d.pad, dilation=d.dilation, wdtype=d.wdtype,
                n_kept=nk.value, n_wt=nw.value)


def out_size(blob, h, w):
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    ho, wo = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib.pp_conv2d_out_size(_ptr(blob), blob.nbytes, h, w, ctypes.byref(ho), ctypes.byref(wo)),
           "pp_conv2d_out_size")
    return ho.value, wo.value


def conv2d_plan(blob, n, h, w, act_dtype=PP_F32, with_workspace=True):
    """(tiling id, channel split) that pp_conv2d_fwd uses for this layer and input."""
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    r, k = ctypes.c_int32(-1), ctypes.c_int32(0)
    _check(lib.pp_conv2d_recipe(_ptr(blob), blob.nbytes, n, h, w, act_dtype, 1 if with_workspace else 0,
                                ctypes.byref(r), ctypes.byref(k)), "pp_conv2d_recipe")
    return r.value, k.value


def conv2d_recipe(blob, n, h, w, act_dtype=PP_F32, with_workspace=True) -> int:
    """Tiling id that pp_conv2d_fwd uses for this layer and input shape."""
    return conv2d_plan(blob, n, h, w, act_dtype, with_workspace)[0]


def jit_library(blob, n, h, w, act_dtype=PP_F32, with_workspace=True) -> None:
    """pp_jit_library: compile and load the kernels specialised for this
    layer's own 4-tap pattern library (seconds; once per process)."""
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    _check(lib.pp_jit_library(_ptr(blob), blob.nbytes, n, h, w, act_dtype, 1 if with_workspace else 0),
           "pp_jit_library")


def conv2d_workspace(blob, n, h, w, act_dtype=PP_F32) -> int:
    """Scratch bytes pp_conv2d_fwd can use for this layer and input."""
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    b = ctypes.c_size_t(0)
    _check(lib.pp_conv2d_workspace(_ptr(blob), blob.nbytes, n, h, w, act_dtype, ctypes.byref(b)),
           "pp_conv2d_workspace")
    return b.value


# ---------------------------------------------------------------------------
# device execution (torch tensors for memory and streams)
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return PP_F32
    if t.dtype == torch.bfloat16:
        return PP_BF16
    raise TypeError(f"activations must be float32 or bfloat16, got {t.dtype}")


def _stream_ptr(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class PackedLayer:
    """A packed layer: host copy (for header parsing) + device copy."""

    def __init__(self, blob: np.ndarray, device="cuda"):
        torch = _torch()
        self.h_blob = np.ascontiguousarray(blob, dtype=np.uint8)
        self.info = blob_info(self.h_blob)
        self.d_blob = torch.from_numpy(self.h_blob.copy()).to(device)
        if self.d_blob.data_ptr() % 256:
            raise RuntimeError("device blob allocation is not 256-byte aligned")
        self.scratch = {}   # conv2d_fwd workspaces by input shape
        self.prepared = None   # matrix-core weights (prepare())

    def prepare(self, stream=None):
        """pp_conv2d_prepare: write this layer's prepared weights once into a
        device buffer kept on the layer (bf16: the matrix-core form's; fp32
        canonical-library stride-1 layers: the lean kernel's expanded
        weights; conv2d_fwd(..., prepared=True) then skips the per-call
        expansion).  Returns the buffer, or None for a layer none of those
        forms runs."""
        torch = _torch()
        lib = load_library()
        nb = ctypes.c_size_t(0)
        st = lib.pp_conv2d_prepare(_ptr(self.h_blob), self.h_blob.nbytes, None, None, ctypes.byref(nb), None)
        if st == PP_EUNSUPPORTED:
            return None
        _check(st, "pp_conv2d_prepare(size)")
        buf = torch.empty(nb.value, dtype=torch.uint8, device=self.d_blob.device)
        if buf.data_ptr() % 256:
            raise RuntimeError("prepared-weights allocation is not 256-byte aligned")
        _check(lib.pp_conv2d_prepare(_ptr(self.h_blob), self.h_blob.nbytes, self.d_blob.data_ptr(), buf.data_ptr(),
                                     ctypes.byref(nb), _stream_ptr(stream)), "pp_conv2d_prepare")
        self.prepared = buf
        return buf

    @classmethod
    def from_weights(cls, w, b, pattern_id, conn, lib_masks, stride=1, pad=1, dilation=1, wdtype=PP_F32,
                     device="cuda"):
        return cls(pack(w, b, pattern_id, conn, lib_masks, stride, pad, dilation, wdtype), device)


def conv2d_fwd(layer: PackedLayer, x, relu=False, out=None, stream=None, workspace="auto", maxpool2=False,
               accumulate=False, pixshuf2=False, upsample2=False, prepared=False):
    """pp_conv2d_fwd on torch tensors; returns y (allocated when out is None).
    workspace: "auto" (a scratch tensor of pp_conv2d_workspace bytes, kept on
    the layer per input shape), None (no scratch) or a uint8 device tensor.
    maxpool2: store the 2 x 2 max pool of the activated output (PP_MAXPOOL2).
    accumulate: add the activated output to ``out`` in place (PP_ACCUMULATE;
    out is required).  pixshuf2: store through PixelShuffle(2)
    (PP_PIXSHUF2).  upsample2: convolve the nearest x2 upsampling of x
    (PP_UPSAMPLE2).  prepared: pass the layer's prepared weights
    (layer.prepare()) at the head of the workspace with PP_PREPARED; when
    the layer can also use split scratch, a copy of them is kept (per input
    shape) at the head of a buffer whose tail is that scratch."""
    torch = _torch()
    lib = load_library()
    if prepared and layer.prepared is None:
        raise ValueError("the layer has no prepared weights (call layer.prepare() first)")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous NCHW")
    n, c, h, w = x.shape
    if c != layer.info["c_in"]:
        raise ValueError(f"x has {c} channels, the layer expects {layer.info['c_in']}")
    hc, wc = (2 * h, 2 * w) if upsample2 else (h, w)   # the conv's input size
    ho, wo = out_size(layer.h_blob, hc, wc)
    c_out = layer.info["c_out"]
    if maxpool2:
        ho, wo = ho // 2, wo // 2
    if pixshuf2:
        c_out, ho, wo = c_out // 4, 2 * ho, 2 * wo
    shape = (n, c_out, ho, wo)
    if accumulate and out is None:
        raise ValueError("accumulate needs out (the residual, updated in place)")
    if out is None:
        out = torch.empty(shape, dtype=x.dtype, device=x.device)
    elif tuple(out.shape) != shape or out.dtype != x.dtype or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {x.dtype} tensor of shape {shape}")
    if prepared:
        nb = conv2d_workspace(layer.h_blob, n, hc, wc, _dtype_code(x))
        workspace = layer.prepared
        if nb:
            key = ("prepared", n, hc, wc, _dtype_code(x), x.device.index)
            head = -(-layer.prepared.numel() // 256) * 256
            workspace = layer.scratch.get(key)
            if workspace is None:
                workspace = torch.empty(head + nb, dtype=torch.uint8, device=x.device)
                workspace[:layer.prepared.numel()].copy_(layer.prepared)
                layer.scratch[key] = workspace
    elif isinstance(workspace, str) and workspace == "auto":
        nb = conv2d_workspace(layer.h_blob, n, hc, wc, _dtype_code(x))
        key = (n, hc, wc, _dtype_code(x), x.device.index)
        workspace = layer.scratch.get(key)
        if nb and (workspace is None or workspace.numel() < nb):
            workspace = torch.empty(nb, dtype=torch.uint8, device=x.device)
            layer.scratch[key] = workspace
        if not nb:
            workspace = None
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel()) if workspace is not None else (None, 0)
    st = lib.pp_conv2d_fwd(_ptr(layer.h_blob), layer.h_blob.nbytes, layer.d_blob.data_ptr(), x.data_ptr(),
                           out.data_ptr(), n, h, w, _dtype_code(x),
                           (PP_RELU if relu else 0) | (PP_MAXPOOL2 if maxpool2 else 0) |
                           (PP_ACCUMULATE if accumulate else 0) | (PP_PIXSHUF2 if pixshuf2 else 0) |
                           (PP_UPSAMPLE2 if upsample2 else 0) | (PP_PREPARED if prepared else 0), ws_ptr, ws_bytes,
                           _stream_ptr(stream))
    _check(st, "pp_conv2d_fwd")
    return out


# ---------------------------------------------------------------------------
# networks: a flat op list over activation slots (pp_net_fwd)
# ---------------------------------------------------------------------------

def round_bf16(a) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), rounded by the library
    (pp_round_bf16: nearest, ties to even) -- the dense weights of a bf16
    network."""
    src = np.ascontiguousarray(a, dtype=np.float32)
    dst = np.empty(src.shape, np.uint16)
    _check(load_library().pp_round_bf16(src.ctypes.data, dst.ctypes.data, src.size), "pp_round_bf16")
    return dst


def _op_array(ops, params, wd, device_tensors):
    """The pp_net_op array of a network spec.  device_tensors(op, prm, blob)
    returns the device buffers of a layer (None for a host-only plan query),
    kept alive by the caller: (d_blob,) for a pruned conv, (d_w, d_b) for a
    dense one.  Returns the array and the host objects it points into."""
    arr = (NetOp * len(ops))()
    keep = []
    for i, (op, prm) in enumerate(zip(ops, params)):
        kind = Net._KIND[op["op"]]
        e = arr[i]
        e.kind = kind
        e.src, e.dst = op["src"], op["dst"]
        e.src2 = op.get("src2", 0)
        e.flags = PP_RELU if op.get("relu") else 0
        if kind == OP_CONV_PP:
            blob = pack(prm["w"], prm["b"], prm["pid"], prm["conn"], prm["lib"], op["stride"], op["pad"], op["dil"], wd)
            dev = device_tensors(op, prm, blob)
            keep.append((blob, dev))
            e.h_blob = blob.ctypes.data
            e.blob_bytes = blob.nbytes
            e.d_blob = dev[0].data_ptr() if dev else None
            prep = dev[1].prepared if dev else None
            e.d_w = prep.data_ptr() if prep is not None else None
        elif kind in (OP_CONV_DENSE, OP_DECONV):
            dev = device_tensors(op, prm, None)
            keep.append(dev)
            e.k, e.stride, e.pad, e.dilation = op["k"], op["stride"], op["pad"], op.get("dil", 1)
            e.c_in, e.c_out = op["c_in"], op["c_out"]
            e.d_w = dev[0].data_ptr() if dev else None
            e.d_b = dev[1].data_ptr() if dev else None
    return arr, keep


def _read_plan(ops, arr, n_ops, n, c, h, w, wd) -> dict:
    lib = load_library()
    flags = (ctypes.c_uint32 * n_ops)()
    recipe = (ctypes.c_int32 * n_ops)()
    _check(lib.pp_net_plan(arr, n_ops, n, c, h, w, wd, flags, recipe), "pp_net_plan")
    fused = {i: ops[i]["op"] for i in range(n_ops) if flags[i] & PP_NET_TAKEN}
    return dict(flags=list(flags), recipe=list(recipe), fused=fused)


def net_plan(ops, params, n, c, h, w, dtype="f32") -> dict:
    """How pp_net_fwd runs a network spec (ops, params as for Net) on an
    n x c x h x w input, as the library plans it (pp_net_plan; host-only):
    ``flags`` per op (a pruned conv's fusion flags, PP_NET_TAKEN for an op
    run inside a conv's launch), ``recipe`` per op (the pruned convs'
    tiling ids, else -1) and ``fused`` = {index: op kind} of the taken ops."""
    wd = PP_BF16 if dtype == "bf16" else PP_F32
    arr, keep = _op_array(ops, params, wd, lambda op, prm, blob: None)
    return _read_plan(ops, arr, len(ops), n, c, h, w, wd)


class Net:
    """A network ready for pp_net_fwd: packed pruned layers and dense weights
    resident on the device, plus the op array.

    ``spec`` is a dict with ``ops`` (list of op dicts: op in conv3 / conv /
    deconv / maxpool2 / up2 / pshuf2 / add, src/src2/dst slots, shapes and
    flags) and ``params`` the matching list of weight dicts (conv3: w, b, pid,
    conn, lib; conv/deconv: w, b)."""

    _KIND = {"conv3": OP_CONV_PP, "conv": OP_CONV_DENSE, "deconv": OP_DECONV, "maxpool2": OP_MAXPOOL2,
             "up2": OP_UPSAMPLE2, "pshuf2": OP_PIXSHUF2, "add": OP_ADD}

    def __init__(self, ops, params, dtype="f32", device="cuda", prepare=True):
        """prepare: write each pruned layer's prepared weights once
        (PackedLayer.prepare: bf16 matrix-core weights, fp32 lean-kernel
        weights) and hand them to pp_net_fwd (pp_net_op.d_w), which reads
        them for the layers it runs in the form they are for instead of
        re-deriving them from the blob on every call."""
        torch = _torch()
        self.dtype = dtype
        self.wd = PP_BF16 if dtype == "bf16" else PP_F32
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.pruned = []     # the PackedLayer of every pruned conv, in op order

        def device_tensors(op, prm, blob):
            if blob is not None:
                L = PackedLayer(blob, device)
                self.pruned.append(L)
                if prepare:
                    L.prepare()
                return (L.d_blob, L)
            w = np.ascontiguousarray(prm["w"], dtype=np.float32)
            if self.wd == PP_BF16:
                dw = torch.from_numpy(round_bf16(w).view(np.int16)).to(device)
            else:
                dw = torch.from_numpy(w).to(device)
            db = torch.from_numpy(np.ascontiguousarray(prm["b"], dtype=np.float32)).to(device)
            return (dw, db)

        arr, self.layers = _op_array(ops, params, self.wd, device_tensors)   # layers: keeps buffers alive
        self.spec_ops = list(ops)
        self.ops = arr
        self.n_ops = len(ops)
        self._ws = None

    def plan(self, n, c, h, w):
        lib = load_library()
        nb = ctypes.c_size_t(0)
        oc, oh, ow = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
        _check(lib.pp_net_workspace(self.ops, self.n_ops, n, c, h, w, self.wd, ctypes.byref(nb), ctypes.byref(oc),
                                    ctypes.byref(oh), ctypes.byref(ow)), "pp_net_workspace")
        return nb.value, (n, oc.value, oh.value, ow.value)

    def launch_plan(self, n, c, h, w) -> dict:
        """net_plan for this network's own op array (pp_net_plan)."""
        return _read_plan(self.spec_ops, self.ops, self.n_ops, n, c, h, w, self.wd)

    def forward(self, x, out=None, workspace=None, stream=None):
        torch = _torch()
        lib = load_library()
        if x.dtype != self.tdtype or not x.is_contiguous():
            raise ValueError("x must be contiguous and of the net's dtype")
        n, c, h, w = x.shape
        nbytes, oshape = self.plan(n, c, h, w)
        if workspace is None:
            if self._ws is None or self._ws.numel() < nbytes:
                self._ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=x.device)
            workspace = self._ws
        if workspace.numel() < nbytes:
            raise ValueError(f"workspace needs {nbytes} bytes")
        if out is None:
            out = torch.empty(oshape, dtype=x.dtype, device=x.device)
        elif tuple(out.shape) != tuple(oshape) or out.dtype != x.dtype or not out.is_contiguous():
            raise ValueError(f"out must be a contiguous {x.dtype} tensor of shape {oshape}")
        _check(lib.pp_net_fwd(self.ops, self.n_ops, x.data_ptr(), out.data_ptr(), n, c, h, w, self.wd,
                              workspace.data_ptr(), workspace.numel(), _stream_ptr(stream)), "pp_net_fwd")
        return out

    def capture(self, x, out, workspace):
        """Record one pp_net_fwd on these fixed buffers (x, out, workspace:
        device tensors that stay alive and in place) as a HIP graph, and
        return it: graph.replay() relaunches the whole network in one call,
        each kernel then costing a graph node's launch instead of a stream
        launch's.  pp_net_fwd launches kernels only (no allocation, copy or
        memset), so the graph holds kernel nodes only.  Replays read x and
        write out as they are at replay time."""
        torch = _torch()
        side = torch.cuda.Stream(device=x.device)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.forward(x, out, workspace, stream=side)   # first call outside the capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize(x.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            self.forward(x, out, workspace)
        return graph
