"""pp_conv2d_fwd_noalloc (scratch in a file-scope device array, no
allocation) against pp_conv2d_fwd with a pp_conv2d_workspace()-sized
workspace: the same plan, so bitwise the same output; two calls in a row on
one layer, the second with a smaller input (the array keeps the first call's
contents); layers that split their channels, run on the bf16 matrix cores,
or need no scratch; the oracle on the small case; and the size limit."""
import ctypes

import numpy as np
import pytest

import workloads
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")

LIMIT = 16 << 20


def _say(*a):
    print(*a, flush=True)


def _run_both(layer, x, relu=True):
    """(noalloc output, pp_conv2d_fwd output) for one input."""
    lib = pp.load_library()
    n, c, h, w = x.shape
    wd = pp.PP_BF16 if x.dtype == torch.bfloat16 else pp.PP_F32
    ho, wo = pp.out_size(layer.h_blob, h, w)
    shape = (n, layer.info["c_out"], ho, wo)
    y_na = torch.full(shape, float("nan"), dtype=x.dtype, device="cuda")
    st = lib.pp_conv2d_fwd_noalloc(layer.h_blob.ctypes.data, layer.h_blob.nbytes, layer.d_blob.data_ptr(),
                                   x.data_ptr(), y_na.data_ptr(), n, h, w, wd, pp.PP_RELU if relu else 0, None)
    assert st == pp.PP_OK, lib.pp_last_error().decode()
    nb = pp.conv2d_workspace(layer.h_blob, n, h, w, wd)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda")
    y_ref = torch.full(shape, float("nan"), dtype=x.dtype, device="cuda")
    st = lib.pp_conv2d_fwd(layer.h_blob.ctypes.data, layer.h_blob.nbytes, layer.d_blob.data_ptr(), x.data_ptr(),
                           y_ref.data_ptr(), n, h, w, wd, pp.PP_RELU if relu else 0,
                           ws.data_ptr() if nb else None, nb, None)
    assert st == pp.PP_OK, lib.pp_last_error().decode()
    torch.cuda.synchronize()
    return y_na, y_ref, nb


@pytest.mark.parametrize("dtype,c_out,c_in,hw1,hw2,n", [
    ("f32", 512, 512, 14, 12, 1),    # channel split over workgroups (partial sums in the scratch)
    ("bf16", 256, 256, 32, 16, 2),   # bf16 channel split, exactly the scratch limit on the first call
    ("bf16", 512, 512, 32, 24, 8),   # bf16 matrix-core form (expanded weights in the scratch)
    ("f32", 16, 16, 32, 20, 1),      # no scratch
])
def test_noalloc_equals_workspace_call(dtype, c_out, c_in, hw1, hw2, n):
    L = workloads.random_layer(c_out + c_in + hw1, c_out, c_in, keep=0.4)
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    for call, hw in enumerate((hw1, hw2)):
        x_np = workloads.random_input(100 * call + hw, (n, c_in, hw, hw), 0.0, 1.0)
        x = torch.from_numpy(x_np).cuda().to(tdt)
        _say("noalloc", dtype, (c_out, c_in), "call", call, "input", (n, c_in, hw, hw),
             "plan", pp.conv2d_plan(layer.h_blob, n, hw, hw, wd))
        y_na, y_ref, nb = _run_both(layer, x)
        assert nb <= LIMIT
        assert torch.equal(y_na, y_ref), f"call {call}: noalloc differs from the workspace call"
        if c_out * c_in <= 256:
            got = y_na.float().cpu().numpy().astype(np.float64)
            args = (x_np, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
            check(got, oconv.conv3x3_pruned(*args, 1, 1, 1, True), oconv.conv3x3_bound(*args, 1, 1, 1), dtype,
                  "noalloc small layer")


def test_noalloc_rejects_layers_beyond_the_scratch():
    # the matrix-core form of this layer needs 37.7 MB of expanded weights
    L = workloads.random_layer(5, 1024, 2048, keep=0.3)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    assert pp.conv2d_workspace(layer.h_blob, 2, 32, 32, pp.PP_BF16) > LIMIT
    lib = pp.load_library()
    x = torch.zeros((2, 2048, 32, 32), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((2, 1024, 32, 32), dtype=torch.bfloat16, device="cuda")
    st = lib.pp_conv2d_fwd_noalloc(layer.h_blob.ctypes.data, layer.h_blob.nbytes, layer.d_blob.data_ptr(),
                                   x.data_ptr(), y.data_ptr(), 2, 32, 32, pp.PP_BF16, pp.PP_RELU, None)
    assert st == pp.PP_ESIZE
    assert b"scratch" in lib.pp_last_error()
    torch.cuda.synchronize()
    assert torch.count_nonzero(y).item() == 0   # nothing was enqueued
