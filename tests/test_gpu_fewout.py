"""GPU parity of the few-output-channel kernel (recipe 61: at most 8 output
channels, fp32 and bf16, stride 1, pad 1, width a multiple of 4) against the
CPU oracle, element by element, every output: 1 to 8 filters, 1 to 70 input
channels, ragged tiles in both directions, two images, the all-ones library
(which the planner sends here) with and without connectivity pruning, and the
canonical and a mixed-size library forced onto it (fp32 layers forced too:
the planner sends bf16 all-ones layers here); plus the full-width
super-resolution output layer (64 -> 3 at 1080 x 1920) on sampled rows.

Every case prints its name, seed and shape before touching the GPU."""
import numpy as np
import pytest

import workloads
from oracle import bf16 as obf16
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")

FEW = 61
MIXED = (0x010, 0x1FF, 0x155, 0x0BA, 0x007, 0x1C0, 0x124, 0x049, 0x03A, 0x111, 0x054)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _say(*a):
    print(*a, flush=True)


def _run(L, x, dtype, relu):
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    if dtype == "bf16":
        x = obf16.round_f32(x)
        w_or = obf16.round_f32(L["w"])
    else:
        w_or = L["w"]
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
    xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    if dtype == "bf16":
        xd = xd.to(torch.bfloat16)
    y = pp.conv2d_fwd(layer, xd, relu=relu)
    torch.cuda.synchronize()
    args = (x, w_or, L["b"], L["pid"], L["conn"], L["lib"])
    return y.float().cpu().numpy().astype(np.float64), args


# (c_out, c_in, n, h, w)
SHAPES = [(3, 64, 1, 40, 132), (1, 5, 2, 9, 12), (4, 17, 1, 33, 68), (6, 70, 1, 37, 64), (8, 3, 2, 8, 4),
          (2, 1, 1, 70, 36)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_fewout_dense9(si, dtype, monkeypatch):
    c_out, c_in, n, h, w = SHAPES[si]
    # (fp32, and layers of at most 4 input channels, which the planner gives
    # the few-input-channel kernel: forced)
    if dtype == "f32" or c_in <= 4:
        monkeypatch.setenv("PP_RECIPE", str(FEW))
    seed = 7000 + 31 * si + (dtype == "bf16")
    keep = 1.0 if si % 2 == 0 else 0.7
    L = workloads.random_layer(seed, c_out, c_in, lib=workloads.DENSE9, keep=keep)
    x = workloads.random_input(seed, (n, c_in, h, w))
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
    used = pp.conv2d_recipe(blob, n, h, w, wd)
    _say("fewout dense9", dtype, "seed", seed, (c_out, c_in, n, h, w), "keep", keep, "runs as", used)
    assert used == FEW
    for relu in (True, False):
        y, args = _run(L, x, dtype, relu)
        ref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu)
        bound = oconv.conv3x3_bound(*args, 1, 1, 1)
        check(y, ref, bound, dtype, f"fewout {SHAPES[si]} {dtype} relu={relu}")


@pytest.mark.parametrize("libname", ["canon8", "mixed"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fewout_forced_other_libraries(libname, dtype, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(FEW))
    lib = workloads.CANON8 if libname == "canon8" else MIXED
    for si, (c_out, c_in, n, h, w) in enumerate([(5, 23, 2, 19, 44), (8, 40, 1, 16, 64)]):
        seed = 7100 + 7 * si + (dtype == "bf16") + 2 * (libname == "mixed")
        L = workloads.random_layer(seed, c_out, c_in, lib=lib, keep=0.6)
        x = workloads.random_input(seed, (n, c_in, h, w))
        wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
        used = pp.conv2d_recipe(blob, n, h, w, wd)
        _say("fewout forced", libname, dtype, "seed", seed, (c_out, c_in, n, h, w), "runs as", used)
        assert used == FEW
        y, args = _run(L, x, dtype, True)
        check(y, oconv.conv3x3_pruned(*args, 1, 1, 1, True), oconv.conv3x3_bound(*args, 1, 1, 1), dtype,
              f"fewout forced {libname} {dtype}")


def test_fewout_not_taken():
    B = pp.PP_BF16
    L = workloads.random_layer(7200, 3, 16, lib=workloads.DENSE9, keep=1.0)
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, B)
    assert pp.conv2d_recipe(blob, 1, 32, 32, B) == FEW
    assert pp.conv2d_recipe(blob, 1, 32, 30, B) != FEW                  # width not a multiple of 4
    f32 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    assert pp.conv2d_recipe(f32, 1, 32, 32, pp.PP_F32) != FEW           # fp32 (unless forced)
    s2 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 1, 1, B)
    assert pp.conv2d_recipe(s2, 1, 32, 32, B) != FEW                    # stride 2
    L9 = workloads.random_layer(7201, 9, 16, lib=workloads.DENSE9, keep=1.0)
    b9 = pp.pack(L9["w"], L9["b"], L9["pid"], L9["conn"], L9["lib"], 1, 1, 1, B)
    assert pp.conv2d_recipe(b9, 1, 32, 32, B) != FEW                    # two slot groups
    Lc = workloads.random_layer(7202, 3, 16, keep=0.5)
    bc = pp.pack(Lc["w"], Lc["b"], Lc["pid"], Lc["conn"], Lc["lib"], 1, 1, 1, B)
    assert pp.conv2d_recipe(bc, 1, 32, 32, B) != FEW                    # pruned canonical library
    L3 = workloads.random_layer(7203, 3, 3, lib=workloads.DENSE9, keep=1.0)
    b3 = pp.pack(L3["w"], L3["b"], L3["pid"], L3["conn"], L3["lib"], 1, 1, 1, B)
    assert pp.conv2d_recipe(b3, 1, 32, 32, B) == 60                     # 3 input channels: that kernel first


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fewout_super_resolution_output_layer(dtype, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(FEW))
    # 64 -> 3 at 1080 x 1920 (the super-resolution network's last layer):
    # every output of rows that start, cross and end wave and workgroup
    # tiles, computed by the oracle on the rows it needs
    seed = 7300 + (dtype == "bf16")
    h, w = 1080, 1920
    L = workloads.random_layer(seed, 3, 64, lib=workloads.DENSE9, keep=1.0)
    x = workloads.random_input(seed, (1, 64, h, w), 0.0, 1.0)
    _say("fewout sr output layer", dtype, "seed", seed)
    y, args = _run(L, x, dtype, False)
    xr = args[0]
    for r0 in (0, 7, 31, 32, 530, 1071):
        lo, hi = max(r0 - 1, 0), min(r0 + 9, h)
        sub = xr[:, :, lo:hi]
        ref = oconv.conv3x3_pruned(sub, *args[1:], 1, 1, 1, False)
        bound = oconv.conv3x3_bound(sub, *args[1:], 1, 1, 1)
        # rows of sub's output that have their true neighbours (not sub's edge)
        a0 = r0 - lo
        a1 = min(r0 + 8, h) - lo
        if lo > 0 and a0 == 0:
            a0 = 1
        keep_hi = a1 if hi == h else min(a1, hi - lo - 1)
        check(y[:, :, lo + a0:lo + keep_hi], ref[:, :, a0:keep_hi], bound[:, :, a0:keep_hi], dtype,
              f"fewout sr rows {r0} {dtype}")
