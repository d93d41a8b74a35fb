"""GPU parity of the few-input-channel kernel (recipe 60: fp32 or bf16, at most
four input channels, stride 1, pad 1, any pattern library) against the CPU oracle,
element by element, every filter: one to four channels, ragged tiles in both
directions, widths that are not a multiple of 4, c_out not a multiple of 8,
more slot groups than one workgroup holds, two images, the canonical,
all-ones and a mixed-size pattern library with connectivity pruning, ReLU on
and off; and the full-size first layer of VGG-16 (3 -> 64 at 224 x 224).

Every case prints its name, seed and shape before touching the GPU."""
import numpy as np
import pytest

import workloads
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")

CIN = 60
MIXED = (0x010, 0x1FF, 0x155, 0x0BA, 0x007, 0x1C0, 0x124, 0x049, 0x03A, 0x111, 0x054)
LIBS = {"canon8": workloads.CANON8, "dense9": workloads.DENSE9, "mixed": MIXED}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _say(*a):
    print(*a, flush=True)


# (c_out, c_in, n, h, w)
SHAPES = [(64, 3, 1, 40, 72), (19, 1, 2, 9, 33), (40, 2, 1, 17, 30), (72, 4, 2, 8, 32), (8, 3, 1, 1, 1),
          (5, 4, 1, 23, 5)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("libname", sorted(LIBS))
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_cin_kernel(libname, si, dtype):
    from oracle import bf16 as obf16
    c_out, c_in, n, h, w = SHAPES[si]
    seed = 6000 + 37 * si + len(libname) + (500 if dtype == "bf16" else 0)
    keep = 1.0 if libname == "dense9" and si % 2 == 0 else 0.6
    L = workloads.random_layer(seed, c_out, c_in, lib=LIBS[libname], keep=keep)
    x = workloads.random_input(seed, (n, c_in, h, w))
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
    used = pp.conv2d_recipe(blob, n, h, w, wd)
    _say("cin kernel", libname, dtype, "seed", seed, (c_out, c_in, n, h, w), "runs as", used)
    assert used == CIN
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
    if dtype == "bf16":
        x = obf16.round_f32(x)
        args = (x, obf16.round_f32(L["w"]), L["b"], L["pid"], L["conn"], L["lib"])
        xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    else:
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        xd = torch.from_numpy(x).cuda()
    bound = oconv.conv3x3_bound(*args, 1, 1, 1)
    for relu in (True, False):
        y = pp.conv2d_fwd(layer, xd, relu=relu)
        torch.cuda.synchronize()
        ref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu)
        check(y.float().cpu().numpy().astype(np.float64), ref, bound, dtype,
              f"cin {libname} {dtype} {SHAPES[si]} relu={relu}")


def test_cin_not_taken_for_strides_or_more_channels():
    L = workloads.random_layer(6100, 16, 3)
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    assert pp.conv2d_recipe(blob, 1, 32, 32, pp.PP_F32) == CIN
    s2 = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 1, 1, pp.PP_F32)
    assert pp.conv2d_recipe(s2, 1, 32, 32, pp.PP_F32) != CIN
    L5 = workloads.random_layer(6101, 16, 5)
    b5 = pp.pack(L5["w"], L5["b"], L5["pid"], L5["conn"], L5["lib"], 1, 1, 1, pp.PP_F32)
    assert pp.conv2d_recipe(b5, 1, 32, 32, pp.PP_F32) != CIN
    bb = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    assert pp.conv2d_recipe(bb, 1, 32, 32, pp.PP_BF16) == CIN   # bf16 too


def test_cin_layer_with_fused_pool_runs_elsewhere():
    # a fused max pool is not this kernel's: the layer still runs, pooled
    seed = 6102
    L = workloads.random_layer(seed, 24, 3)
    x = workloads.random_input(seed, (1, 3, 20, 36))
    _say("cin fused pool seed", seed)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    y = pp.conv2d_fwd(layer, torch.from_numpy(x).cuda(), relu=True, maxpool2=True)
    torch.cuda.synchronize()
    args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
    ref = ref.reshape(1, 24, 10, 2, 18, 2).max(axis=(3, 5))
    bound = oconv.conv3x3_bound(*args, 1, 1, 1).reshape(1, 24, 10, 2, 18, 2).max(axis=(3, 5))
    check(y.cpu().numpy().astype(np.float64), ref, bound, "f32", "cin fused pool")


def test_cin_vgg16_first_layer_full_width():
    # 3 -> 64 at 224 x 224, unpruned (the all-ones library): every output
    seed = 6200
    L = workloads.random_layer(seed, 64, 3, lib=workloads.DENSE9, keep=1.0)
    x = workloads.random_input(seed, (1, 3, 224, 224))
    _say("cin vgg16 first layer seed", seed)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    y = pp.conv2d_fwd(layer, torch.from_numpy(x).cuda(), relu=True)
    torch.cuda.synchronize()
    args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
    check(y.cpu().numpy().astype(np.float64), ref, oconv.conv3x3_bound(*args, 1, 1, 1), "f32", "cin vgg16 3->64")
