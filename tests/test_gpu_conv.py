"""GPU parity of pp_conv2d_fwd against the CPU oracle (fp64 masked-dense
direct convolution), element by element, plus bitwise invariants.

Run on an MI355X with ``pytest -m gpu``.  Every case prints its name, seed
and shape before touching the GPU."""
import numpy as np
import pytest

import workloads
from oracle import bf16 as obf16
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _say(*a):
    print(*a, flush=True)


def _to_dev(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def _from_dev(y):
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64)


def run_layer(L, x, stride=1, pad=1, dil=1, relu=True, dtype="f32", out_channels=None):
    """GPU result and oracle (result, bound) on the same rounded inputs."""
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    if dtype == "bf16":
        x = obf16.round_f32(x)
        w_or = obf16.round_f32(L["w"])
    else:
        w_or = L["w"]
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], stride, pad, dil, wd)
    y = _from_dev(pp.conv2d_fwd(layer, _to_dev(x, dtype), relu=relu))
    sel = slice(None) if out_channels is None else out_channels
    args = (x, w_or[sel], L["b"][sel], L["pid"][sel], L["conn"][sel], L["lib"])
    ref = oconv.conv3x3_pruned(*args, stride, pad, dil, relu)
    bound = oconv.conv3x3_bound(*args, stride, pad, dil)
    return y[:, sel], ref, bound


def test_config1_layer():
    spec = workloads.net_spec(1)
    op = spec["ops"][0]
    L = workloads.layer_params(1, 0, op)
    x = workloads.net_input(1)
    _say("config 1 layer 16->16 32x32 fp32 relu")
    y, ref, bound = run_layer(L, x, relu=True)
    check(y, ref, bound, "f32", "config 1")


# (c_out, c_in, h, w, stride, pad, dil, n): sizes the oracle finishes in
# seconds; they span several tiles and channel chunks and end in ragged tails
SHAPES = [
    (16, 16, 32, 32, 1, 1, 1, 1),
    (19, 13, 23, 29, 1, 1, 1, 2),      # small-map tiling, ragged groups/chunks
    (24, 21, 57, 61, 1, 1, 1, 1),      # medium-map tiling
    (12, 10, 101, 131, 1, 1, 1, 1),    # large-map tiling
    (33, 9, 45, 38, 2, 1, 1, 1),       # stride 2
    (20, 17, 34, 30, 1, 2, 2, 1),      # dilation 2
    (9, 11, 41, 27, 2, 2, 2, 1),       # stride 2 + dilation 2
    (8, 3, 5, 7, 1, 0, 1, 1),          # no padding, tiny map
    (5, 4, 1, 1, 1, 1, 1, 3),          # 1x1 map
    (64, 64, 17, 16, 1, 1, 1, 1),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}x{s[1]}_{s[2]}x{s[3]}_s{s[4]}p{s[5]}d{s[6]}" for s in SHAPES])
def test_random_shapes(shape, dtype):
    c_out, c_in, h, w, s, p, d, n = shape
    seed = hash(shape) % 10000
    L = workloads.random_layer(seed, c_out, c_in, keep=0.45)
    x = workloads.random_input(seed, (n, c_in, h, w))
    _say("random layer", shape, dtype, "seed", seed)
    y, ref, bound = run_layer(L, x, s, p, d, relu=bool(seed % 2), dtype=dtype)
    check(y, ref, bound, dtype, f"{shape} {dtype}")


@pytest.mark.parametrize("libname", ["dense9", "generic", "canon8_permuted"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pattern_libraries(libname, dtype):
    rng = np.random.default_rng(3)
    if libname == "dense9":
        lib = np.array([0x1FF], np.uint16)
    elif libname == "generic":
        lib = np.array([0x010, 0x1FF, 0x155, 0x0BA, 0x007, 0x1C0, 0x124, 0x049, 0x03A, 0x111, 0x054], np.uint16)
    else:   # same masks as the canonical library, different order -> generic path
        lib = np.array(workloads.CANON8[::-1], np.uint16)
    L = workloads.random_layer(77, 21, 11, lib=lib, keep=0.6)
    x = workloads.random_input(77, (2, 11, 29, 35))
    for (s, p, d) in ((1, 1, 1), (2, 1, 1), (1, 2, 2)):
        _say("library", libname, dtype, (s, p, d))
        y, ref, bound = run_layer(L, x, s, p, d, relu=False, dtype=dtype)
        check(y, ref, bound, dtype, f"{libname} {dtype} {(s, p, d)}")


def test_generic_library_short_patterns():
    # patterns of 1-3 taps: the last entries of the weight array hold fewer
    # than 4 weights per kernel (a clamp assuming 4 would read the wrong ones)
    lib = np.array([0x002, 0x010, 0x030, 0x111, 0x0C0, 0x100], np.uint16)
    L = workloads.random_layer(91, 24, 9, lib=lib, keep=0.7)
    x = workloads.random_input(91, (2, 9, 15, 13))
    for dtype in ("f32", "bf16"):
        _say("short-pattern library", dtype)
        y, ref, bound = run_layer(L, x, 1, 1, 1, relu=False, dtype=dtype)
        check(y, ref, bound, dtype, f"short patterns {dtype}")


def test_all_kernels_pruned_gives_relu_bias_exactly():
    L = workloads.random_layer(8, 13, 6)
    L["conn"][:] = 0
    x = workloads.random_input(8, (1, 6, 20, 20))
    for relu in (False, True):
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        y = _from_dev(pp.conv2d_fwd(layer, _to_dev(x, "f32"), relu=relu))
        b = np.maximum(L["b"], 0) if relu else L["b"]
        assert np.array_equal(y, np.broadcast_to(b.astype(np.float64)[None, :, None, None], y.shape))


def test_empty_filters_and_unused_channels():
    L = workloads.random_layer(9, 17, 9, keep=0.5)
    L["conn"][3] = 0           # filter 3: no kept kernel
    L["conn"][:, 4] = 0        # channel 4: read by no filter
    x = workloads.random_input(9, (1, 9, 24, 24))
    y, ref, bound = run_layer(L, x)
    check(y, ref, bound, "f32", "empty filter")
    assert np.array_equal(y[:, 3], np.broadcast_to(np.float64(max(L["b"][3], 0)), y[:, 3].shape))


def test_determinism_and_invariants():
    L = workloads.random_layer(10, 24, 16, keep=0.4)
    x = workloads.random_input(10, (1, 16, 40, 44))
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    xd = _to_dev(x, "f32")
    y1 = _from_dev(pp.conv2d_fwd(layer, xd))
    y2 = _from_dev(pp.conv2d_fwd(layer, xd))
    assert np.array_equal(y1, y2), "run-to-run results differ"
    # zero input -> bias, bitwise
    y0 = _from_dev(pp.conv2d_fwd(layer, torch.zeros_like(xd), relu=True))
    assert np.array_equal(y0, np.broadcast_to(np.maximum(L["b"], 0).astype(np.float64)[None, :, None, None], y0.shape))
    # a channel pruned for filter o does not influence it, bitwise
    c = 5
    x2 = x.copy()
    x2[:, c] += 3.0
    y3 = _from_dev(pp.conv2d_fwd(layer, _to_dev(x2, "f32")))
    for o in range(24):
        if not L["conn"][o, c]:
            assert np.array_equal(y1[:, o], y3[:, o]), o
    # power-of-two scaling with zero bias is exact
    L0 = dict(L, b=np.zeros_like(L["b"]))
    layer0 = pp.PackedLayer.from_weights(L0["w"], L0["b"], L0["pid"], L0["conn"], L0["lib"])
    ya = _from_dev(pp.conv2d_fwd(layer0, xd))
    yb = _from_dev(pp.conv2d_fwd(layer0, xd * 4.0))
    assert np.array_equal(4.0 * ya, yb)


def test_filter_order_does_not_change_results():
    # packing the same filters in a different order moves output channels
    # only; the per-filter accumulation order is unchanged, so bitwise equal
    L = workloads.random_layer(11, 20, 12, keep=0.5)
    x = workloads.random_input(11, (1, 12, 30, 30))
    perm = np.random.default_rng(0).permutation(20)
    La = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    Lb = pp.PackedLayer.from_weights(L["w"][perm], L["b"][perm], L["pid"][perm], L["conn"][perm], L["lib"])
    xd = _to_dev(x, "f32")
    ya = _from_dev(pp.conv2d_fwd(La, xd))
    yb = _from_dev(pp.conv2d_fwd(Lb, xd))
    assert np.array_equal(ya[:, perm], yb)


def _vgg_layers():
    spec = workloads.net_spec(2)
    h = spec["h"]
    out = []
    for i, op in enumerate(spec["ops"]):
        if op["op"] == "maxpool2":
            h //= 2
        elif op["op"] == "conv3":
            out.append((i, op, h))
    return out


@pytest.mark.parametrize("idx", range(13))
def test_vgg16_full_size_layer_sampled(idx):
    # full-size VGG-16 layer (224x224 input), the launch configuration the
    # benchmark times; the oracle computes 8 sampled filters completely
    i, op, h = _vgg_layers()[idx]
    L = workloads.layer_params(2, i, op)
    x = workloads.random_input(500 + i, (1, op["c_in"], h, h), 0.0, 1.0)
    sel = np.sort(np.random.default_rng(i).choice(op["c_out"], size=8, replace=False))
    _say("vgg16 layer", i, op["c_in"], "->", op["c_out"], f"{h}x{h}")
    y, ref, bound = run_layer(L, x, relu=True, out_channels=sel)
    check(y, ref, bound, "f32", f"vgg layer {i}")


# the 28 x 28 and 14 x 14 VGG-16 layers at full size and full width: every
# filter against the oracle, in the plan the network runs (the 14 x 14
# layers split their channels over workgroups; the last layer of each block
# with the max pool the network fuses into it)
@pytest.mark.parametrize("idx,pool", [(8, False), (9, True), (10, False), (12, True)])
def test_vgg16_full_width_small_maps(idx, pool):
    i, op, h = _vgg_layers()[idx]
    L = workloads.layer_params(2, i, op)
    x = workloads.random_input(600 + i, (1, op["c_in"], h, h), 0.0, 1.0)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    plan = pp.conv2d_plan(layer.h_blob, 1, h, h, pp.PP_F32)
    _say("vgg16 layer", i, op["c_in"], "->", op["c_out"], f"{h}x{h}", "pool", pool, "plan", plan, "all filters")
    y = _from_dev(pp.conv2d_fwd(layer, _to_dev(x, "f32"), relu=True, maxpool2=pool))
    args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
    ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
    bound = oconv.conv3x3_bound(*args, 1, 1, 1)
    if pool:
        ref, bound = oconv.maxpool2(ref), oconv.maxpool2(bound)
    check(y, ref, bound, "f32", f"vgg layer {i} full width")


# every compiled tiling, forced through the PP_RECIPE override of the planner
RECIPES = list(range(40))


@pytest.mark.parametrize("recipe", RECIPES)
def test_every_tiling(recipe, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    # widths 44/48 (multiples of 4) take the 16-byte staging path, 45/50/33/70 the element-wise one
    for (s, p, d), dtype, shape in (((1, 1, 1), "f32", (19, 21, 37, 45)), ((1, 1, 1), "f32", (19, 21, 37, 44)),
                                    ((2, 1, 1), "f32", (17, 9, 41, 50)), ((2, 1, 1), "f32", (17, 9, 41, 48)),
                                    ((1, 2, 2), "f32", (11, 13, 29, 33)), ((1, 1, 1), "bf16", (24, 17, 33, 70)),
                                    ((1, 1, 1), "bf16", (24, 17, 33, 68))):
        c_out, c_in, h, w = shape
        seed = 40 + recipe
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        used = pp.conv2d_recipe(pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d,
                                        pp.PP_BF16 if dtype == "bf16" else pp.PP_F32), 2, h, w,
                                pp.PP_BF16 if dtype == "bf16" else pp.PP_F32)
        _say("recipe", recipe, "runs as", used, (s, p, d), dtype, shape)
        if (s, p, d) == (1, 1, 1) and dtype == "f32":
            assert used == recipe, "the forced tiling must run for a stride-1 fp32 canonical layer"
        y, ref, bound = run_layer(L, x, s, p, d, relu=True, dtype=dtype)
        check(y, ref, bound, dtype, f"recipe {recipe} {(s, p, d)} {dtype}")


# conv + ReLU + 2 x 2 max pool (PP_MAXPOOL2): against the oracle conv pooled
# (max is 1-Lipschitz: the pooled S bounds the error), and bitwise against
# pooling the unpooled output of the same plan; odd output sizes drop the
# last row / column.  Forced splits pool in the second pass, also for
# tilings with one output row per lane (24, 25).
POOL_RECIPES = [(None, 0), (20, 0), (21, 0), (22, 0), (23, 0), (26, 0), (27, 0), (28, 0), (31, 0), (32, 0),
                (33, 0), (34, 0), (35, 0), (37, 0), (24, 3), (25, 2), (20, 4)]


@pytest.mark.parametrize("recipe,ksplit", POOL_RECIPES)
def test_fused_maxpool(recipe, ksplit, monkeypatch):
    if recipe is not None:
        monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    for (s, p, d), dtype, shape in (((1, 1, 1), "f32", (19, 21, 37, 45)), ((1, 1, 1), "f32", (16, 24, 30, 44)),
                                    ((2, 1, 1), "f32", (17, 9, 41, 50)), ((1, 2, 2), "f32", (11, 13, 29, 33)),
                                    ((1, 1, 1), "bf16", (24, 17, 33, 70)), ((1, 1, 1), "bf16", (8, 20, 14, 14))):
        c_out, c_in, h, w = shape
        seed = 500 + (recipe or 0)
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        if dtype == "bf16":
            x = obf16.round_f32(x)
            w_or = obf16.round_f32(L["w"])
        else:
            w_or = L["w"]
        wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, wd)
        _say("fused maxpool, recipe", recipe, "ksplit", ksplit, (s, p, d), dtype, shape)
        xd = _to_dev(x, dtype)
        yp = pp.conv2d_fwd(layer, xd, relu=True, maxpool2=True)
        args = (x, w_or, L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.maxpool2(oconv.conv3x3_pruned(*args, s, p, d, True))
        bound = oconv.maxpool2(oconv.conv3x3_bound(*args, s, p, d))
        got = _from_dev(yp)
        check(got, ref, bound, dtype, f"fused maxpool recipe {recipe} {(s, p, d)} {dtype} {shape}")
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, wd)
        if recipe is not None and plan[0] == recipe and (not ksplit or plan[1] == ksplit):
            # the same plan unpooled (the pooled plan keeps the forced tiling
            # and the planner's split), pooled on the CPU
            y = pp.conv2d_fwd(layer, xd, relu=True)
            pooled = torch.nn.functional.max_pool2d(y.float().cpu(), 2)
            if dtype == "bf16":
                pooled = pooled.to(torch.bfloat16)
            torch.cuda.synchronize()
            assert torch.equal(yp.cpu(), pooled), f"recipe {recipe}: fused pool differs from pooling the output"


# conv + activation fused with a residual add (PP_ACCUMULATE: y += act(conv))
# or a pixel shuffle (PP_PIXSHUF2): against the oracle conv followed by the
# op (x -> x + r is 1-Lipschitz and the shuffle moves data, so S + |r| and
# the shuffled S bound the error), and bitwise against the same plan's plain
# store followed by the op in torch.  Ragged and vector-store widths, stride
# 2, dilation 2, bf16, and forced channel splits (the second pass takes the
# epilogue).
EPI_RECIPES = [(None, 0), (20, 0), (21, 0), (23, 0), (24, 0), (25, 0), (26, 0), (29, 0), (31, 0), (32, 0),
               (34, 0), (36, 0), (37, 0), (24, 3), (25, 2), (20, 4)]


@pytest.mark.parametrize("recipe,ksplit", EPI_RECIPES)
@pytest.mark.parametrize("mode", ["add", "pshuf2"])
def test_fused_add_pixshuf(mode, recipe, ksplit, monkeypatch):
    if recipe is not None:
        monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    cases = (((1, 1, 1), "f32", (20, 21, 37, 45), True), ((1, 1, 1), "f32", (16, 24, 30, 44), False),
             ((2, 1, 1), "f32", (12, 9, 41, 50), True), ((1, 2, 2), "f32", (8, 13, 29, 36), False),
             ((1, 1, 1), "bf16", (24, 17, 33, 70), False), ((1, 1, 1), "bf16", (8, 20, 14, 16), True))
    for (s, p, d), dtype, shape, relu in cases:
        c_out, c_in, h, w = shape
        seed = 700 + (recipe or 0) + (50 if mode == "add" else 0)
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        if dtype == "bf16":
            x = obf16.round_f32(x)
            w_or = obf16.round_f32(L["w"])
        else:
            w_or = L["w"]
        wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, wd)
        ho, wo = pp.out_size(layer.h_blob, h, w)
        _say("fused", mode, "recipe", recipe, "ksplit", ksplit, (s, p, d), dtype, shape, "relu", relu)
        xd = _to_dev(x, dtype)
        args = (x, w_or, L["b"], L["pid"], L["conn"], L["lib"])
        cref = oconv.conv3x3_pruned(*args, s, p, d, relu)
        cbound = oconv.conv3x3_bound(*args, s, p, d)
        if mode == "add":
            r = workloads.random_input(seed + 1, (2, c_out, ho, wo))
            if dtype == "bf16":
                r = obf16.round_f32(r)
            rd = _to_dev(r, dtype)
            yd = rd.clone()
            pp.conv2d_fwd(layer, xd, relu=relu, out=yd, accumulate=True)
            ref, bound = cref + r.astype(np.float64), cbound + np.abs(r.astype(np.float64))
        else:
            yd = pp.conv2d_fwd(layer, xd, relu=relu, pixshuf2=True)
            ref, bound = oconv.pixel_shuffle2(cref), oconv.pixel_shuffle2(cbound)
        check(_from_dev(yd), ref, bound, dtype, f"fused {mode} recipe {recipe} {(s, p, d)} {dtype} {shape}")
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, wd)
        if recipe is not None and plan[0] == recipe and (not ksplit or plan[1] == ksplit):
            y = pp.conv2d_fwd(layer, xd, relu=relu)
            want = rd + y if mode == "add" else torch.nn.functional.pixel_shuffle(y, 2)
            torch.cuda.synchronize()
            assert torch.equal(yd.cpu(), want.cpu()), f"recipe {recipe}: fused {mode} differs from the op after the conv"


# convolving the nearest x2 upsampling of x, read on the fly (PP_UPSAMPLE2),
# alone and with a fused epilogue: against the oracle conv of the upsampled
# input, and bitwise against the same plan run on the upsampled tensor
UP_RECIPES = [(None, 0), (20, 0), (23, 0), (25, 0), (26, 0), (31, 0), (32, 0), (36, 0), (24, 3), (20, 4)]


@pytest.mark.parametrize("recipe,ksplit", UP_RECIPES)
@pytest.mark.parametrize("mode", ["plain", "add", "maxpool2"])
def test_fused_upsample(mode, recipe, ksplit, monkeypatch):
    if recipe is not None:
        monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    cases = (((1, 1, 1), "f32", (16, 21, 13, 22)), ((1, 1, 1), "f32", (12, 9, 15, 16)),
             ((2, 1, 1), "f32", (8, 11, 17, 12)), ((1, 2, 2), "f32", (20, 7, 9, 14)),
             ((1, 1, 1), "bf16", (24, 17, 11, 35)))
    for (s, p, d), dtype, shape in cases:
        c_out, c_in, h, w = shape
        seed = 900 + (recipe or 0)
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        if dtype == "bf16":
            x = obf16.round_f32(x)
            w_or = obf16.round_f32(L["w"])
        else:
            w_or = L["w"]
        xu = np.ascontiguousarray(np.repeat(np.repeat(x, 2, axis=2), 2, axis=3))
        wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, wd)
        ho, wo = pp.out_size(layer.h_blob, 2 * h, 2 * w)
        _say("fused upsample", mode, "recipe", recipe, "ksplit", ksplit, (s, p, d), dtype, shape)
        args = (xu, w_or, L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.conv3x3_pruned(*args, s, p, d, True)
        bound = oconv.conv3x3_bound(*args, s, p, d)
        xd = _to_dev(x, dtype)
        kw = dict(relu=True, upsample2=True)
        if mode == "add":
            r = workloads.random_input(seed + 1, (2, c_out, ho, wo))
            r = obf16.round_f32(r) if dtype == "bf16" else r
            rd = _to_dev(r, dtype)
            yd = rd.clone()
            pp.conv2d_fwd(layer, xd, out=yd, accumulate=True, **kw)
            ref, bound = ref + r.astype(np.float64), bound + np.abs(r.astype(np.float64))
        elif mode == "maxpool2":
            yd = pp.conv2d_fwd(layer, xd, maxpool2=True, **kw)
            ref, bound = oconv.maxpool2(ref), oconv.maxpool2(bound)
        else:
            yd = pp.conv2d_fwd(layer, xd, **kw)
        check(_from_dev(yd), ref, bound, dtype, f"upsample {mode} recipe {recipe} {(s, p, d)} {dtype} {shape}")
        plan = pp.conv2d_plan(layer.h_blob, 2, 2 * h, 2 * w, wd)
        # (a pooled call cannot keep a tiling with odd R or CC unless it splits)
        same = mode != "maxpool2" or ksplit or recipe not in (25, 36)
        if recipe is not None and same and plan[0] == recipe and (not ksplit or plan[1] == ksplit):
            y = pp.conv2d_fwd(layer, _to_dev(xu, dtype), relu=True)
            if mode == "add":
                want = rd + y
            elif mode == "maxpool2":
                want = torch.nn.functional.max_pool2d(y.float(), 2).to(y.dtype)
            else:
                want = y
            torch.cuda.synchronize()
            assert torch.equal(yd.cpu(), want.cpu()), f"recipe {recipe}: fused upsample ({mode}) differs"


def test_fused_flags_rejected():
    # at most one fused op; the shuffle needs c_out % 4 == 0
    L = workloads.random_layer(9, 6, 8, keep=0.5)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    xd = _to_dev(workloads.random_input(9, (1, 8, 12, 12)), "f32")
    with pytest.raises(pp.PPError):
        pp.conv2d_fwd(layer, xd, maxpool2=True, accumulate=True, out=torch.zeros((1, 6, 6, 6), device="cuda"))
    with pytest.raises(pp.PPError):
        pp.conv2d_fwd(layer, xd, pixshuf2=True, out=torch.zeros((1, 1, 24, 24), device="cuda"))


# channel split over workgroups (partial sums in the workspace, added by a
# second kernel in split order): forced splits, ragged channel shares, both
# activation dtypes
@pytest.mark.parametrize("recipe,ksplit", [(20, 2), (21, 3), (23, 4), (25, 7), (27, 5), (22, 16)])
def test_channel_split(recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    for dtype, shape in (("f32", (21, 77, 29, 36)), ("f32", (16, 64, 14, 14)), ("bf16", (19, 70, 23, 28))):
        c_out, c_in, h, w = shape
        seed = 300 + recipe
        L = workloads.random_layer(seed, c_out, c_in, keep=0.4)
        x = workloads.random_input(seed, (1, c_in, h, w))
        wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, wd)
        used = pp.conv2d_plan(blob, 1, h, w, wd)
        _say("split", recipe, ksplit, dtype, shape, "runs as", used)
        if dtype == "f32":
            assert used == (recipe, ksplit)
        y, ref, bound = run_layer(L, x, relu=True, dtype=dtype)
        check(y, ref, bound, dtype, f"split {recipe}/{ksplit} {dtype} {shape}")
        # repeated calls (counters left at zero, partials rewritten): bitwise equal
        layer = pp.PackedLayer(blob)
        xd = _to_dev(obf16.round_f32(x) if dtype == "bf16" else x, dtype)
        y1 = _from_dev(pp.conv2d_fwd(layer, xd, relu=True))
        y2 = _from_dev(pp.conv2d_fwd(layer, xd, relu=True))
        assert np.array_equal(y1, y2)
