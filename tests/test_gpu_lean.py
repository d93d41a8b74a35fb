"""GPU parity of the lean pruned-conv kernel (tilings 40-50: fp32, canonical
library, stride 1, pad 1, image width a multiple of 4) against the CPU
oracle, element by element, every filter; fused max pool bitwise against
pooling the unpooled output of the same plan; forced channel splits; and
full-width parity on full-size VGG-16 layers.

Every case prints its name, seed and shape before touching the GPU."""
import numpy as np
import pytest

import workloads
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")

# tilings 40-50 and 58 stage the halo by 16-byte DMAs (image width a
# multiple of 4), 51-57 and 59 by 4-byte DMAs (any width)
LEAN = list(range(40, 60))
V4 = set(range(40, 51)) | {58}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _say(*a):
    print(*a, flush=True)


def _run(L, x, relu=True, maxpool2=False):
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    y = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=maxpool2)
    torch.cuda.synchronize()
    return layer, xd, y


# shapes: (c_out, c_in, h, w): ragged tiles in both directions, c_out not a
# multiple of 8 (padding slots), fewer channels than waves, 2 images; odd
# and not-multiple-of-4 widths for the 4-byte staging tilings
SHAPES = [(19, 21, 37, 44), (16, 64, 32, 32), (24, 5, 20, 40), (8, 40, 70, 68)]
SHAPES_B32 = [(19, 21, 37, 45), (16, 64, 14, 14), (24, 5, 21, 30), (8, 40, 33, 17)]


@pytest.mark.parametrize("recipe", LEAN)
def test_lean_tiling(recipe, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    for si, (c_out, c_in, h, w) in enumerate(SHAPES + ([] if recipe in V4 else SHAPES_B32)):
        seed = 1000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
        used = pp.conv2d_recipe(blob, 2, h, w, pp.PP_F32)
        _say("lean tiling", recipe, "runs as", used, "seed", seed, (c_out, c_in, h, w))
        assert used == recipe
        for relu in (True, False):
            _, _, y = _run(L, x, relu=relu)
            got = y.cpu().numpy().astype(np.float64)
            args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
            ref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu)
            bound = oconv.conv3x3_bound(*args, 1, 1, 1)
            check(got, ref, bound, "f32", f"lean {recipe} {(c_out, c_in, h, w)} relu={relu}")


# (tiling 54 has one output row per lane: it pools only under a channel split)
@pytest.mark.parametrize("recipe", [r for r in LEAN if r != 54])
def test_lean_fused_maxpool(recipe, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    shapes = [(19, 21, 37, 44), (16, 24, 30, 44), (8, 33, 64, 64)]
    if recipe not in V4:
        shapes += [(16, 24, 14, 14), (8, 19, 29, 31)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 2000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        _say("lean fused maxpool", recipe, "seed", seed, (c_out, c_in, h, w))
        layer, xd, yp = _run(L, x, maxpool2=True)
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.maxpool2(oconv.conv3x3_pruned(*args, 1, 1, 1, True))
        bound = oconv.maxpool2(oconv.conv3x3_bound(*args, 1, 1, 1))
        check(yp.cpu().numpy().astype(np.float64), ref, bound, "f32", f"lean pool {recipe}")
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_F32)
        assert plan[0] == recipe
        y = pp.conv2d_fwd(layer, xd, relu=True)
        pooled = torch.nn.functional.max_pool2d(y.cpu(), 2)
        assert torch.equal(yp.cpu(), pooled), f"lean {recipe}: fused pool differs from pooling the output"


@pytest.mark.parametrize("recipe,ksplit", [(40, 2), (45, 3), (47, 4), (48, 2), (49, 5), (42, 2), (51, 2), (52, 4),
                                           (54, 3), (55, 2), (58, 2), (59, 3)])
def test_lean_channel_split(recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(21, 77, 29, 36), (16, 64, 12, 16), (24, 40, 28, 28)]
    if recipe not in V4:
        shapes += [(16, 64, 14, 14), (21, 77, 29, 35)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 3000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.4)
        x = workloads.random_input(seed, (1, c_in, h, w))
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
        used = pp.conv2d_plan(blob, 1, h, w, pp.PP_F32)
        _say("lean split", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "runs as", used)
        assert used == (recipe, ksplit)
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        for pool in (False, True):
            layer, xd, y = _run(L, x, maxpool2=pool)
            ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
            bound = oconv.conv3x3_bound(*args, 1, 1, 1)
            if pool:
                ref, bound = oconv.maxpool2(ref), oconv.maxpool2(bound)
            check(y.cpu().numpy().astype(np.float64), ref, bound, "f32", f"lean split {recipe}/{ksplit} pool={pool}")
        y1 = pp.conv2d_fwd(layer, xd, relu=True)
        y2 = pp.conv2d_fwd(layer, xd, relu=True)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2), "repeated split calls must be bitwise equal"


# conv + activation fused with a residual add (PP_ACCUMULATE) or a pixel
# shuffle (PP_PIXSHUF2): against the oracle conv followed by the op, and
# bitwise against the same plan's plain store followed by the op in torch;
# forced splits take the epilogue in the second pass
@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN] + [(40, 3), (48, 2), (54, 2), (52, 4)])
@pytest.mark.parametrize("mode", ["add", "pshuf2"])
def test_lean_fused_add_pixshuf(mode, recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(20, 21, 37, 44, True), (16, 24, 30, 44, False)]
    if recipe not in V4:
        shapes += [(8, 13, 29, 35, True)]
    for si, (c_out, c_in, h, w, relu) in enumerate(shapes):
        seed = 4000 + 10 * recipe + si + (5 if mode == "add" else 0)
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        _say("lean fused", mode, "recipe", recipe, "ksplit", ksplit, "seed", seed, (c_out, c_in, h, w), "relu", relu)
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
        xd = torch.from_numpy(x).cuda()
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        cref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu)
        cbound = oconv.conv3x3_bound(*args, 1, 1, 1)
        if mode == "add":
            r = workloads.random_input(seed + 1, (2, c_out, h, w))
            rd = torch.from_numpy(r).cuda()
            yd = rd.clone()
            pp.conv2d_fwd(layer, xd, relu=relu, out=yd, accumulate=True)
            ref, bound = cref + r.astype(np.float64), cbound + np.abs(r.astype(np.float64))
        else:
            yd = pp.conv2d_fwd(layer, xd, relu=relu, pixshuf2=True)
            ref, bound = oconv.pixel_shuffle2(cref), oconv.pixel_shuffle2(cbound)
        torch.cuda.synchronize()
        check(yd.cpu().numpy().astype(np.float64), ref, bound, "f32", f"lean fused {mode} recipe {recipe}")
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_F32)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        y = pp.conv2d_fwd(layer, xd, relu=relu)
        want = rd + y if mode == "add" else torch.nn.functional.pixel_shuffle(y, 2)
        torch.cuda.synchronize()
        assert torch.equal(yd.cpu(), want.cpu()), f"lean {recipe}: fused {mode} differs from the op after the conv"


# convolving the nearest x2 upsampling of x read on the fly (PP_UPSAMPLE2,
# 4-byte staging tilings), alone and with a fused add or max pool: against
# the oracle conv of the upsampled input, and bitwise against the same plan
# run on the upsampled tensor
@pytest.mark.parametrize("recipe,ksplit", [(51, 0), (52, 0), (53, 0), (55, 0), (56, 0), (57, 0), (54, 2), (52, 3)])
@pytest.mark.parametrize("mode", ["plain", "add", "maxpool2"])
def test_lean_fused_upsample(mode, recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    for si, (c_out, c_in, h, w) in enumerate([(16, 21, 13, 22), (12, 9, 15, 16), (8, 24, 14, 14)]):
        seed = 5000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        xu = np.ascontiguousarray(np.repeat(np.repeat(x, 2, axis=2), 2, axis=3))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
        _say("lean fused upsample", mode, "recipe", recipe, "ksplit", ksplit, "seed", seed, (c_out, c_in, h, w))
        args = (xu, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
        bound = oconv.conv3x3_bound(*args, 1, 1, 1)
        xd = torch.from_numpy(x).cuda()
        kw = dict(relu=True, upsample2=True)
        if mode == "add":
            r = workloads.random_input(seed + 1, (2, c_out, 2 * h, 2 * w))
            rd = torch.from_numpy(r).cuda()
            yd = rd.clone()
            pp.conv2d_fwd(layer, xd, out=yd, accumulate=True, **kw)
            ref, bound = ref + r.astype(np.float64), bound + np.abs(r.astype(np.float64))
        elif mode == "maxpool2":
            yd = pp.conv2d_fwd(layer, xd, maxpool2=True, **kw)
            ref, bound = oconv.maxpool2(ref), oconv.maxpool2(bound)
        else:
            yd = pp.conv2d_fwd(layer, xd, **kw)
        torch.cuda.synchronize()
        check(yd.cpu().numpy().astype(np.float64), ref, bound, "f32", f"lean upsample {mode} recipe {recipe}")
        plan = pp.conv2d_plan(layer.h_blob, 2, 2 * h, 2 * w, pp.PP_F32)
        assert plan[0] == recipe
        if mode == "maxpool2" and recipe == 54 and not ksplit:
            continue   # one output row per lane: pools only under a split
        y = pp.conv2d_fwd(layer, torch.from_numpy(xu).cuda(), relu=True)
        if mode == "add":
            want = rd + y
        elif mode == "maxpool2":
            want = torch.nn.functional.max_pool2d(y, 2)
        else:
            want = y
        torch.cuda.synchronize()
        assert torch.equal(yd.cpu(), want.cpu()), f"lean {recipe}: fused upsample ({mode}) differs"


# ---- bf16 activations (the tilings built for bf16: 16-byte staging needs a
# width that is a multiple of 8, 4-byte staging an even width).  Inputs and
# weights are rounded to bf16 for the oracle too; the output is rounded once.
LEAN_BF = [40, 56, 46, 55, 58, 59, 48, 51, 54]
V4_BF = {40, 46, 58, 48}


def _run_bf16(L, x, relu=True, maxpool2=False):
    from oracle import bf16 as obf16
    xr = obf16.round_f32(x)
    wr = obf16.round_f32(L["w"])
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    xd = torch.from_numpy(np.ascontiguousarray(xr, np.float32)).cuda().to(torch.bfloat16)
    y = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=maxpool2)
    torch.cuda.synchronize()
    args = (xr, wr, L["b"], L["pid"], L["conn"], L["lib"])
    return layer, xd, y, args


@pytest.mark.parametrize("recipe", LEAN_BF)
def test_lean_bf16_tiling(recipe, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    shapes = [(19, 21, 37, 48), (16, 64, 32, 32), (24, 5, 20, 40), (8, 40, 70, 64)]
    if recipe not in V4_BF:
        shapes += [(19, 21, 37, 46), (16, 64, 14, 14), (24, 5, 21, 30), (8, 40, 33, 18)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 8000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
        used = pp.conv2d_recipe(blob, 2, h, w, pp.PP_BF16)
        _say("lean bf16 tiling", recipe, "runs as", used, "seed", seed, (c_out, c_in, h, w))
        assert used == recipe
        for relu in (True, False):
            _, _, y, args = _run_bf16(L, x, relu=relu)
            ref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu)
            bound = oconv.conv3x3_bound(*args, 1, 1, 1)
            check(y.float().cpu().numpy().astype(np.float64), ref, bound, "bf16",
                  f"lean bf16 {recipe} {(c_out, c_in, h, w)} relu={relu}")


@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN_BF if r != 54] + [(48, 2), (51, 4), (54, 2), (46, 3)])
def test_lean_bf16_pool_and_split(recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(19, 21, 36, 48), (16, 64, 32, 32)]
    if recipe not in V4_BF:
        shapes += [(16, 64, 14, 14), (8, 19, 29, 30)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 8500 + 10 * recipe + si + ksplit
        L = workloads.random_layer(seed, c_out, c_in, keep=0.4)
        x = workloads.random_input(seed, (1, c_in, h, w))
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
        plan = pp.conv2d_plan(blob, 1, h, w, pp.PP_BF16)
        _say("lean bf16 pool/split", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "runs as", plan)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        for pool in ((False, True) if ksplit else (True,)):
            layer, xd, y, args = _run_bf16(L, x, maxpool2=pool)
            ref = oconv.conv3x3_pruned(*args, 1, 1, 1, True)
            bound = oconv.conv3x3_bound(*args, 1, 1, 1)
            if pool:
                ref, bound = oconv.maxpool2(ref), oconv.maxpool2(bound)
            check(y.float().cpu().numpy().astype(np.float64), ref, bound, "bf16",
                  f"lean bf16 {recipe}/{ksplit} pool={pool}")
            if pool:
                yu = pp.conv2d_fwd(layer, xd, relu=True)
                pooled = torch.nn.functional.max_pool2d(yu.float().cpu(), 2)
                assert torch.equal(y.float().cpu(), pooled), f"lean bf16 {recipe}: fused pool differs"


def test_lean_bf16_not_for_other_epilogues():
    # the bf16 lean tilings take ReLU, the max pool and the residual add: a
    # fused pixel shuffle or upsample, or an odd width, runs on another kernel
    L = workloads.random_layer(8900, 16, 32, keep=0.5)
    blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    assert pp.conv2d_recipe(blob, 1, 56, 56, pp.PP_BF16) in LEAN_BF
    assert pp.conv2d_recipe(blob, 1, 56, 55, pp.PP_BF16) not in range(40, 60)   # odd width


# fp32 prepared weights (pp_conv2d_prepare; PP_PREPARED): the tilings built
# for them read the expanded weights by scalar loads and give bitwise what
# the same tiling gives staging them from the blob, with and without a
# channel split (whose scratch follows the prepared weights)
PW = [40, 56, 46, 55, 58, 59, 48, 51, 54]


@pytest.mark.parametrize("recipe", PW)
def test_lean_prepared_weights_bitwise(recipe, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    shapes = [(19, 21, 37, 44), (16, 64, 32, 32), (8, 40, 20, 40)]
    if recipe not in V4:
        shapes += [(19, 21, 37, 45), (16, 64, 14, 14)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 9000 + 10 * recipe + si
        L = workloads.random_layer(seed, c_out, c_in, keep=0.4)
        x = workloads.random_input(seed, (2, c_in, h, w))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
        _say("lean prepared", recipe, "seed", seed, (c_out, c_in, h, w))
        assert layer.prepare() is not None
        xd = torch.from_numpy(x).cuda()
        for relu, pool in ((True, False), (False, False), (True, True)):
            if pool and (recipe == 54 or h % 2 or w % 2):
                continue
            # the same plan both ways (a split gets its scratch behind the
            # prepared weights)
            ya = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=pool)
            yb = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=pool, prepared=True)
            torch.cuda.synchronize()
            assert torch.equal(ya, yb), f"prepared {recipe} relu={relu} pool={pool}"
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        check(yb.cpu().numpy().astype(np.float64) if not pool else
              pp.conv2d_fwd(layer, xd, relu=True, prepared=True).cpu().numpy().astype(np.float64),
              oconv.conv3x3_pruned(*args, 1, 1, 1, True), oconv.conv3x3_bound(*args, 1, 1, 1), "f32",
              f"lean prepared {recipe}")


# bf16 layers' prepared lean weights (the fp32 widening of the bf16 weights,
# after the matrix-core part when c_in is a multiple of 32): every bf16
# tiling, bitwise what the blob-staged weights give, with the pool and a
# channel split
@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN_BF] + [(51, 4), (46, 3)])
def test_lean_bf16_prepared_weights_bitwise(recipe, ksplit, monkeypatch):
    from oracle import bf16 as obf16
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(19, 21, 36, 48), (16, 64, 32, 32), (8, 40, 20, 40)]
    if recipe not in V4_BF:
        shapes += [(19, 21, 37, 46), (16, 64, 14, 14)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 9500 + 10 * recipe + si + ksplit
        L = workloads.random_layer(seed, c_out, c_in, keep=0.4)
        x = workloads.random_input(seed, (2, c_in, h, w))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_BF16)
        _say("lean bf16 prepared", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "runs as", plan)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        assert layer.prepare() is not None
        xr = obf16.round_f32(x)
        xd = torch.from_numpy(np.ascontiguousarray(xr, np.float32)).cuda().to(torch.bfloat16)
        for relu, pool in ((True, False), (False, False), (True, True)):
            if pool and (recipe == 54 or h % 2 or w % 2):
                continue
            ya = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=pool)
            yb = pp.conv2d_fwd(layer, xd, relu=relu, maxpool2=pool, prepared=True)
            torch.cuda.synchronize()
            assert torch.equal(ya, yb), f"bf16 prepared {recipe}/{ksplit} relu={relu} pool={pool}"
        args = (xr, obf16.round_f32(L["w"]), L["b"], L["pid"], L["conn"], L["lib"])
        y = pp.conv2d_fwd(layer, xd, relu=False, prepared=True)
        check(y.float().cpu().numpy().astype(np.float64), oconv.conv3x3_pruned(*args, 1, 1, 1, False),
              oconv.conv3x3_bound(*args, 1, 1, 1), "bf16", f"lean bf16 prepared {recipe}/{ksplit}")


# bf16 conv fused with a residual add (PP_ACCUMULATE): the activated value
# rounded to bf16, added to the stored residual and rounded again -- bitwise
# the same plan's plain store followed by a bf16 add in torch -- with and
# without prepared weights, on every bf16 tiling and through the split's
# second pass
@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN_BF] + [(46, 3), (51, 4), (54, 2)])
def test_lean_bf16_fused_add(recipe, ksplit, monkeypatch):
    from oracle import bf16 as obf16
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(20, 21, 36, 48, True), (16, 64, 32, 32, False)]
    if recipe not in V4_BF:
        shapes += [(8, 13, 29, 34, True), (16, 64, 14, 14, False)]
    for si, (c_out, c_in, h, w, relu) in enumerate(shapes):
        seed = 9700 + 10 * recipe + si + ksplit
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = obf16.round_f32(workloads.random_input(seed, (2, c_in, h, w)))
        r = obf16.round_f32(workloads.random_input(seed + 1, (2, c_out, h, w)))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_BF16)
        _say("lean bf16 fused add", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "relu", relu, "runs as", plan)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        assert layer.prepare() is not None
        xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda().to(torch.bfloat16)
        rd = torch.from_numpy(np.ascontiguousarray(r, np.float32)).cuda().to(torch.bfloat16)
        y_plain = pp.conv2d_fwd(layer, xd, relu=relu)
        ya = rd.clone()
        pp.conv2d_fwd(layer, xd, relu=relu, out=ya, accumulate=True)
        yb = rd.clone()
        pp.conv2d_fwd(layer, xd, relu=relu, out=yb, accumulate=True, prepared=True)
        torch.cuda.synchronize()
        assert torch.equal(ya, rd + y_plain), f"bf16 fused add {recipe}/{ksplit} differs from the add after the conv"
        assert torch.equal(ya, yb), f"bf16 fused add {recipe}/{ksplit}: prepared weights differ"
        args = (x, obf16.round_f32(L["w"]), L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.conv3x3_pruned(*args, 1, 1, 1, relu) + r.astype(np.float64)
        bound = oconv.conv3x3_bound(*args, 1, 1, 1) + np.abs(r.astype(np.float64))
        check(ya.float().cpu().numpy().astype(np.float64), ref, bound, "bf16", f"lean bf16 add {recipe}/{ksplit}")


# dilation 2 (pad 2, fp32): every tiling built for it against the oracle,
# with the fused max pool, channel splits, and prepared weights (bitwise the
# blob-staged ones)
LEAN_D2 = [40, 56, 46, 55, 48, 51, 54]


@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN_D2] + [(46, 3), (51, 4), (54, 2)])
def test_lean_dilation2(recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(19, 21, 36, 44), (16, 64, 32, 32), (8, 40, 20, 40)]
    if recipe not in V4:
        shapes += [(19, 21, 37, 45), (16, 64, 14, 14), (8, 13, 5, 7)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 9900 + 10 * recipe + si + ksplit
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 2, 2, pp.PP_F32)
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_F32)
        _say("lean dilation 2", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "runs as", plan)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        assert layer.prepare() is not None
        xd = torch.from_numpy(x).cuda()
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.conv3x3_pruned(*args, 1, 2, 2, True)
        bound = oconv.conv3x3_bound(*args, 1, 2, 2)
        for pool in (False, True):
            if pool and (h % 2 or w % 2 or (recipe == 54 and not ksplit)):
                continue
            y = pp.conv2d_fwd(layer, xd, relu=True, maxpool2=pool)
            yp = pp.conv2d_fwd(layer, xd, relu=True, maxpool2=pool, prepared=True)
            torch.cuda.synchronize()
            assert torch.equal(y, yp), f"dilation 2 {recipe}/{ksplit} pool={pool}: prepared weights differ"
            r, b = (oconv.maxpool2(ref), oconv.maxpool2(bound)) if pool else (ref, bound)
            check(y.cpu().numpy().astype(np.float64), r, b, "f32", f"lean d2 {recipe}/{ksplit} pool={pool}")


# stride 2 (pad 1, fp32): every tiling built for it against the oracle, with
# the fused max pool, channel splits, and prepared weights (bitwise the
# blob-staged ones); odd input sizes give ragged output tiles
LEAN_S2 = [45, 47, 49, 50, 52, 53, 54]


@pytest.mark.parametrize("recipe,ksplit", [(r, 0) for r in LEAN_S2] + [(49, 2), (53, 4), (54, 3)])
def test_lean_stride2(recipe, ksplit, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(recipe))
    if ksplit:
        monkeypatch.setenv("PP_KSPLIT", str(ksplit))
    shapes = [(19, 21, 36, 44), (16, 64, 64, 64), (8, 40, 20, 40)]
    if recipe not in V4:
        shapes += [(19, 21, 37, 45), (16, 64, 29, 14), (8, 13, 5, 7)]
    for si, (c_out, c_in, h, w) in enumerate(shapes):
        seed = 9950 + 10 * recipe + si + ksplit
        L = workloads.random_layer(seed, c_out, c_in, keep=0.5)
        x = workloads.random_input(seed, (2, c_in, h, w))
        layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 2, 1, 1, pp.PP_F32)
        plan = pp.conv2d_plan(layer.h_blob, 2, h, w, pp.PP_F32)
        _say("lean stride 2", recipe, ksplit, "seed", seed, (c_out, c_in, h, w), "runs as", plan)
        assert plan[0] == recipe and (not ksplit or plan[1] == ksplit)
        assert layer.prepare() is not None
        xd = torch.from_numpy(x).cuda()
        args = (x, L["w"], L["b"], L["pid"], L["conn"], L["lib"])
        ref = oconv.conv3x3_pruned(*args, 2, 1, 1, True)
        bound = oconv.conv3x3_bound(*args, 2, 1, 1)
        ho, wo = ref.shape[2], ref.shape[3]
        for pool in (False, True):
            if pool and (ho % 2 or wo % 2 or (recipe == 54 and not ksplit)):
                continue
            y = pp.conv2d_fwd(layer, xd, relu=True, maxpool2=pool)
            yp = pp.conv2d_fwd(layer, xd, relu=True, maxpool2=pool, prepared=True)
            torch.cuda.synchronize()
            assert torch.equal(y, yp), f"stride 2 {recipe}/{ksplit} pool={pool}: prepared weights differ"
            r, b = (oconv.maxpool2(ref), oconv.maxpool2(bound)) if pool else (ref, bound)
            check(y.cpu().numpy().astype(np.float64), r, b, "f32", f"lean s2 {recipe}/{ksplit} pool={pool}")


# the colourization network's dilated and strided layers at full size and
# full width (8 images, every output channel): the dilation-2 and stride-2
# lean paths as the network runs them, with prepared weights
@pytest.mark.parametrize("opi,hw", [(10, 32), (6, 64), (3, 128), (1, 256)])
def test_colourization_dilated_and_strided_layers_full_width(opi, hw):
    spec = workloads.net_spec(5)
    params = workloads.net_params(5)
    op, prm = spec["ops"][opi], params[opi]
    layer = pp.PackedLayer.from_weights(prm["w"], prm["b"], prm["pid"], prm["conn"], prm["lib"], op["stride"],
                                        op["pad"], op["dil"], pp.PP_F32)
    assert layer.prepare() is not None
    x = workloads.random_input(5000 + opi, (8, op["c_in"], hw, hw), 0.0, 1.0)
    plan = pp.conv2d_plan(layer.h_blob, 8, hw, hw, pp.PP_F32)
    _say("colourization layer", opi, op["c_in"], "->", op["c_out"], f"{hw}x{hw}", "stride", op["stride"], "dil",
         op["dil"], "plan", plan, "all filters")
    assert plan[0] in range(40, 60)
    y = pp.conv2d_fwd(layer, torch.from_numpy(x).cuda(), relu=op["relu"], prepared=True)
    torch.cuda.synchronize()
    args = (x, prm["w"], prm["b"], prm["pid"], prm["conn"], prm["lib"], op["stride"], op["pad"], op["dil"])
    check(y.cpu().numpy().astype(np.float64), oconv.conv3x3_pruned(*args, op["relu"]), oconv.conv3x3_bound(*args),
          "f32", f"colourization layer {opi} full width")
