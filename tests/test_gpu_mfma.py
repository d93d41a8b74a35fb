"""GPU parity of the matrix-core form of a pruned bf16 layer (the zero-filled
dense contraction on the bf16 matrix cores, plan id 64) against the CPU
oracle, for every kind of pattern library, stride, dilation, padding, ragged
tiles and the fused epilogues; bitwise equality of its fused epilogues with
the op after the conv; and the planner's choice.

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
MFMA = 64

LIBS = {
    "canon8": np.array(workloads.CANON8, np.uint16),
    "lib6": np.array([0x00F, 0x0B2, 0x1C8, 0x055, 0x113, 0x0A9], np.uint16),     # other 4-tap patterns
    "mixed": np.array([0x010, 0x003, 0x007, 0x01F, 0x155, 0x1EF], np.uint16),    # 1, 2, 3, 5, 5, 8 taps
    "dense9": np.array([0x1FF], np.uint16),                                       # all taps
}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _say(*a):
    print(*a, flush=True)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda().to(torch.bfloat16)


def _host(y):
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64)


def _layer(seed, c_out, c_in, lib, keep, s, p, d):
    L = workloads.random_layer(seed, c_out, c_in, lib=LIBS[lib], keep=keep)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, pp.PP_BF16)
    return L, layer


def _oracle(L, x, s, p, d, relu, sel=slice(None)):
    w = obf16.round_f32(L["w"])
    args = (x, w[sel], L["b"][sel], L["pid"][sel], L["conn"][sel], L["lib"])
    return oconv.conv3x3_pruned(*args, s, p, d, relu), oconv.conv3x3_bound(*args, s, p, d)


CASES = [  # library, (stride, pad, dilation), (n, c_out, c_in, h, w), keep, relu
    ("canon8", (1, 1, 1), (1, 64, 64, 37, 45), 0.5, True),
    ("canon8", (1, 1, 1), (2, 40, 32, 19, 23), 0.5, False),     # c_out not a multiple of 8 or 32
    ("canon8", (2, 1, 1), (1, 136, 96, 33, 30), 0.4, True),     # two filter tiles of 128, the second ragged
    ("canon8", (1, 2, 2), (1, 72, 64, 26, 31), 0.6, True),
    ("canon8", (2, 2, 2), (2, 24, 32, 21, 17), 0.5, True),
    ("canon8", (1, 0, 1), (1, 8, 32, 12, 9), 0.7, False),       # no padding; 8 filters
    ("lib6", (1, 1, 1), (1, 100, 64, 29, 33), 0.5, True),
    ("lib6", (2, 0, 1), (2, 48, 32, 25, 26), 0.5, False),
    ("mixed", (1, 1, 1), (1, 64, 96, 22, 27), 0.5, True),       # 1..8 taps per pattern (odd counts padded in bf16)
    ("mixed", (1, 2, 2), (1, 33, 32, 18, 40), 0.3, False),
    ("dense9", (1, 1, 1), (2, 64, 32, 17, 19), 1.0, True),
    ("dense9", (2, 1, 1), (1, 130, 64, 31, 29), 1.0, False),
    # k steps of 64 (reductions 9 c_in >= 1152); with c_in an odd multiple
    # of 32 the last step is a half step
    ("canon8", (1, 1, 1), (1, 40, 160, 20, 22), 0.4, True),     # half step, 64-filter tiles
    ("canon8", (1, 1, 1), (1, 100, 128, 18, 21), 0.4, True),    # whole steps, 128-filter tiles
    ("canon8", (1, 2, 2), (2, 136, 224, 15, 17), 0.3, False),   # half step, 128-filter tiles, ragged second tile
    # more than 256 tiles: one wave group per tile
    ("canon8", (1, 1, 1), (1, 48, 160, 200, 172), 0.3, True),   # 269 tiles, long k with a half step
    ("canon8", (1, 1, 1), (1, 130, 64, 130, 128), 0.5, True),   # 260 tiles of 128 filters, short k
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_mfma_against_oracle(case, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    lib, (s, p, d), (n, c_out, c_in, h, w), keep, relu = CASES[case]
    seed = 1200 + case
    L, layer = _layer(seed, c_out, c_in, lib, keep, s, p, d)
    x = obf16.round_f32(workloads.random_input(seed, (n, c_in, h, w)))
    _say("mfma", lib, (s, p, d), (n, c_out, c_in, h, w), "keep", keep, "relu", relu, "seed", seed)
    assert pp.conv2d_recipe(layer.h_blob, n, h, w, pp.PP_BF16) == MFMA
    ho = (h + 2 * p - 2 * d - 1) // s + 1
    wo = (w + 2 * p - 2 * d - 1) // s + 1
    bm = 128 if c_out > 64 else 64
    tiles = -(-n * ho * wo // 128) * -(-c_out // bm)
    _say("  k step", 64 if 9 * c_in >= 1152 else 32, "half last step", (9 * c_in) % 64 == 32 and 9 * c_in >= 1152,
         "tiles", tiles, "wave groups per tile", 2 if tiles <= 256 else 1)
    y = _host(pp.conv2d_fwd(layer, _dev(x), relu=relu))
    ref, bound = _oracle(L, x, s, p, d, relu)
    check(y, ref, bound, "bf16", f"mfma {lib} {(s, p, d)} {(n, c_out, c_in, h, w)}")


def test_mfma_all_kernels_pruned(monkeypatch):
    # every kernel pruned: the expansion writes zeros everywhere, the output is act(bias)
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    L = workloads.random_layer(1290, 40, 64, keep=0.5)
    L["conn"][:] = 0
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    x = obf16.round_f32(workloads.random_input(1290, (1, 64, 11, 13)))
    _say("mfma all pruned")
    y = _host(pp.conv2d_fwd(layer, _dev(x), relu=True))
    want = obf16.round_f32(np.maximum(L["b"], 0.0)).astype(np.float64)[None, :, None, None]
    assert np.array_equal(y, np.broadcast_to(want, y.shape))


@pytest.mark.parametrize("mode", ["add", "pshuf2", "up2", "up2+add"])
def test_mfma_fused_epilogues(mode, monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    for (s, p, d), (n, c_out, c_in, h, w), relu in (((1, 1, 1), (2, 64, 32, 15, 22), True),
                                                    ((1, 2, 2), (1, 136, 64, 13, 17), False),
                                                    ((2, 1, 1), (1, 40, 32, 14, 18), True)):
        seed = 1300 + c_out + (7 if "add" in mode else 0)
        L, layer = _layer(seed, c_out, c_in, "canon8", 0.5, s, p, d)
        x = obf16.round_f32(workloads.random_input(seed, (n, c_in, h, w)))
        up = mode.startswith("up2")
        xin = np.ascontiguousarray(np.repeat(np.repeat(x, 2, axis=2), 2, axis=3)) if up else x
        hi, wi = xin.shape[2], xin.shape[3]
        ho, wo = pp.out_size(layer.h_blob, hi, wi)
        _say("mfma fused", mode, (s, p, d), (n, c_out, c_in, h, w), "relu", relu)
        assert pp.conv2d_recipe(layer.h_blob, n, hi, wi, pp.PP_BF16) == MFMA
        ref, bound = _oracle(L, xin, s, p, d, relu)
        xd = _dev(x)
        y_plain = pp.conv2d_fwd(layer, _dev(xin), relu=relu)   # the same plan, unfused
        if "add" in mode:
            r = obf16.round_f32(workloads.random_input(seed + 1, (n, c_out, ho, wo)))
            rd = _dev(r)
            yd = rd.clone()
            pp.conv2d_fwd(layer, xd, relu=relu, out=yd, accumulate=True, upsample2=up)
            ref, bound = ref + r.astype(np.float64), bound + np.abs(r.astype(np.float64))
            want = rd + y_plain
        elif mode == "pshuf2":
            yd = pp.conv2d_fwd(layer, xd, relu=relu, pixshuf2=True)
            ref, bound = oconv.pixel_shuffle2(ref), oconv.pixel_shuffle2(bound)
            want = torch.nn.functional.pixel_shuffle(y_plain, 2)
        else:
            yd = pp.conv2d_fwd(layer, xd, relu=relu, upsample2=True)
            want = y_plain
        check(_host(yd), ref, bound, "bf16", f"mfma fused {mode} {(s, p, d)} {(n, c_out, c_in, h, w)}")
        torch.cuda.synchronize()
        assert torch.equal(yd.cpu(), want.cpu()), f"fused {mode} differs from the op after the conv"


def test_mfma_not_planned_where_it_cannot_run(monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    L, layer = _layer(1400, 32, 24, "canon8", 0.5, 1, 1, 1)          # c_in not a multiple of 32
    assert pp.conv2d_recipe(layer.h_blob, 1, 20, 20, pp.PP_BF16) != MFMA
    L, layer = _layer(1401, 32, 32, "canon8", 0.5, 1, 1, 1)
    assert pp.conv2d_recipe(layer.h_blob, 1, 20, 20, pp.PP_BF16) == MFMA
    assert pp.conv2d_recipe(layer.h_blob, 1, 20, 20, pp.PP_BF16, with_workspace=False) != MFMA   # needs scratch
    lf = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_F32)
    assert pp.conv2d_recipe(lf.h_blob, 1, 20, 20, pp.PP_F32) != MFMA                          # bf16 only
    # a fused max pool takes the vector kernels
    x = obf16.round_f32(workloads.random_input(1401, (1, 32, 20, 20)))
    _say("mfma maxpool2 falls back")
    yd = pp.conv2d_fwd(layer, _dev(x), relu=True, maxpool2=True)
    ref, bound = _oracle(L, x, 1, 1, 1, True)
    check(_host(yd), oconv.maxpool2(ref), oconv.maxpool2(bound), "bf16", "maxpool2 fallback")
    # no workspace: the vector kernels
    _say("mfma without workspace falls back")
    y = pp.conv2d_fwd(layer, _dev(x), relu=True, workspace=None)
    check(_host(y), ref, bound, "bf16", "no-workspace fallback")


def test_planner_takes_mfma_for_large_bf16_layers():
    # the super-resolution body layer (64 -> 64 at 270 x 480) and a colourization layer: the matrix cores;
    # the 14 x 14 VGG-16 layer (a long reduction over few tiles): the vector kernels
    L, layer = _layer(1500, 64, 64, "canon8", 0.5, 1, 1, 1)
    assert pp.conv2d_recipe(layer.h_blob, 1, 270, 480, pp.PP_BF16) == MFMA
    L2, layer2 = _layer(1501, 256, 256, "canon8", 0.5, 1, 1, 1)
    assert pp.conv2d_recipe(layer2.h_blob, 8, 64, 64, pp.PP_BF16) == MFMA
    L3, layer3 = _layer(1502, 512, 512, "canon8", 1 / 3, 1, 1, 1)
    assert pp.conv2d_recipe(layer3.h_blob, 1, 14, 14, pp.PP_BF16) != MFMA
    # full-size super-resolution layer, sampled filters against the oracle
    x = obf16.round_f32(workloads.random_input(1500, (1, 64, 270, 480)))
    _say("mfma full-size 64->64 270x480")
    y = _host(pp.conv2d_fwd(layer, _dev(x), relu=True))
    sel = np.array([0, 17, 38, 63])
    ref, bound = _oracle(L, x, 1, 1, 1, True, sel)
    check(y[:, sel], ref, bound, "bf16", "mfma sr 270x480 sampled filters")


def test_mfma_full_colourization_layer():
    # a whole 512 -> 512 dilated layer of the colourization network (batch 8,
    # 32 x 32, bf16), the form and launch the network runs, every filter
    spec = workloads.net_spec(5)
    i = next(j for j, op in enumerate(spec["ops"]) if op["op"] == "conv3" and op["c_in"] == 512 and op["dil"] == 2)
    op = spec["ops"][i]
    L = workloads.layer_params(5, i, op)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], op["stride"], op["pad"],
                                        op["dil"], pp.PP_BF16)
    x = obf16.round_f32(workloads.random_input(1300 + i, (8, 512, 32, 32), 0.0, 1.0))
    _say("colourization layer", i, "512 -> 512 dilation 2, 8 x 32 x 32 bf16, all filters")
    assert pp.conv2d_recipe(layer.h_blob, 8, 32, 32, pp.PP_BF16) == MFMA
    y = _host(pp.conv2d_fwd(layer, _dev(x), relu=True))
    ref, bound = _oracle(L, x, op["stride"], op["pad"], op["dil"], True)
    check(y, ref, bound, "bf16", f"colourization layer {i}")


@pytest.mark.parametrize("case", [0, 2, 12, 15])
def test_prepared_weights_equal_per_call_expansion(case, monkeypatch):
    # the weights written once by pp_conv2d_prepare and passed with
    # PP_PREPARED give bitwise the output of the call that expands them
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    lib, (s, p, d), (n, c_out, c_in, h, w), keep, relu = CASES[case]
    seed = 1400 + case
    L, layer = _layer(seed, c_out, c_in, lib, keep, s, p, d)
    x = _dev(obf16.round_f32(workloads.random_input(seed, (n, c_in, h, w))))
    _say("prepared", lib, (s, p, d), (n, c_out, c_in, h, w), "seed", seed)
    assert pp.conv2d_recipe(layer.h_blob, n, h, w, pp.PP_BF16) == MFMA
    want = _host(pp.conv2d_fwd(layer, x, relu=relu))
    assert layer.prepare() is not None
    for _ in range(2):
        got = _host(pp.conv2d_fwd(layer, x, relu=relu, prepared=True))
        assert np.array_equal(got, want)


def test_prepared_weights_ignored_off_the_matrix_cores():
    # a layer the planner keeps on the vector ALUs: with PP_PREPARED the call
    # ignores the prepared weights (left untouched) and runs the plan a call
    # without the flag runs (its split scratch behind them)
    spec = workloads.net_spec(2)
    i = next(j for j, op in enumerate(spec["ops"]) if op["op"] == "conv3" and op["c_in"] == 512)
    op = spec["ops"][i]
    L = workloads.layer_params(2, i, op)
    layer = pp.PackedLayer.from_weights(L["w"], L["b"], L["pid"], L["conn"], L["lib"], 1, 1, 1, pp.PP_BF16)
    x = _dev(obf16.round_f32(workloads.random_input(1500, (1, 512, 14, 14), 0.0, 1.0)))
    _say("prepared off the matrix cores: VGG-16 layer", i, "bf16 14 x 14")
    assert pp.conv2d_recipe(layer.h_blob, 1, 14, 14, pp.PP_BF16) != MFMA
    buf = layer.prepare()
    before = buf.clone()
    want = _host(pp.conv2d_fwd(layer, x, relu=True))
    got = _host(pp.conv2d_fwd(layer, x, relu=True, prepared=True))
    assert np.array_equal(got, want)
    assert torch.equal(buf, before)
