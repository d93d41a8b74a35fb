"""Run-time specialised kernels (pp_jit_library) for a layer's own library
of 4-tap patterns: against the oracle, and bitwise against the same layer
packed with the canonical library when the library is a reordering of it
(the same taps in the same order per kernel, so the same arithmetic)."""
import numpy as np
import pytest

import workloads
from oracle import bf16 as obf16
from oracle import conv as oconv
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")
CANON8 = np.array(workloads.CANON8, np.uint16)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _dev(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def test_reordered_canonical_library_bitwise(monkeypatch):
    order = np.array([7, 2, 5, 0, 3, 6, 1, 4])
    lib = CANON8[order]                                   # pattern i of lib is canonical pattern order[i]
    for (c_out, c_in, h, w, s, p, d) in ((40, 24, 33, 45, 1, 1, 1), (24, 512, 14, 14, 1, 1, 1),
                                         (16, 20, 29, 30, 2, 1, 1), (20, 12, 27, 31, 1, 2, 2)):
        L = workloads.random_layer(c_out + c_in, c_out, c_in, lib=lib, keep=0.5)
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], lib, s, p, d)
        cblob = pp.pack(L["w"], L["b"], order[L["pid"]].astype(np.uint8), L["conn"], CANON8, s, p, d)
        x = workloads.random_input(c_in, (1, c_in, h, w))
        print("reordered library", (c_out, c_in, h, w, s, p, d), flush=True)
        pp.jit_library(blob, 1, h, w)
        # run-time kernels exist for the wave-pipeline tilings (20-39); the
        # canonical library runs the same tiling when forced to it
        rec = pp.conv2d_recipe(blob, 1, h, w)
        assert 20 <= rec < 40
        layer, clayer = pp.PackedLayer(blob), pp.PackedLayer(cblob)
        y = pp.conv2d_fwd(layer, _dev(x, "f32"), relu=True)
        monkeypatch.setenv("PP_RECIPE", str(rec))
        assert pp.conv2d_recipe(cblob, 1, h, w) == rec
        yc = pp.conv2d_fwd(clayer, _dev(x, "f32"), relu=True)
        monkeypatch.delenv("PP_RECIPE")
        torch.cuda.synchronize()
        assert torch.equal(y, yc)


LIB6 = np.array([0x00F, 0x0B2, 0x1C8, 0x055, 0x113, 0x0A9], np.uint16)   # 4 taps each, not the canonical ones


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_other_four_tap_library(dtype):
    assert all(bin(int(m)).count("1") == 4 for m in LIB6)
    wd = pp.PP_BF16 if dtype == "bf16" else pp.PP_F32
    for (c_out, c_in, h, w, s, p, d, n) in ((33, 17, 26, 35, 1, 1, 1, 2), (64, 256, 14, 14, 1, 1, 1, 1),
                                            (24, 16, 31, 28, 2, 1, 1, 1), (16, 9, 25, 22, 1, 2, 2, 1)):
        L = workloads.random_layer(c_out * 7 + c_in, c_out, c_in, lib=LIB6, keep=0.6)
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], LIB6, s, p, d, wd)
        x = workloads.random_input(c_out, (n, c_in, h, w))
        w_or = L["w"]
        if dtype == "bf16":
            x, w_or = obf16.round_f32(x), obf16.round_f32(L["w"])
        print("library of 6", dtype, (c_out, c_in, h, w, s, p, d, n), flush=True)
        pp.jit_library(blob, n, h, w, wd)
        assert pp.conv2d_recipe(blob, n, h, w, wd) >= 20
        y = pp.conv2d_fwd(pp.PackedLayer(blob), _dev(x, dtype), relu=False)
        args = (x, w_or, L["b"], L["pid"], L["conn"], LIB6)
        check(y.float().cpu().numpy(), oconv.conv3x3_pruned(*args, s, p, d, False),
              oconv.conv3x3_bound(*args, s, p, d), dtype, f"library of 6 {dtype}")


def test_jit_rejects_other_libraries():
    L = workloads.random_layer(3, 8, 4)
    for lib in (CANON8, np.array([0x007, 0x0B2], np.uint16), np.array(list(CANON8) + [0x0F0], np.uint16)):
        pid = np.minimum(L["pid"], len(lib) - 1).astype(np.uint8)
        blob = pp.pack(L["w"], L["b"], pid, L["conn"], lib)
        with pytest.raises(pp.PPError):
            pp.jit_library(blob, 1, 16, 16)
    blob = pp.pack(L["w"], L["b"], np.minimum(L["pid"], 3).astype(np.uint8), L["conn"], LIB6[:4], 1, 0, 1)  # pad != dil
    with pytest.raises(pp.PPError):
        pp.jit_library(blob, 1, 16, 16)
