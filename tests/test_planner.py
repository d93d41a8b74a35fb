"""Planner choices that need no GPU (pp_conv2d_recipe is host-only): where
the bf16 matrix-core form (plan id 64) is taken and where it cannot be."""
import numpy as np
import pytest

import workloads

pp = pytest.importorskip("paper_2004_11250_amd")
MFMA = 64


def _blob(seed, c_out, c_in, dt, keep=0.5, s=1, p=1, d=1, lib=None):
    lib = np.array(workloads.CANON8 if lib is None else lib, np.uint16)
    L = workloads.random_layer(seed, c_out, c_in, lib=lib, keep=keep)
    return pp.pack(L["w"], L["b"], L["pid"], L["conn"], lib, s, p, d, dt)


@pytest.fixture(autouse=True)
def _no_forced_plan(monkeypatch):
    monkeypatch.delenv("PP_RECIPE", raising=False)
    monkeypatch.delenv("PP_KSPLIT", raising=False)


def test_large_bf16_layers_take_the_matrix_cores():
    assert pp.conv2d_recipe(_blob(1, 64, 64, pp.PP_BF16), 1, 270, 480, pp.PP_BF16) == MFMA      # super-resolution body
    assert pp.conv2d_recipe(_blob(2, 512, 512, pp.PP_BF16), 8, 32, 32, pp.PP_BF16) == MFMA     # colourization
    # the style network's 128 -> 128 at 128 x 128: the lean kernel (25.6 us
    # with prepared weights against 29.3 on the matrix cores)
    assert pp.conv2d_recipe(_blob(3, 128, 128, pp.PP_BF16), 1, 128, 128, pp.PP_BF16) == 46
    # any library: the form reads the blob's own masks
    other = [0x00F, 0x0B2, 0x1C8, 0x055, 0x113, 0x0A9]
    assert pp.conv2d_recipe(_blob(4, 64, 64, pp.PP_BF16, lib=other), 1, 270, 480, pp.PP_BF16) == MFMA


def test_small_or_ineligible_layers_stay_on_the_vector_kernels():
    b = _blob(5, 512, 512, pp.PP_BF16, keep=1 / 3)
    assert pp.conv2d_recipe(b, 1, 14, 14, pp.PP_BF16) != MFMA           # few tiles, long reduction
    assert pp.conv2d_recipe(b, 1, 28, 28, pp.PP_BF16) != MFMA
    assert pp.conv2d_recipe(_blob(6, 3, 64, pp.PP_BF16), 1, 1080, 1920, pp.PP_BF16) != MFMA   # 3 filters
    sr = _blob(7, 64, 64, pp.PP_BF16)
    assert pp.conv2d_recipe(sr, 1, 270, 480, pp.PP_BF16, with_workspace=False) != MFMA        # needs scratch
    assert pp.conv2d_recipe(_blob(8, 64, 48, pp.PP_BF16), 1, 270, 480, pp.PP_BF16) != MFMA    # c_in % 32
    assert pp.conv2d_recipe(_blob(9, 64, 64, pp.PP_F32), 1, 270, 480, pp.PP_F32) != MFMA       # fp32


def test_forced_matrix_core_plan(monkeypatch):
    monkeypatch.setenv("PP_RECIPE", str(MFMA))
    assert pp.conv2d_recipe(_blob(10, 40, 32, pp.PP_BF16), 2, 19, 23, pp.PP_BF16) == MFMA
    assert pp.conv2d_recipe(_blob(11, 40, 24, pp.PP_BF16), 2, 19, 23, pp.PP_BF16) != MFMA   # cannot run: ignored


def test_workspace_covers_the_matrix_core_form():
    b = _blob(12, 64, 64, pp.PP_BF16)
    ws = pp.conv2d_workspace(b, 1, 270, 480, pp.PP_BF16)
    assert ws >= 64 * 9 * 64 * 2 + 64 * 4   # the expanded weights and the bias
