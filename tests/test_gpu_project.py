"""The pack-side helpers end to end on the GPU: dense weights projected onto
pattern + connectivity structure (or column structure, which runs through
the generic-library kernel), a batch norm folded in, packed, and run by
pp_conv2d_fwd; against the oracle conv of the same projected, folded
weights."""
import numpy as np
import pytest

import workloads
from oracle import conv as oconv
from oracle import project as opj
from tests.tolerance import check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pp = pytest.importorskip("paper_2004_11250_amd")
CANON8 = np.array(workloads.CANON8, dtype=np.uint16)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    pp.load_library()
    yield
    torch.cuda.synchronize()


def _bn(rng, c_out):
    return (rng.normal(1.0, 0.2, c_out).astype(np.float32), rng.normal(0, 0.1, c_out).astype(np.float32),
            rng.normal(0, 0.1, c_out).astype(np.float32), rng.random(c_out).astype(np.float32) + 0.5)


@pytest.mark.parametrize("c_out,c_in,h,w,keep", [(64, 64, 28, 28, 1 / 3), (40, 24, 17, 23, 0.5)])
def test_pattern_connectivity_pipeline(c_out, c_in, h, w, keep):
    rng = np.random.default_rng(c_out + c_in)
    wd = rng.normal(0, np.sqrt(2 / (9 * c_in)), (c_out, c_in, 3, 3)).astype(np.float32)
    gamma, beta, mean, var = _bn(rng, c_out)
    wf, bf = pp.fold_bn(wd, None, gamma, beta, mean, var, 1e-5)
    pid, e = pp.project_patterns(wf, CANON8)
    conn = pp.project_connectivity(e, int(round(keep * c_out * c_in)))
    layer = pp.PackedLayer.from_weights(wf, bf, pid, conn, CANON8)
    x = workloads.random_input(3, (1, c_in, h, w))
    print("pattern pipeline", c_out, c_in, h, w, flush=True)
    y = pp.conv2d_fwd(layer, torch.from_numpy(x).cuda(), relu=True)
    torch.cuda.synchronize()
    owf, obf = opj.fold_bn(wd, None, gamma, beta, mean, var, 1e-5)
    opid, oe = opj.project_patterns(owf, CANON8)
    oconn = opj.project_connectivity(oe, int(round(keep * c_out * c_in)))
    args = (x, owf, obf, opid, oconn, CANON8)
    check(y.cpu().numpy(), oconv.conv3x3_pruned(*args, 1, 1, 1, True), oconv.conv3x3_bound(*args, 1, 1, 1), "f32",
          "pattern + connectivity pipeline")


def test_column_pruning_pipeline():
    rng = np.random.default_rng(77)
    c_out, c_in, h, w = 32, 16, 20, 18
    wd = rng.normal(0, 0.2, (c_out, c_in, 3, 3)).astype(np.float32)
    b = rng.normal(0, 0.1, c_out).astype(np.float32)
    m = pp.project_columns(wd, 9 * c_in // 3)
    lib, pid, conn = pp.column_library(m, c_out)
    layer = pp.PackedLayer.from_weights(wd, b, pid, conn, lib)
    x = workloads.random_input(4, (2, c_in, h, w))
    print("column pipeline", len(lib), "masks", flush=True)
    y = pp.conv2d_fwd(layer, torch.from_numpy(x).cuda(), relu=False)
    torch.cuda.synchronize()
    olib, opid, oconn = opj.column_library(opj.project_columns(wd, 9 * c_in // 3), c_out)
    args = (x, wd, b, opid, oconn, olib)
    check(y.cpu().numpy(), oconv.conv3x3_pruned(*args, 1, 1, 1, False), oconv.conv3x3_bound(*args, 1, 1, 1), "f32",
          "column pipeline")
