"""The library's pruning projections and batch-norm folding (host C code
behind the C-ABI) against the oracle: bitwise, since both take their integer
decisions on the same double sums and fold in the same double arithmetic.
Layer shapes of the evaluated networks, ties, edge cases and errors."""
import numpy as np
import pytest

import workloads
from oracle import project as opj

pp = pytest.importorskip("paper_2004_11250_amd")
CANON8 = np.array(workloads.CANON8, dtype=np.uint16)


@pytest.fixture(scope="module", autouse=True)
def lib():
    return pp.load_library()


@pytest.mark.parametrize("shape", [(1, 1), (8, 3), (64, 64), (512, 256), (33, 70)])
def test_pattern_and_connectivity_projection(shape):
    c_out, c_in = shape
    rng = np.random.default_rng(c_out * 1000 + c_in)
    w = rng.normal(size=(c_out, c_in, 3, 3)).astype(np.float32)
    w[0, 0] = 0.0                                           # all-tie kernel
    if c_in > 1:
        w[0, 1] = 1.0
    pid, e = pp.project_patterns(w, CANON8)
    opid, oe = opj.project_patterns(w, CANON8)
    assert np.array_equal(pid, opid)
    assert np.array_equal(e, oe)
    for keep in (0.0, 1.0 / 3.0, 0.5, 1.0):
        n = int(round(keep * c_out * c_in))
        assert np.array_equal(pp.project_connectivity(e, n), opj.project_connectivity(oe, n))


def test_projection_with_other_libraries():
    rng = np.random.default_rng(5)
    w = rng.normal(size=(9, 11, 3, 3)).astype(np.float32)
    for lib in ([0x1FF], [0x010, 0x1FF, 0x0BA], list(range(1, 256))):
        pid, e = pp.project_patterns(w, lib)
        opid, oe = opj.project_patterns(w, lib)
        assert np.array_equal(pid, opid) and np.array_equal(e, oe)


def test_connectivity_ties():
    e = np.zeros((3, 4))
    e[1, 2] = 1.0
    conn = pp.project_connectivity(e, 3)
    assert conn.reshape(-1).tolist() == [1, 1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 0]


@pytest.mark.parametrize("shape,keep", [((32, 64), 0.5), ((64, 32), 0.25), ((5, 3), 1.0), ((7, 2), 0.0)])
def test_column_projection_and_library(shape, keep):
    c_out, c_in = shape
    rng = np.random.default_rng(c_out + 7 * c_in)
    w = rng.normal(size=(c_out, c_in, 3, 3)).astype(np.float32)
    n = int(round(keep * 9 * c_in))
    m = pp.project_columns(w, n)
    assert np.array_equal(m, opj.project_columns(w, n))
    lib, pid, conn = pp.column_library(m, c_out)
    olib, opid, oconn = opj.column_library(m, c_out)
    assert np.array_equal(lib, olib) and np.array_equal(conn, oconn)
    assert np.array_equal(pid[conn == 1], opid[oconn == 1])


def test_column_library_limits():
    m = np.arange(1, 300, dtype=np.uint16)                 # 299 distinct masks
    with pytest.raises(pp.PPError):
        pp.column_library(m, 2)
    with pytest.raises(pp.PPError):
        pp.column_library(np.array([0x200], np.uint16), 2)  # not a 9-bit mask
    lib, pid, conn = pp.column_library(np.zeros(4, np.uint16), 3)
    assert lib.tolist() == [1] and conn.sum() == 0


@pytest.mark.parametrize("k", [3, 9, 1])
def test_fold_bn(k):
    rng = np.random.default_rng(k)
    c_out, c_in = 24, 5
    w = rng.normal(size=(c_out, c_in, k, k)).astype(np.float32)
    b = rng.normal(size=c_out).astype(np.float32)
    g, bt, mu = (rng.normal(size=c_out).astype(np.float32) for _ in range(3))
    v = rng.random(c_out).astype(np.float32)
    v[0] = 0.0                                              # var 0: eps keeps it finite
    for bias in (b, None):
        wf, bf = pp.fold_bn(w, bias, g, bt, mu, v, 1e-3)
        owf, obf = opj.fold_bn(w, bias, g, bt, mu, v, 1e-3)
        assert np.array_equal(wf, owf) and np.array_equal(bf, obf)


def test_helpers_reject_bad_arguments():
    w = np.zeros((2, 2, 3, 3), np.float32)
    with pytest.raises(pp.PPError):
        pp.project_patterns(w, [0])                         # empty mask
    with pytest.raises(pp.PPError):
        pp.project_patterns(w, [0x200])
    with pytest.raises(pp.PPError):
        pp.project_connectivity(np.zeros((2, 2)), 5)
    with pytest.raises(pp.PPError):
        pp.project_connectivity(np.full((2, 2), np.nan), 1)
    with pytest.raises(pp.PPError):
        pp.project_columns(w, 19)
    with pytest.raises(pp.PPError):
        pp.fold_bn(w, None, np.ones(2), np.zeros(2), np.zeros(2), -np.ones(2), 1e-5)
