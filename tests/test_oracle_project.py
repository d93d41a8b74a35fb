"""Pins of the oracle's pruning projections and batch-norm folding against
what the mathematics fixes (not against themselves): least-squares
projections onto each pattern subspace (numpy.linalg.lstsq), order
statistics (numpy.sort / partition), an einsum of the column energies, and
a float64 torch conv + batch norm for the folding."""
import numpy as np
import pytest

import workloads
from oracle import project as opj

CANON8 = np.array(workloads.CANON8, dtype=np.uint16)


def _taps(mask):
    return [t for t in range(9) if (int(mask) >> t) & 1]


def test_pattern_projection_is_the_nearest_pattern_kernel():
    rng = np.random.default_rng(11)
    w = rng.normal(size=(6, 7, 3, 3)).astype(np.float32)
    pid, kept = opj.project_patterns(w, CANON8)
    for o in range(6):
        for c in range(7):
            k = w[o, c].reshape(9).astype(np.float64)
            dist = []
            for m in CANON8:
                basis = np.eye(9)[:, _taps(m)]                       # the pattern's subspace
                coef = np.linalg.lstsq(basis, k, rcond=None)[0]
                dist.append(np.sum((k - basis @ coef) ** 2))
            dist = np.array(dist)
            assert dist[pid[o, c]] <= dist.min() * (1 + 1e-12) + 1e-300
            # the kept energy is what the projection keeps: |k|^2 - distance
            assert kept[o, c] == pytest.approx(np.sum(k * k) - dist[pid[o, c]], rel=1e-12)


def test_pattern_projection_exact_cases():
    w = np.zeros((1, 10, 3, 3), np.float32)
    for q in range(8):                     # supported on exactly one pattern's taps
        for t in _taps(CANON8[q]):
            w[0, q].reshape(9)[t] = 1.0 + t
    w[0, 8] = 1.0                          # all taps equal: every pattern ties -> pattern 0
    # channel 9 all zero: every pattern ties at 0 -> pattern 0
    pid, kept = opj.project_patterns(w, CANON8)
    assert list(pid[0, :8]) == list(range(8))
    assert pid[0, 8] == 0 and pid[0, 9] == 0 and kept[0, 9] == 0.0
    assert kept[0, 8] == 4.0


def test_connectivity_keeps_the_largest_kernels():
    rng = np.random.default_rng(12)
    e = rng.random((9, 13))
    for n in (0, 1, 50, 117):
        conn = opj.project_connectivity(e, n)
        assert conn.sum() == n
        kept, dropped = e[conn == 1], e[conn == 0]
        if n and len(dropped):
            assert kept.min() >= dropped.max()
        assert np.sum(kept) == pytest.approx(np.sort(e.reshape(-1))[::-1][:n].sum(), rel=1e-12)
    # ties go to the lower flat index
    t = np.ones((2, 3))
    assert opj.project_connectivity(t, 4).reshape(-1).tolist() == [1, 1, 1, 1, 0, 0]
    with pytest.raises(ValueError):
        opj.project_connectivity(t, 7)


def test_column_projection():
    rng = np.random.default_rng(13)
    w = rng.normal(size=(5, 4, 3, 3)).astype(np.float32)
    w64 = w.astype(np.float64).reshape(5, 4, 9)
    np.testing.assert_allclose(opj.column_energy(w), np.einsum("oct,oct->ct", w64, w64), rtol=1e-13)
    for n in (0, 7, 20, 36):
        m = opj.project_columns(w, n)
        bits = ((m[:, None].astype(np.int64) >> np.arange(9)) & 1).astype(bool)
        assert bits.sum() == n
        e = np.einsum("oct,oct->ct", w64, w64)
        if 0 < n < 36:
            assert e[bits].min() >= e[~bits].max()
    # a column library reproduces the masks per channel, the same for every filter
    m = np.array([0x1FF, 0, 0x012, 0x1FF], np.uint16)
    lib, pid, conn = opj.column_library(m, 3)
    assert lib.tolist() == [0x012, 0x1FF]
    assert conn.tolist() == [[1, 0, 1, 1]] * 3
    assert [int(lib[p]) for p, k in zip(pid[0], conn[0]) if k] == [0x1FF, 0x012, 0x1FF]


def test_fold_bn_matches_conv_then_batch_norm():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(14)
    c_out, c_in = 6, 4
    w = rng.normal(size=(c_out, c_in, 3, 3)).astype(np.float32)
    b = rng.normal(size=c_out).astype(np.float32)
    gamma, beta = rng.normal(size=c_out).astype(np.float32), rng.normal(size=c_out).astype(np.float32)
    mean, var = rng.normal(size=c_out).astype(np.float32), rng.random(c_out).astype(np.float32) + 0.1
    x = torch.from_numpy(rng.normal(size=(2, c_in, 9, 8))).double()
    ref = F.batch_norm(F.conv2d(x, torch.from_numpy(w).double(), torch.from_numpy(b).double(), padding=1),
                       torch.from_numpy(mean).double(), torch.from_numpy(var).double(),
                       torch.from_numpy(gamma).double(), torch.from_numpy(beta).double(), False, 0.0, 1e-5)
    wf, bf = opj.fold_bn(w, b, gamma, beta, mean, var, 1e-5)
    got = F.conv2d(x, torch.from_numpy(wf).double(), torch.from_numpy(bf).double(), padding=1)
    scale = ref.abs().max().item()
    assert (got - ref).abs().max().item() <= 1e-6 * scale
    # no bias: treated as zero
    wf0, bf0 = opj.fold_bn(w, None, gamma, beta, mean, var, 1e-5)
    np.testing.assert_array_equal(wf0, wf)
    s = gamma.astype(np.float64) / np.sqrt(var.astype(np.float64) + np.float64(np.float32(1e-5)))
    np.testing.assert_allclose(bf0, (beta - mean * s).astype(np.float32), rtol=1e-6)
