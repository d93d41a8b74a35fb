"""The C++ packer (pp_pack) against the oracle's independent packer: the two
must emit identical bytes, and both must match the hand-derived golden
example.  Runs on the CPU (host code only)."""
import numpy as np
import pytest

import workloads
from oracle import ppk1
from tests.golden_io import ppk1_small

pp = pytest.importorskip("paper_2004_11250_amd")


@pytest.fixture(scope="module", autouse=True)
def _lib():
    pp.load_library()


def _small_layer():
    w = np.zeros((4, 3, 9), np.float32)
    for o in range(4):
        for c in range(3):
            for t in range(9):
                w[o, c, t] = 100 * o + 10 * c + t
    pid = np.array([[0, 4, 4], [2, 2, 7], [1, 0, 3], [4, 4, 0]], np.uint8)
    conn = np.array([[1, 0, 1], [1, 1, 1], [0, 0, 0], [1, 1, 0]], np.uint8)
    return w.reshape(4, 3, 3, 3), np.array([0.5, 1.5, 2.5, 3.5], np.float32), pid, conn


def test_golden_small_bytes():
    w, b, pid, conn = _small_layer()
    lib = np.array(workloads.CANON8, np.uint16)
    blob = pp.pack(w, b, pid, conn, lib)
    assert blob.tobytes() == ppk1.pack(w, b, pid, conn, lib)
    d = ppk1.parse(blob.tobytes())
    g = ppk1_small()
    assert list(d["perm"]) == g["perm"] and list(d["codes"].ravel()) == g["codes"]
    assert list(d["woff"]) == g["woff"] and list(d["w"]) == g["w"] and list(d["bias"]) == g["bias"]
    assert len(blob) == g["total_bytes"][0]
    info = pp.blob_info(blob)
    assert info["n_kept"] == 7 and info["n_wt"] == 28 and info["c_out"] == 4 and info["c_in"] == 3


@pytest.mark.parametrize("wd", [0, 1])
def test_random_layers_bytes_match_oracle(wd):
    rng = np.random.default_rng(100 + wd)
    for trial in range(60):
        c_out, c_in = int(rng.integers(1, 40)), int(rng.integers(1, 20))
        n_p = int(rng.integers(1, 12))
        lib = rng.integers(1, 512, size=n_p).astype(np.uint16)
        keep = float(rng.uniform(0, 1))
        L = workloads.random_layer(1000 + trial, c_out, c_in, lib=lib, keep=keep)
        if trial % 7 == 0:
            L["w"][..., 1, 1] = 0.0    # planted zeros inside kept patterns are stored
        s, d = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        p = int(rng.integers(0, 3))
        a = pp.pack(L["w"], L["b"], L["pid"], L["conn"], lib, s, p, d, wd)
        o = ppk1.pack(L["w"], L["b"], L["pid"], L["conn"], lib, s, p, d, wd)
        assert a.tobytes() == o, trial


# every pruned (and all-ones) 3x3 layer of the five workloads, in both weight
# dtypes, byte for byte: the largest blobs (512 x 512 layers: the most slot
# groups and the largest weight offsets) included
@pytest.mark.parametrize("wd", [0, 1])
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_layers_bytes_match_oracle(cfg, wd):
    spec = workloads.net_spec(cfg)
    for i, op in enumerate(spec["ops"]):
        if op["op"] != "conv3":
            continue
        prm = workloads.layer_params(cfg, i, op)
        args = (prm["w"], prm["b"], prm["pid"], prm["conn"], prm["lib"], op["stride"], op["pad"], op["dil"], wd)
        assert pp.pack(*args).tobytes() == ppk1.pack(*args), (cfg, i, wd)


def test_bf16_rounding_ties_match_oracle():
    # weights sitting exactly on bf16 midpoints (ties to even) and just off them
    base = np.array([1.0, 1.5, -2.0, 3.25], np.float32).view(np.uint32)
    vals = np.concatenate([(base | 0x8000), (base | 0x8001), (base | 0x7FFF), base + 0x18000]).view(np.float32)
    w = np.resize(vals, 2 * 2 * 9).reshape(2, 2, 3, 3).astype(np.float32)
    lib = np.array([0x1FF, 0x03A], np.uint16)
    pid = np.array([[0, 1], [1, 0]], np.uint8)
    conn = np.ones((2, 2), np.uint8)
    assert pp.pack(w, None, pid, conn, lib, wdtype=1).tobytes() == ppk1.pack(w, None, pid, conn, lib, wdtype=1)


def test_size_query_and_small_buffer():
    import ctypes
    w, b, pid, conn = _small_layer()
    lib = pp.load_library()
    masks = np.array(workloads.CANON8, np.uint16)
    d = pp.LayerDesc(4, 3, 1, 1, 1, 0)
    n = ctypes.c_size_t(0)
    args = (ctypes.byref(d), w.ctypes.data, b.ctypes.data, pid.ctypes.data, conn.ctypes.data, masks.ctypes.data, 8)
    assert lib.pp_pack(*args, None, ctypes.byref(n)) == pp.PP_OK and n.value == 576
    buf = np.zeros(100, np.uint8)
    n2 = ctypes.c_size_t(100)
    assert lib.pp_pack(*args, buf.ctypes.data, ctypes.byref(n2)) == pp.PP_ESIZE and n2.value == 576
    assert np.all(buf == 0)
