"""Byte parity of the C++ packer with the oracle's packer, blob validation
on corrupted blobs and the packer's argument checks, run in a Python process
that has loaded the host-only packer library built with AddressSanitizer
and UndefinedBehaviorSanitizer (started by tests/test_sanitize.py with the
sanitizer runtime preloaded).  argv[1]: that library."""
import sys

import numpy as np

sys.path.insert(0, sys.argv[2])
import paper_2004_11250_amd as pp  # noqa: E402
import workloads  # noqa: E402
from oracle import ppk1  # noqa: E402

lib = pp.load_library(sys.argv[1])
assert not hasattr(lib, "pp_conv2d_fwd"), "expected the host-only library"

n = 0
# every 3x3 layer of the one-layer workload and of VGG-16 up to 256 -> 256,
# both storage types, then seeded random layers over several libraries
layers = []
for cfg in (1, 2):
    spec = workloads.net_spec(cfg)
    for i, op in enumerate(spec["ops"]):
        if op["op"] == "conv3" and op["c_in"] * op["c_out"] <= 256 * 256:
            layers.append((workloads.layer_params(cfg, i, op), op["stride"], op["pad"], op["dil"]))
rng = np.random.default_rng(5)
for k in range(40):
    lib_m = [workloads.CANON8, workloads.DENSE9, (0x010, 0x003, 0x1EF), (0x00F, 0x0B2, 0x1C8, 0x055)][k % 4]
    L = workloads.random_layer(900 + k, int(rng.integers(1, 40)), int(rng.integers(1, 40)), lib=lib_m,
                               keep=float(rng.uniform(0, 1)))
    layers.append((L, int(rng.integers(1, 3)), int(rng.integers(0, 3)), int(rng.integers(1, 3))))
for L, s, p, d in layers:
    for wd in (pp.PP_F32, pp.PP_BF16):
        blob = pp.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, wd)
        want = ppk1.pack(L["w"], L["b"], L["pid"], L["conn"], L["lib"], s, p, d, wd)
        assert blob.tobytes() == want, "packer bytes differ from the oracle's"
        info = pp.blob_info(blob)
        assert info["n_kept"] == int(L["conn"].sum())
        # truncated and corrupted copies: any status, no out-of-bounds read
        raw = blob.tobytes()
        for cut in (0, 1, 95, 96, len(raw) // 2, len(raw) - 1):
            try:
                pp.blob_info(np.frombuffer(raw[:cut], np.uint8).copy())
                raise AssertionError("truncated blob accepted")
            except pp.PPError:
                pass
        for t in range(16):
            c = np.frombuffer(raw, np.uint8).copy()
            idx = rng.integers(0, len(c), size=int(rng.integers(1, 6)))
            c[idx] ^= (1 << rng.integers(0, 8, size=len(idx))).astype(np.uint8)
            try:
                pp.blob_info(c)
            except pp.PPError:
                pass
        n += 1
# argument checks
L = layers[0][0]
bad = L["conn"].copy()
bad[0, 0] = 3
try:
    pp.pack(L["w"], L["b"], L["pid"], bad, L["lib"])
    raise AssertionError("conn value 3 accepted")
except pp.PPError:
    pass
print(f"asan packer parity: {n} blobs identical, corruption and argument checks passed")
