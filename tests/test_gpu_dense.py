"""GPU parity of the dense layers of the evaluated networks (k x k conv,
stride 1; 4 x 4 stride-2 transposed conv), which run as implicit GEMMs on
the matrix cores (small dense convs on the vector kernels: the tiled 9 x 9
one and the per-row one), against the oracle: ragged filter counts and pixel counts
(partial tiles in both GEMM dimensions), K not a multiple of the K step,
several images, paddings, ReLU on and off, fp32 and bf16."""
import numpy as np
import pytest

from oracle import bf16 as obf16
from oracle import net as onet
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


def _run(op, prm, x, dtype):
    xs = obf16.round_f32(x) if dtype == "bf16" else x
    net = pp.Net([dict(op, src=0, dst=1)], [prm], dtype)
    xd = torch.from_numpy(xs).cuda()
    xd = xd.to(torch.bfloat16) if dtype == "bf16" else xd
    y = net.forward(xd.contiguous())
    torch.cuda.synchronize()
    ref, bound = onet.run_op(op, prm, xs, None, dtype)
    return y.float().cpu().numpy(), ref, bound


# the first five run on the matrix cores (16+ filters, reduction >= 256), the
# others on the vector kernel
CONV_CASES = [  # (k, pad, c_in, c_out, n, h, w, relu)
    (1, 0, 256, 313, 1, 9, 11, False),
    (1, 0, 300, 45, 2, 13, 17, True),
    (3, 1, 40, 48, 2, 10, 23, True),
    (9, 4, 4, 20, 1, 15, 22, False),
    (9, 3, 5, 70, 2, 11, 12, True),
    (1, 0, 19, 45, 2, 13, 17, True),
    (3, 1, 7, 33, 2, 10, 23, True),
    (3, 0, 5, 64, 1, 12, 9, False),
    (9, 4, 3, 32, 1, 21, 30, True),
    (9, 4, 32, 3, 1, 19, 26, False),
    (9, 2, 2, 70, 2, 11, 12, True),
    # 9 x 9, pad 4, width a multiple of 4: the tiled 9 x 9 kernel (F filters
    # per wave, channels split S ways inside the workgroup)
    (9, 4, 32, 3, 1, 19, 28, False),     # F 3, S 8 (two tiles per workgroup, the last one dead)
    (9, 4, 3, 32, 2, 21, 36, True),      # F 4, eight filter groups, S 1
    (9, 4, 4, 4, 1, 9, 8, True),         # F 4, S 4 (one channel each), a dead tile in the last workgroup
    (9, 4, 10, 5, 2, 13, 260, False),    # ragged second column tile, S 8 with empty splits, 3 dead filters
    (9, 4, 7, 10, 1, 5, 4, True),        # image shorter than the kernel, S 4, a half-dead last filter group
    (9, 4, 50, 2, 1, 6, 12, False),      # the largest reduction whose weights fit LDS at F 3
    (9, 4, 51, 3, 1, 6, 12, True),       # one channel more: the per-row vector kernel
    (9, 4, 37, 8, 1, 7, 16, False),      # the largest reduction whose weights fit LDS at F 4
    (9, 4, 38, 8, 1, 7, 16, True),       # one channel more: the per-row vector kernel
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", CONV_CASES)
def test_dense_conv(case, dtype):
    k, pad, c_in, c_out, n, h, w, relu = case
    rng = np.random.default_rng(40 + k + c_out)
    std = np.sqrt(2.0 / (c_in * k * k))
    prm = dict(w=rng.normal(0, std, (c_out, c_in, k, k)).astype(np.float32),
               b=rng.normal(0, 0.1, c_out).astype(np.float32))
    op = dict(op="conv", c_in=c_in, c_out=c_out, k=k, stride=1, pad=pad, dil=1, relu=relu)
    x = rng.uniform(-1, 1, (n, c_in, h, w)).astype(np.float32)
    print("dense conv", case, dtype, flush=True)
    y, ref, bound = _run(op, prm, x, dtype)
    check(y, ref, bound, dtype, f"conv {case} {dtype}")


DECONV_CASES = [  # (c_in, c_out, n, h, w, relu)
    (16, 24, 2, 7, 9, True),
    (33, 70, 1, 5, 13, False),
    (512, 256, 1, 8, 8, True),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", DECONV_CASES)
def test_transposed_conv(case, dtype):
    c_in, c_out, n, h, w, relu = case
    rng = np.random.default_rng(90 + c_out)
    std = np.sqrt(2.0 / (c_in * 16))
    prm = dict(w=rng.normal(0, std, (c_in, c_out, 4, 4)).astype(np.float32),
               b=rng.normal(0, 0.1, c_out).astype(np.float32))
    op = dict(op="deconv", c_in=c_in, c_out=c_out, k=4, stride=2, pad=1, relu=relu)
    x = rng.uniform(-1, 1, (n, c_in, h, w)).astype(np.float32)
    print("transposed conv", case, dtype, flush=True)
    y, ref, bound = _run(op, prm, x, dtype)
    assert y.shape == (n, c_out, 2 * h, 2 * w)
    check(y, ref, bound, dtype, f"deconv {case} {dtype}")


# large layers take the 128 x 128 tiles (128+ filters, a reduction of 512+,
# 512+ tiles), here with a partial last K step: checked on a sample of
# output channels (the oracle on the matching slices of the weights)
BIG_CASES = [  # (op, c_in, c_out, n, h, w)
    ("conv", 600, 200, 2, 128, 128),
    ("deconv", 130, 160, 2, 64, 64),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", BIG_CASES)
def test_large_dense_layers_sampled(case, dtype):
    kind, c_in, c_out, n, h, w = case
    rng = np.random.default_rng(c_out + c_in)
    k = 1 if kind == "conv" else 4
    shape = (c_out, c_in, k, k) if kind == "conv" else (c_in, c_out, 4, 4)
    prm = dict(w=rng.normal(0, np.sqrt(2.0 / (c_in * k * k)), shape).astype(np.float32),
               b=rng.normal(0, 0.1, c_out).astype(np.float32))
    op = dict(op=kind, c_in=c_in, c_out=c_out, k=k, stride=1 if kind == "conv" else 2, pad=0 if k == 1 else 1,
              dil=1, relu=True)
    x = rng.uniform(-1, 1, (n, c_in, h, w)).astype(np.float32)
    xs = obf16.round_f32(x) if dtype == "bf16" else x
    print("large", case, dtype, flush=True)
    net = pp.Net([dict(op, src=0, dst=1)], [prm], dtype)
    xd = torch.from_numpy(xs).cuda()
    y = net.forward((xd.to(torch.bfloat16) if dtype == "bf16" else xd).contiguous())
    torch.cuda.synchronize()
    sel = np.sort(rng.choice(c_out, size=5, replace=False))
    sub = dict(prm, b=prm["b"][sel], w=prm["w"][sel] if kind == "conv" else prm["w"][:, sel])
    ref, bound = onet.run_op(dict(op, c_out=len(sel)), sub, xs, None, dtype)
    check(y[:, sel].float().cpu().numpy(), ref, bound, dtype, f"large {case} {dtype}")


# the style network's 9 x 9 layers at full size (512 x 512), every output of
# sampled rows (the oracle on the 9 input rows each needs)
STYLE9 = [(3, 32, True), (32, 3, False)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", STYLE9)
def test_style_9x9_layers_full_size_sampled(case, dtype):
    c_in, c_out, relu = case
    h = w = 512
    rng = np.random.default_rng(500 + c_out)
    prm = dict(w=rng.normal(0, np.sqrt(2.0 / (c_in * 81)), (c_out, c_in, 9, 9)).astype(np.float32),
               b=rng.normal(0, 0.1, c_out).astype(np.float32))
    op = dict(op="conv", c_in=c_in, c_out=c_out, k=9, stride=1, pad=4, dil=1, relu=relu)
    x = rng.uniform(0, 1, (1, c_in, h, w)).astype(np.float32)
    xs = obf16.round_f32(x) if dtype == "bf16" else x
    print("style 9x9 full size", case, dtype, flush=True)
    net = pp.Net([dict(op, src=0, dst=1)], [prm], dtype)
    xd = torch.from_numpy(xs).cuda()
    y = net.forward((xd.to(torch.bfloat16) if dtype == "bf16" else xd).contiguous())
    torch.cuda.synchronize()
    y = y.float().cpu().numpy()
    for r in (0, 3, 4, 255, 508, 511):
        lo, hi = max(r - 4, 0), min(r + 5, h)
        ref, bound = onet.run_op(op, prm, xs[:, :, lo:hi], None, dtype)
        check(y[:, :, r:r + 1], ref[:, :, r - lo:r - lo + 1], bound[:, :, r - lo:r - lo + 1], dtype,
              f"style 9x9 {case} {dtype} row {r}")
