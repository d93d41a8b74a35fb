"""GPU parity of the dense layers of the evaluated networks (k x k conv,
stride 1; 4 x 4 stride-2 transposed conv), which run as implicit GEMMs on
the matrix cores (small dense convs on a vector kernel), against the oracle: ragged filter counts and pixel counts
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
