"""GPU parity of pp_net_fwd on the five evaluated networks at full size.

Teacher-forced check: every op's GPU output is compared with the oracle run
on that op's GPU input (sampled output channels for the large layers), so
errors do not compound.  The op outputs come from pp_net_fwd itself, run on
the op-list prefix that ends with that op.  A max pool that pp_net_fwd fuses
into the pruned conv before it is checked as that conv followed by the pool.
pp_net_fwd must also equal the chain of single-layer calls bitwise."""
import numpy as np
import pytest

import workloads
from oracle import bf16 as obf16
from oracle import conv as oconv
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


def _say(*a):
    print(*a, flush=True)


def _input(cfg, dtype):
    x = workloads.net_input(cfg)
    if dtype == "bf16":
        x = obf16.round_f32(x)
    t = torch.from_numpy(x).cuda()
    return x, (t.to(torch.bfloat16) if dtype == "bf16" else t)


def _np(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy()


def _sampled(op, prm, n_keep, seed):
    """Restrict an op to a subset of its output channels (oracle cost)."""
    if op["op"] not in ("conv3", "conv", "deconv") or op["c_out"] <= n_keep:
        return op, prm, slice(None)
    sel = np.sort(np.random.default_rng(seed).choice(op["c_out"], size=n_keep, replace=False))
    p = dict(prm)
    if op["op"] == "deconv":
        p["w"] = prm["w"][:, sel]
    else:
        p["w"] = prm["w"][sel]
        for k in ("pid", "conn"):
            if k in prm:
                p[k] = prm[k][sel]
    p["b"] = prm["b"][sel]
    return dict(op, c_out=len(sel)), p, sel


def _fused_pool(ops, i):
    """pp_net_fwd runs op i (a 2 x 2 max pool) inside the pruned conv before
    it: the pool reads that conv's output, which no later op reads before
    rewriting it, and the conv's padding equals its dilation (the fused
    tilings)."""
    if i < 1 or ops[i]["op"] != "maxpool2" or ops[i - 1]["op"] != "conv3":
        return False
    cv, mp = ops[i - 1], ops[i]
    if mp["src"] != cv["dst"] or cv["dst"] == 1 or (mp["dst"] == cv["src"] and cv["src"] < 2) or \
            cv["pad"] != cv["dil"]:
        return False
    for o in ops[i + 1:]:
        if o["src"] == cv["dst"] or (o["op"] == "add" and o.get("src2") == cv["dst"]):
            return False
        if o["dst"] == cv["dst"]:
            return True
    return True


def teacher_forced(cfg, dtype, n_keep=6):
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    net = pp.Net(spec["ops"], params, dtype)
    x_np, x = _input(cfg, dtype)
    slots = {0: x_np}
    worst = 0.0
    for i, (op, prm) in enumerate(zip(spec["ops"], params)):
        _say(f"cfg {cfg} {dtype} op {i} {op['op']} c_in={op.get('c_in')} c_out={op.get('c_out')}")
        # pp_net_fwd on the prefix ending at op i, with op i writing slot 1
        sub = pp.Net.__new__(pp.Net)
        sub.__dict__.update(net.__dict__)
        arr = (pp.NetOp * (i + 1))()
        for j in range(i + 1):
            arr[j] = net.ops[j]
        arr[i].dst = 1
        sub.ops, sub.n_ops, sub._ws = arr, i + 1, None
        y = _np(sub.forward(x))
        if _fused_pool(spec["ops"][:i + 1], i):
            # conv + pool in one launch: the oracle conv on the conv's GPU input,
            # pooled (max is 1-Lipschitz, so the pooled bound is the pooled S)
            cop, cprm = spec["ops"][i - 1], params[i - 1]
            sop, sprm, sel = _sampled(cop, cprm, n_keep, 1000 * cfg + i)
            cref, cbound = onet.run_op(sop, sprm, slots[cop["src"]], None, dtype)
            worst = max(worst, check(y[:, sel], oconv.maxpool2(cref), oconv.maxpool2(cbound), dtype,
                                     f"cfg {cfg} op {i} (conv3 + maxpool2)"))
            slots[op["dst"]] = y
            continue
        src = slots[op["src"]]
        src2 = slots.get(op.get("src2")) if "src2" in op else None
        sop, sprm, sel = _sampled(op, prm, n_keep, 1000 * cfg + i)
        ref, bound = onet.run_op(sop, sprm, src, src2, dtype)
        yi = y[:, sel]
        if bound is None:
            # data movement only: must be exact
            assert np.array_equal(yi, onet.store(ref, dtype)), f"cfg {cfg} op {i}"
        else:
            worst = max(worst, check(yi, ref, bound, dtype, f"cfg {cfg} op {i} ({op['op']})"))
        slots[op["dst"]] = y
    return worst


@pytest.mark.parametrize("cfg,dtype", [(1, "f32"), (2, "f32"), (3, "f32"), (4, "f32"), (4, "bf16"), (5, "f32"),
                                       (5, "bf16")])
def test_network_teacher_forced(cfg, dtype):
    worst = teacher_forced(cfg, dtype)
    _say(f"cfg {cfg} {dtype}: worst |err|/S = {worst:.3e}")


def test_vgg16_net_equals_chained_layer_calls():
    spec = workloads.net_spec(2)
    params = workloads.net_params(2)
    net = pp.Net(spec["ops"], params, "f32")
    _, x = _input(2, "f32")
    _say("vgg16 pp_net_fwd vs chained pp_conv2d_fwd (pool fused where the net fuses it) + maxpool")
    y_net = _np(net.forward(x))
    ops = spec["ops"]
    cur = x
    li = 0
    for i, (op, prm) in enumerate(zip(ops, params)):
        if op["op"] == "conv3":
            fuse = i + 1 < len(ops) and _fused_pool(ops, i + 1)
            cur = pp.conv2d_fwd(net.pruned[li], cur, relu=op["relu"], maxpool2=fuse)
            li += 1
        elif _fused_pool(ops, i):
            continue
        else:
            one = pp.Net([dict(op, src=0, dst=1)], [prm], "f32")
            cur = one.forward(cur)
    assert np.array_equal(y_net, _np(cur))


def test_vgg16_net_graph_replays():
    # pp_net_fwd captured as a HIP graph: every replay, with eager work and
    # synchronisation between replays and a new input each time, equals the
    # eager pp_net_fwd on that input bitwise
    spec = workloads.net_spec(2)
    params = workloads.net_params(2)
    net = pp.Net(spec["ops"], params, "f32")
    _, x0 = _input(2, "f32")
    nbytes, oshape = net.plan(*x0.shape)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    xg = x0.clone()
    yg = torch.empty(oshape, dtype=torch.float32, device="cuda")
    _say("vgg16 graph capture")
    graph = net.capture(xg, yg, ws)
    for rep in range(4):
        _say("vgg16 graph replay", rep)
        xg.copy_(x0 * (1.0 + 0.25 * rep))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _np(yg)
        ref = _np(net.forward(xg.clone()))   # eager, its own workspace and output
        assert np.array_equal(got, ref), f"replay {rep} differs from the eager run"


def test_vgg16_end_to_end_vs_oracle_chain():
    # informational bound: the all-oracle chain vs the GPU chain, errors compound
    spec = workloads.net_spec(2)
    params = workloads.net_params(2)
    net = pp.Net(spec["ops"], params, "f32")
    x_np, x = _input(2, "f32")
    y = _np(net.forward(x)).astype(np.float64)
    ref = onet.run_net(spec, params, x_np, "f32").astype(np.float64)
    rel = np.max(np.abs(y - ref)) / np.max(np.abs(ref))
    _say(f"vgg16 end-to-end max|err|/max|ref| = {rel:.3e}")
    assert rel < 1e-4
