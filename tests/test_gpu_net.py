"""GPU parity of pp_net_fwd on the five evaluated networks at full size.

Teacher-forced check: every op's GPU output is compared with the oracle run
on that op's GPU input (sampled output channels for the large layers), so
errors do not compound.  The op outputs come from pp_net_fwd itself, run on
the op-list prefix that ends with that op.  An op that pp_net_fwd fuses into
the pruned conv before it (max pool, residual add, pixel shuffle) is checked
as that conv followed by the op; its prefix keeps the real slots (so the
fusion, with its buffer renaming, happens as in the whole network) and ends
with a nearest x2 upsample of the op's output into slot 1, which is exact
data movement.  pp_net_fwd must also equal the chain of single-layer calls
bitwise."""
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


def _sampled(op, prm, n_keep, seed, group=1):
    """Restrict an op to a subset of its output channels (oracle cost); with
    group g whole aligned groups of g channels (n_keep groups)."""
    if op["op"] not in ("conv3", "conv", "deconv") or op["c_out"] <= n_keep * group:
        return op, prm, slice(None)
    g = np.sort(np.random.default_rng(seed).choice(op["c_out"] // group, size=n_keep, replace=False))
    sel = (group * g[:, None] + np.arange(group)[None, :]).reshape(-1)
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


def _prefix_net(net, i, readout):
    """pp_net_fwd on ops 0..i: op i writes slot 1, or (readout) keeps its slot
    and an x2 upsample copies that slot into slot 1."""
    sub = pp.Net.__new__(pp.Net)
    sub.__dict__.update(net.__dict__)
    arr = (pp.NetOp * (i + 1 + readout))()
    for j in range(i + 1):
        arr[j] = net.ops[j]
    if readout:
        arr[i + 1].kind = pp.OP_UPSAMPLE2
        arr[i + 1].src, arr[i + 1].dst = net.ops[i].dst, 1
    else:
        arr[i].dst = 1
    sub.ops, sub.n_ops, sub._ws = arr, i + 1 + readout, None
    return sub


def teacher_forced(cfg, dtype, n_keep=6):
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    net = pp.Net(spec["ops"], params, dtype)
    fused = net.launch_plan(spec["batch"], spec["c"], spec["h"], spec["w"])["fused"]
    x_np, x = _input(cfg, dtype)
    slots = {0: x_np}
    worst = 0.0
    for i, (op, prm) in enumerate(zip(spec["ops"], params)):
        _say(f"cfg {cfg} {dtype} op {i} {op['op']} c_in={op.get('c_in')} c_out={op.get('c_out')}"
             f"{' (fused into op %d)' % (i - 1) if i in fused else ''}")
        if i in fused and fused[i] != "up2":
            # the fused pair in one launch: the oracle conv on the conv's GPU
            # input, then the op (max and x -> x + r are 1-Lipschitz, the
            # shuffle moves data: the pair's bound is the op applied to S,
            # plus |r| for the add)
            if op["dst"] == 1:
                y = _np(_prefix_net(net, i, False).forward(x))   # already the output slot
            else:
                y = _np(_prefix_net(net, i, True).forward(x))[:, :, ::2, ::2]
            cop, cprm = spec["ops"][i - 1], params[i - 1]
            group = 4 if op["op"] == "pshuf2" else 1
            sop, sprm, sel = _sampled(cop, cprm, n_keep, 1000 * cfg + i, group)
            cref, cbound = onet.run_op(sop, sprm, slots[cop["src"]], None, dtype)
            if op["op"] == "maxpool2":
                ref, bound, got = oconv.maxpool2(cref), oconv.maxpool2(cbound), y[:, sel]
            elif op["op"] == "pshuf2":
                ref, bound = oconv.pixel_shuffle2(cref), oconv.pixel_shuffle2(cbound)
                got = y if isinstance(sel, slice) else y[:, sel[::4] // 4]
            else:
                r = slots[op["src2"] if op["src"] == cop["dst"] else op["src"]][:, sel].astype(np.float64)
                ref, bound, got = cref + r, cbound + np.abs(r), y[:, sel]
            worst = max(worst, check(got, ref, bound, dtype, f"cfg {cfg} op {i} (conv3 + {op['op']})"))
            slots[op["dst"]] = y
            continue
        y = _np(_prefix_net(net, i, False).forward(x))
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


@pytest.mark.parametrize("cfg,dtype", [(1, "f32"), (2, "f32"), (2, "bf16"), (3, "f32"), (4, "f32"), (4, "bf16"),
                                       (5, "f32"), (5, "bf16")])
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
    fused = net.launch_plan(spec["batch"], spec["c"], spec["h"], spec["w"])["fused"]
    cur = x
    li = 0
    for i, (op, prm) in enumerate(zip(ops, params)):
        if op["op"] == "conv3":
            cur = pp.conv2d_fwd(net.pruned[li], cur, relu=op["relu"], maxpool2=fused.get(i + 1) == "maxpool2")
            li += 1
        elif i in fused:
            continue
        else:
            one = pp.Net([dict(op, src=0, dst=1)], [prm], "f32")
            cur = one.forward(cur)
    assert np.array_equal(y_net, _np(cur))


@pytest.mark.parametrize("cfg,dtype", [(3, "f32"), (3, "bf16"), (4, "f32"), (4, "bf16")])
def test_net_fused_equals_unfused(cfg, dtype):
    # the fused residual adds and pixel shuffles give bitwise the output of
    # the same network run op by op (each op its own pp_net_fwd), whose
    # convs are the same plans with the plain store
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    ops = spec["ops"]
    fused = pp.net_plan(ops, params, spec["batch"], spec["c"], spec["h"], spec["w"], dtype)["fused"]
    assert any(k == "add" for k in fused.values()), "the network has fusable residual adds"
    if cfg == 4:
        assert sum(k == "pshuf2" for k in fused.values()) == 2
    if cfg == 3:
        assert sum(k == "up2" for k in fused.values()) == 2
    net = pp.Net(ops, params, dtype)
    _, x = _input(cfg, dtype)
    _say(f"cfg {cfg} {dtype}: pp_net_fwd ({len(fused)} fused ops) vs op-by-op")
    y_net = _np(net.forward(x))
    slots = {0: x}
    li = 0
    for i, (op, prm) in enumerate(zip(ops, params)):
        if op["op"] == "conv3":
            slots[op["dst"]] = pp.conv2d_fwd(net.pruned[li], slots[op["src"]], relu=op["relu"])
            li += 1
        elif op["op"] == "add":
            slots[op["dst"]] = slots[op["src"]] + slots[op["src2"]]
        else:
            one = pp.Net([dict(op, src=0, dst=1)], [prm], dtype)
            slots[op["dst"]] = one.forward(slots[op["src"]].contiguous())
    assert np.array_equal(y_net, _np(slots[1]))


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


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_prepared_fp32_net_is_bitwise_the_same(cfg):
    # fp32 networks: the lean kernel's prepared weights (pp_net_op.d_w, read
    # by scalar loads) give bitwise the frame that stages them from the blob
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    _, x = _input(cfg, "f32")
    _say(f"cfg {cfg} f32: prepared vs blob-staged weights")
    a = pp.Net(spec["ops"], params, "f32", prepare=False)
    b = pp.Net(spec["ops"], params, "f32", prepare=True)
    assert sum(L.prepared is not None for L in b.pruned) > 0
    ya = _np(a.forward(x))
    for _ in range(2):
        assert np.array_equal(_np(b.forward(x)), ya)


@pytest.mark.parametrize("cfg", [4, 5])
def test_prepared_net_equals_per_call_expansion(cfg):
    # bf16 networks: prepared matrix-core weights (pp_net_op.d_w) give
    # bitwise the frame that expands them on every call
    spec = workloads.net_spec(cfg)
    params = workloads.net_params(cfg)
    _, x = _input(cfg, "bf16")
    _say(f"cfg {cfg} bf16: prepared vs per-call expansion")
    a = pp.Net(spec["ops"], params, "bf16", prepare=False)
    b = pp.Net(spec["ops"], params, "bf16", prepare=True)
    assert sum(L.prepared is not None for L in b.pruned) > 0
    ya = _np(a.forward(x))
    for _ in range(2):
        assert np.array_equal(_np(b.forward(x)), ya)


def test_trace_ranges_change_nothing(tmp_path):
    # PP_TRACE (read once per process): the same VGG-16 frame, bitwise, in a
    # child process that traces every op
    import os
    import subprocess
    import sys
    spec = workloads.net_spec(2)
    params = workloads.net_params(2)
    net = pp.Net(spec["ops"], params, "f32")
    _, x = _input(2, "f32")
    want = _np(net.forward(x))
    out = tmp_path / "traced.npy"
    code = ("import numpy as np, torch, workloads, paper_2004_11250_amd as pp\n"
            "spec = workloads.net_spec(2); params = workloads.net_params(2)\n"
            "net = pp.Net(spec['ops'], params, 'f32')\n"
            "x = torch.from_numpy(workloads.net_input(2)).cuda()\n"
            f"np.save({str(out)!r}, net.forward(x).cpu().numpy())\n")
    env = dict(os.environ, PP_TRACE="1")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    _say("traced VGG-16 frame in a child process")
    subprocess.run([sys.executable, "-c", code], env=env, cwd=root, check=True, timeout=300)
    assert np.array_equal(np.load(out), want)
