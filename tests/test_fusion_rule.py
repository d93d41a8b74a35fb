"""Host-side checks of the rule by which pp_net_fwd fuses the op after a
pruned conv (or the x2 upsample before it) into the conv's launch, read from
the library's own plan (pp_net_plan), which the GPU tests then exercise."""
import numpy as np
import pytest

import workloads

pp = pytest.importorskip("paper_2004_11250_amd")

# a 3-pattern library that is neither the canonical 8 nor all-ones: the
# generic-mask kernel, which takes no fused op
GENERIC3 = (0x03A, 0x1B0, 0x145)


def _c3(src, dst, c_out=8, pad=1, dil=1, lib="canon8", stride=1):
    return dict(op="conv3", src=src, dst=dst, c_in=8, c_out=c_out, stride=stride, pad=pad, dil=dil, lib=lib)


def _params(ops):
    out = []
    for i, op in enumerate(ops):
        if op["op"] != "conv3":
            out.append({})
            continue
        lib = {"canon8": workloads.CANON8, "dense9": workloads.DENSE9, "generic": GENERIC3}[op["lib"]]
        out.append(workloads.random_layer(100 + i, op["c_out"], op["c_in"], lib=lib))
    return out


def fused(ops, hw=16):
    return pp.net_plan(ops, _params(ops), 1, 8, hw, hw)["fused"]


def test_workload_fusions():
    want = {1: {}, 2: {i: "maxpool2" for i in (2, 5, 9, 13, 17)},
            3: {**{i: "add" for i in (5, 8, 11, 14, 17)}, 18: "up2", 20: "up2"},
            4: {**{3 * k + 3: "add" for k in range(16)}, 50: "pshuf2", 52: "pshuf2"}, 5: {}}
    for cfg, w in want.items():
        spec = workloads.net_spec(cfg)
        n, c, h, wd = spec["batch"], spec["c"], spec["h"], spec["w"]
        for dtype in ("f32", "bf16"):
            plan = pp.net_plan(spec["ops"], workloads.net_params(cfg), n, c, h, wd, dtype)
            assert plan["fused"] == w, (cfg, dtype)
            # every taken op has a pruned conv beside it that carries its flag
            for i in w:
                j = i + 1 if w[i] == "up2" else i - 1
                assert spec["ops"][j]["op"] == "conv3" and plan["recipe"][j] >= 0
                assert plan["flags"][i] == pp.PP_NET_TAKEN
            assert all(r >= 0 for r, o in zip(plan["recipe"], spec["ops"]) if o["op"] == "conv3")


def test_residual_add_rule():
    add = dict(op="add", src=2, src2=4, dst=3)
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, _c3(3, 1)]) == {3: "add"}
    # the skip operand is read later: no in-place accumulation
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, dict(op="add", src=3, src2=2, dst=1)]) == {}
    # the conv's output is read later
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, dict(op="add", src=3, src2=4, dst=1)]) == {}
    # skip operand = the conv's input, or outside the workspace, or dst slot 1
    assert fused([_c3(0, 2), _c3(2, 4), dict(op="add", src=2, src2=4, dst=3), _c3(3, 1)]) == {}
    assert fused([_c3(0, 4), dict(op="add", src=0, src2=4, dst=3), _c3(3, 1)]) == {}
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4), dict(op="add", src=2, src2=4, dst=1)]) == {}
    # both operands are the conv's output
    assert fused([_c3(0, 2), _c3(2, 4), dict(op="add", src=4, src2=4, dst=3), _c3(3, 1)]) == {}
    # a layer the fused tilings do not take: padding other than the dilation
    # (the pad-0 conv shrinks the map by 2, the pad-2 conv grows it back)
    assert fused([_c3(0, 2), _c3(2, 3, pad=0), _c3(3, 4, pad=2), add, _c3(3, 1)]) == {}
    # ... or the generic-library kernel
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4, lib="generic"), add, _c3(3, 1)]) == {}
    # the dense (all-ones library) path fuses like the canonical one
    assert fused([_c3(0, 2), _c3(2, 3), _c3(3, 4, lib="dense9"), add, _c3(3, 1)]) == {3: "add"}


def test_upsample_rule():
    up = dict(op="up2", src=2, dst=3)
    assert fused([_c3(0, 2), up, _c3(3, 4), _c3(4, 1)]) == {1: "up2"}
    # the conv writes the upsample's input slot: still fused (buffer swap)
    assert fused([_c3(0, 2), up, _c3(3, 2), _c3(2, 1)]) == {1: "up2"}
    # ... but then no op after the conv is fused
    assert fused([_c3(0, 2), up, _c3(3, 2), dict(op="maxpool2", src=2, dst=4), _c3(4, 1)]) == {1: "up2"}
    # otherwise both sides fuse
    assert fused([_c3(0, 2), up, _c3(3, 4), dict(op="maxpool2", src=4, dst=5), _c3(5, 1)]) == \
        {1: "up2", 3: "maxpool2"}
    # the upsample's output is read later, or is slot 1, or the conv is not a fusable layer
    assert fused([_c3(0, 2), up, _c3(3, 4), dict(op="add", src=4, src2=3, dst=1)]) == {}
    assert fused([_c3(0, 2), dict(op="up2", src=2, dst=1), _c3(1, 4), _c3(4, 5)]) == {}
    assert fused([_c3(0, 2), up, _c3(3, 4, lib="generic"), _c3(4, 1)]) == {}
    # the network input upsampled straight into the conv
    assert fused([dict(op="up2", src=0, dst=3), _c3(3, 1)]) == {0: "up2"}
    # the conv writes the upsample's input slot outside the workspace (slot 1;
    # a stride-2 conv brings the map back to the size slot 1 had), against
    # the same list in the workspace
    assert fused([_c3(0, 2), dict(op="up2", src=2, dst=3), _c3(3, 2, stride=2),
                  dict(op="maxpool2", src=2, dst=1)]) == {1: "up2"}
    assert fused([_c3(0, 1), dict(op="up2", src=1, dst=3), _c3(3, 1, stride=2)]) == {}
    # a pool after it that would write the upsample's input slot 1
    assert fused([_c3(0, 1), dict(op="up2", src=1, dst=3), _c3(3, 4), dict(op="maxpool2", src=4, dst=1)]) == \
        {1: "up2"}


def test_pool_and_shuffle_rule():
    assert fused([_c3(0, 2), dict(op="pshuf2", src=2, dst=1)]) == {1: "pshuf2"}
    assert fused([_c3(0, 2), _c3(2, 3), dict(op="maxpool2", src=3, dst=2), _c3(2, 1)]) == {2: "maxpool2"}
    # a conv that writes slot 1 keeps its own store (the pool is its own op);
    # the shuffle after the next conv brings slot 1 back to its first shape
    c32 = dict(_c3(2, 3), c_out=32)
    assert fused([_c3(0, 1), dict(op="maxpool2", src=1, dst=2), c32, dict(op="pshuf2", src=3, dst=1)]) == \
        {3: "pshuf2"}
    # a fused pair is not the start of another one
    assert fused([_c3(0, 2), dict(op="maxpool2", src=2, dst=3), dict(op="maxpool2", src=3, dst=1)]) == \
        {1: "maxpool2"}
    # a ragged map (odd size: the pool drops the last row and column) still fuses
    assert fused([_c3(0, 2), dict(op="maxpool2", src=2, dst=1)], hw=15) == {1: "maxpool2"}


def test_plan_rejects_what_the_runner_rejects():
    # a pixel shuffle of 6 channels is no valid network: the plan query fails
    # as pp_net_workspace and pp_net_fwd would
    with pytest.raises(pp.PPError):
        fused([_c3(0, 2, c_out=6), dict(op="pshuf2", src=2, dst=1)])
    with pytest.raises(pp.PPError):
        fused([_c3(0, 2), dict(op="maxpool2", src=2, dst=0)])       # the input x is read-only
    ops = [_c3(0, 2), dict(op="maxpool2", src=2, dst=1)]
    with pytest.raises(pp.PPError):
        pp.net_plan(ops, _params(ops), 1, 7, 16, 16)     # channels do not match the blob


def test_plan_matches_workspace_query_shape():
    # the plan query is host-only: no device pointer is needed, and it agrees
    # with pp_net_workspace about which convs run (every conv has a recipe)
    spec = workloads.net_spec(1)
    n, c, h, w = spec["batch"], spec["c"], spec["h"], spec["w"]
    plan = pp.net_plan(spec["ops"], workloads.net_params(1), n, c, h, w)
    assert plan["flags"] == [0] and plan["recipe"][0] >= 0
    assert np.all(np.array(plan["recipe"]) < 64)
