"""Host-side checks of the rule by which pp_net_fwd fuses the op after a
pruned conv into the conv's launch (paper_2004_11250_amd.fused_ops mirrors
the rule of the C runner, which the GPU tests then exercise)."""
import pytest

import workloads

pp = pytest.importorskip("paper_2004_11250_amd")


def _c3(src, dst, c_out=8, pad=1, dil=1, lib="canon8"):
    return dict(op="conv3", src=src, dst=dst, c_in=8, c_out=c_out, pad=pad, dil=dil, lib=lib)


def test_workload_fusions():
    want = {1: {}, 2: {i: "maxpool2" for i in (2, 5, 9, 13, 17)},
            3: {**{i: "add" for i in (5, 8, 11, 14, 17)}, 18: "up2", 20: "up2"},
            4: {**{3 * k + 3: "add" for k in range(16)}, 50: "pshuf2", 52: "pshuf2"}, 5: {}}
    for cfg, w in want.items():
        assert pp.fused_ops(workloads.net_spec(cfg)["ops"]) == w, cfg


def test_residual_add_rule():
    add = dict(op="add", src=2, src2=4, dst=3)
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, _c3(3, 1)]) == {3: "add"}
    # the skip operand is read later: no in-place accumulation
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, dict(op="add", src=3, src2=2, dst=1)]) == {}
    # the conv's output is read later
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4), add, dict(op="add", src=3, src2=4, dst=1)]) == {}
    # skip operand = the conv's input, or outside the workspace, or dst slot 1
    assert pp.fused_ops([_c3(0, 2), _c3(2, 4), dict(op="add", src=2, src2=4, dst=3), _c3(3, 1)]) == {}
    assert pp.fused_ops([_c3(0, 4), dict(op="add", src=0, src2=4, dst=3), _c3(3, 1)]) == {}
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4), dict(op="add", src=2, src2=4, dst=1)]) == {}
    # both operands are the conv's output
    assert pp.fused_ops([_c3(0, 2), _c3(2, 4), dict(op="add", src=4, src2=4, dst=3), _c3(3, 1)]) == {}
    # a layer the fused tilings do not take (pad != dilation, generic library)
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4, pad=2), add, _c3(3, 1)]) == {}
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), _c3(3, 4, lib="generic"), add, _c3(3, 1)]) == {}


def test_upsample_rule():
    up = dict(op="up2", src=2, dst=3)
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 4), _c3(4, 1)]) == {1: "up2"}
    # the conv writes the upsample's input slot: still fused (buffer swap)
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 2), _c3(2, 1)]) == {1: "up2"}
    # ... but then no op after the conv is fused
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 2), dict(op="maxpool2", src=2, dst=4), _c3(4, 1)]) == {1: "up2"}
    # otherwise both sides fuse
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 4), dict(op="maxpool2", src=4, dst=5), _c3(5, 1)]) == \
        {1: "up2", 3: "maxpool2"}
    # the upsample's output is read later, or is slot 1, or the conv is not a fusable layer
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 4), dict(op="add", src=4, src2=3, dst=1)]) == {}
    assert pp.fused_ops([_c3(0, 2), dict(op="up2", src=2, dst=1), _c3(1, 4), _c3(4, 5)]) == {}
    assert pp.fused_ops([_c3(0, 2), up, _c3(3, 4, pad=2), _c3(4, 1)]) == {}
    # the network input upsampled straight into the conv
    assert pp.fused_ops([dict(op="up2", src=0, dst=3), _c3(3, 1)]) == {0: "up2"}
    # the conv writes the upsample's input slot outside the workspace (slot 1)
    assert pp.fused_ops([_c3(0, 1), dict(op="up2", src=1, dst=3), _c3(3, 1)]) == {}


def test_pool_and_shuffle_rule():
    assert pp.fused_ops([_c3(0, 2), dict(op="pshuf2", src=2, dst=1)]) == {1: "pshuf2"}
    assert pp.fused_ops([_c3(0, 2, c_out=6), dict(op="pshuf2", src=2, dst=1)]) == {}   # c_out % 4
    assert pp.fused_ops([_c3(0, 2), dict(op="maxpool2", src=2, dst=0)]) == {}          # into the input x
    assert pp.fused_ops([_c3(0, 2), _c3(2, 3), dict(op="maxpool2", src=3, dst=2), _c3(2, 1)]) == {2: "maxpool2"}
    assert pp.fused_ops([_c3(0, 1), dict(op="maxpool2", src=1, dst=2), _c3(2, 1)]) == {}   # conv writes slot 1
    # a fused pair is not the start of another one
    assert pp.fused_ops([_c3(0, 2), dict(op="maxpool2", src=2, dst=3), dict(op="maxpool2", src=3, dst=1)]) == \
        {1: "maxpool2"}
