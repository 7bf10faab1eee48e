"""The ResNet-50 step program, planned on the host (no kernels run): the
network has ResNet-50's layer count and parameter count (Section 5.1), every
buffer a call reads is written earlier in the step, and no buffer is written
twice."""

import numpy as np

import paper_1911_07384_amd as F
import pytest

from paper_1911_07384_amd.network import ResNet50


@pytest.fixture(scope="module")
def net():
    return ResNet50(n=1, image=224, device="cpu")


def test_layer_and_parameter_counts(net):
    kinds = [o.kind for o in net.fwd]
    # 53 convolutions + the classifier; 53 BNs, each fused with the conv before
    # it except the stem's, fused with the max pool after it
    assert kinds.count("conv_fwd") + kinds.count("conv_bn_fwd") == 54
    assert kinds.count("bn_maxpool_fwd") + kinds.count("conv_bn_fwd") == 53
    assert kinds.count("conv_bn_fwd") == 52 and kinds.count("conv_fwd") == 2
    assert kinds.count("bn_fwd") == kinds.count("maxpool_fwd") == 0
    unfused = ResNet50(n=1, image=64, device="cpu", fuse_bn_stats=False)
    uk = [o.kind for o in unfused.fwd]
    assert uk.count("conv_fwd") == 54 and uk.count("bn_fwd") == 53
    conv_w = sum(int(np.prod(net.buffers[c["name"]].shape)) for c in net.convs if c["name"] != "fc")
    assert conv_w == 23_454_912
    assert net.n_weights == 23_454_912 + 2_048_000 + 1000
    assert net.n_bn == 53_120
    assert net.n_weights + net.n_bn == 25_557_032  # ResNet-50's parameter count


def test_conv_flops_at_batch_128(net):
    # FLOPs scale with the batch; at 128 the forward convolutions + classifier
    # are 1.0468 TFLOP (the classifier is 2*128*2048*1000)
    f = 128 * net.conv_flops()
    assert abs(f - 1.0468e12) < 0.0005e12
    assert net.step_flops() == 3 * net.conv_flops() - 2 * 112 * 112 * 64 * 3 * 49


OUTPUTS = {"conv_fwd": ["y"], "conv_bn_fwd": ["y", "z", "stats", "mask"], "conv_dgrad": ["dx"],
           "conv_dgrad_add": ["dx"],
           "conv_wgrad": ["dw"], "bn_fwd": ["y", "stats", "mask"],
           "bn_bwd": ["dx", "dgamma", "dbeta", "dres"], "maxpool_fwd": ["y", "idx"],
           "maxpool_bwd": ["dx"], "avgpool_fwd": ["y"], "avgpool_bwd": ["dx"],
           "bn_maxpool_fwd": ["stats", "y", "idx"],
           "softmax_ce": ["loss", "dz", "dbias"], "dgrad_filter": ["wf"]}


def test_dataflow(net):
    # every buffer a call reads is an input, a parameter, or written earlier in
    # the step; every output is written exactly once
    params = {c["name"] for c in net.convs} | {"fc.bias"}
    for name, _ in net._bnspecs:
        params |= {name + ".gamma", name + ".beta"}
    written = {"image", "labels"} | params
    seen = set()
    # (the data-gradient filters are rearranged from the weights before the
    # forward, on the side stream)
    for op in net.prep + net.fwd + net.bwd:
        outs = [k for k in OUTPUTS[op.kind] if op.a.get(k) is not None]
        # ("mask_of" names a BN, whose kept mask the call reads)
        reads = [v for k, v in op.a.items()
                 if isinstance(v, str) and k not in outs and k != "mask_of"]
        if op.kind in ("bn_fwd", "bn_bwd", "conv_bn_fwd", "bn_maxpool_fwd"):
            reads += [op.name + ".gamma", op.name + ".beta"]
        for v in reads:
            assert v in net.buffers and v in written, (op.name, op.kind, v)
        for k in outs:
            v = op.a[k]
            assert v in net.buffers and v not in seen, (op.name, k, v)
            seen.add(v)
            written.add(v)
    # every weight and BN parameter receives a gradient
    grads = {op.a["dw"] for op in net.bwd if op.kind == "conv_wgrad"}
    assert grads == {"d:" + c["name"] for c in net.convs}
    bn_grads = {op.a["dgamma"] for op in net.bwd if op.kind == "bn_bwd"}
    assert bn_grads == {name + ".dgamma" for name, _ in net._bnspecs}
    # every data gradient reads a rearranged filter made from its own weights
    prep = {op.a["wf"]: op.a["w"] for op in net.prep}
    for op in net.bwd:
        if op.kind in ("conv_dgrad", "conv_dgrad_add"):
            assert prep[op.a["wf"]] == op.a["w"] == op.name


def test_block_last_bns_keep_their_relu_mask(net):
    # the 16 BNs whose ReLU follows the shortcut write the mask in the forward
    # and their backward reads it instead of the shortcut
    fwd = {o.name: o for o in net.fwd if o.kind in ("bn_fwd", "conv_bn_fwd", "bn_maxpool_fwd")}
    kept = {n for n, o in fwd.items() if o.a.get("mask") is not None}
    assert kept == {n for n, o in fwd.items() if o.a.get("res") is not None}
    assert len(kept) == 16 and all(n.endswith(".bn3") for n in kept)
    for o in net.bwd:
        if o.kind == "bn_bwd":
            assert o.a["mask"] == fwd[o.a["mask_of"]].a.get("mask")
            # no block-last BN writes its shortcut gradient: the downsampling
            # shortcut's BN takes the block-last BN's gradient under its mask
            assert o.a["dres"] is None
            if o.name.endswith(".bnd"):
                assert o.a["mask_of"] == o.name[:-4] + ".bn3" and o.a["desc"].relu == 1
            else:
                assert o.a["mask_of"] == o.name
    # the identity blocks' input gradients add the block-last BN's incoming
    # gradient under its mask
    adds = {o.name: o for o in net.bwd if o.kind == "conv_dgrad_add"}
    assert len(adds) == 16
    for nm, o in adds.items():
        blk = nm[:-3]
        if blk.endswith(".0"):
            assert o.a["amask"] is None and o.a["addend"] == "dds:" + blk
        else:
            bn3 = [b for b in net.bwd if b.kind == "bn_bwd" and b.name == blk + ".bn3"][0]
            assert o.a["amask"] == fwd[blk + ".bn3"].a["mask"]
            assert o.a["addend"] == bn3.a["dy"]
    swapped = ResNet50(n=1, image=64, device="cpu", bn_swap=True)
    assert all(o.a["mask"] is None for o in swapped.fwd if o.kind in ("bn_fwd", "conv_bn_fwd"))


def test_stem_bn_feeds_the_pool_directly(net):
    # the stem BN + ReLU and the max pool are one call; the BN output is not
    # kept (its backward recomputes the mask from the conv output)
    kinds = [o.kind for o in net.fwd[:3]]
    assert kinds == ["conv_fwd", "bn_maxpool_fwd", "conv_bn_fwd"]
    f = net.fwd[1].a
    assert (f["x"], f["y"], f["idx"]) == ("stem.y", "pool.y", "pool.idx")
    assert "stem.bn.y" not in net.buffers and "d:stem.bn.y" in net.buffers
    b = next(o for o in net.bwd if o.kind == "bn_bwd" and o.name == "stem.bn")
    assert b.a["y"] is None and b.a["mask"] is None and b.a["x"] == "stem.y"
    plain = ResNet50(n=1, image=64, device="cpu", fuse_bn_stats=False)
    assert [o.kind for o in plain.fwd[:3]] == ["conv_fwd", "bn_fwd", "maxpool_fwd"]


def test_strided_shortcut_gradient_on_its_own_grid(net):
    # a stride-2 1x1 shortcut's data gradient is a 1x1 stride-1 problem on the
    # shortcut's output grid, added by the block input's data gradient at stride 2
    for st in (2, 3, 4):
        blk = f"l{st}.0"
        ds = next(o for o in net.bwd if o.name == blk + ".ds" and o.kind == "conv_dgrad")
        add = next(o for o in net.bwd if o.name == blk + ".c1" and o.kind == "conv_dgrad_add")
        fwd = next(c for c in net.convs if c["name"] == blk + ".ds")["desc"]
        d = ds.a["desc"]
        p, q = F.fp16_conv_out_dims(fwd)
        assert (d.n, d.c, d.h, d.w, d.k, d.r, d.s, d.stride_h, d.pad_h) == \
            (fwd.n, fwd.c, p, q, fwd.k, 1, 1, 1, 0)
        assert tuple(net.buffers[ds.a["dx"]].shape) == (fwd.n, p, q, fwd.c)
        assert add.a["addend"] == ds.a["dx"] and add.a["astride"] == 2
        wgrad = next(o for o in net.bwd if o.name == blk + ".ds" and o.kind == "conv_wgrad")
        assert wgrad.a["desc"] is fwd
    l1 = next(o for o in net.bwd if o.name == "l1.0.c1" and o.kind == "conv_dgrad_add")
    assert l1.a["astride"] == 1


def test_forward_shortcut_branches(net):
    # each downsampling shortcut starts with its block's first call and is
    # joined by the block-last BN, which adds it
    br = {net.fwd[k].name: net.fwd[v].name for k, v in net._fwd_branch.items()}
    assert br == {f"l{s}.0.bn1": f"l{s}.0.bnd" for s in (1, 2, 3, 4)}
    for k, v in net._fwd_branch.items():
        assert net.fwd[k].a["x"] == net.fwd[v].a["x"] and k < v
        later = [o for o in net.fwd[v + 1:] if o.a.get("res") == net.fwd[v].a["z"]]
        assert [o.name for o in later] == [net.fwd[v].name[:-4] + ".bn3"]
        # nothing between the block's first call and the shortcut reads its output
        assert all(net.fwd[v].a["z"] not in o.a.values() for o in net.fwd[k:v])


def test_weight_gradient_workgroup_targets(net):
    # the weight gradients beside the backward take the per-stage targets; the
    # first layer's, the last call of the backward, the default
    for op in net.bwd:
        if op.kind != "conv_wgrad":
            continue
        if op.name == "stem":
            assert op.a["wg"] == 0
        elif op.name == "fc":
            assert op.a["wg"] == net.SIDE_WORKGROUPS[-1]
        else:
            assert op.a["wg"] == net.SIDE_WORKGROUPS[int(op.name[1]) - 1]
        assert 0 <= op.a["wg"] <= 512


def test_bn_swap_and_zero_gamma_options():
    net = ResNet50(n=1, image=64, device="cpu", bn_swap=True, zero_gamma_last=True)
    bns = [(o, o.a["bn"] if o.kind == "conv_bn_fwd" else o.a["desc"]) for o in net.fwd
           if o.kind in ("bn_fwd", "conv_bn_fwd")]
    last = [o for o, _ in bns if o.name.endswith(".bn3")]
    assert len(last) == 16 and all(d.swap == 1 for o, d in bns if o.name.endswith(".bn3"))
    others = [o for o, d in bns if not o.name.endswith(".bn3")]
    assert all(d.swap == 0 for o, d in bns if not o.name.endswith(".bn3"))
    assert all(float(net.buffers[o.name + ".gamma"].abs().max()) == 0.0 for o in last)
    assert all(float(net.buffers[o.name + ".gamma"].min()) == 1.0 for o in others)
