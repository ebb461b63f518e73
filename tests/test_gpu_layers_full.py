"""GPU: every layer of the 2048x1024 networks held element-wise to the oracle, one layer
at a time, with all of the layer's inputs drawn on the host (no GPU value enters the
oracle).

For ResNet-50, SwiftNet-18 and SwiftNet-50 at 2048x1024 (128-pixel blocks, 38 of the 128 blocks
active, clustered): the layer's input, residual and previous output are drawn seeded on
the host and uploaded into the runner's own persistent buffers, the oracle's folded
weights into the runner's weight tensors; the layer then runs alone through the runner
(run_layer, or run_pair where the frame launches two layers together) on the frame's
index, in the launch configuration of the benchmark's frame. Checked (Section 3.1):
* every element outside the active blocks keeps the uploaded previous bits;
* active outputs of convolutions match the oracle's dense definition within 2e-2 max
  abs-rel on sampled points (computed one by one at full size); max pooling on every
  active output bit for bit (a maximum of stored values is exact); the decoder's
  upsample-add and pyramid pooling on every active output within 2e-2.
Also: the frame with and without paired launches gives the same bits in every buffer,
and every layer of the policy network (Section 3.3) is held element-wise at the
workload's size.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import network as onet
from tests._util import block_select, from_dev, max_abs_rel, to_dev, weights_dev

pytestmark = pytest.mark.gpu

H, W, GH, GW = 1024, 2048, 8, 16
TABLES = {"resnet50": onet.resnet_table(50), "swiftnet18": onet.swiftnet_table(18),
          "swiftnet50": onet.swiftnet_table(50)}
SAMPLES = 2000


@pytest.fixture(scope="module")
def R(gpu):
    from paper_2108_09376_amd import bc, resnet
    return bc, resnet


_NETS = {}


def _net(R, kind):
    """The runner at 2048x1024 with the oracle's parameters, after a full frame (so every
    registered buffer is valid), and the frame's 38-block index."""
    if kind in _NETS:
        return _NETS[kind]
    _NETS.clear()                                    # one network resident at a time
    torch.cuda.empty_cache()
    bc, resnet = R
    table = TABLES[kind]
    params = onet.make_params(table, seed0=1000, bn_random=True)
    folded = onet.fold_params(table, params, "bf16")
    if kind == "resnet50":
        net = resnet.SparseResNet(50, H, W, 128, params=params)
    else:
        net = resnet.SparseSwiftNet(int(kind[-2:]), H, W, 128, params=params)
    for i, f in enumerate(folded):
        if f is None:
            continue
        if "levels" in f:                            # pyramid pooling: [levels][cl][c]
            wl = np.stack([q["w_bits"].reshape(q["w_bits"].shape[:2]) for q in f["levels"]])
            net.weights[i].copy_(torch.from_numpy(wl.view(np.int16)).view(torch.bfloat16).cuda())
            net.biases[i].copy_(torch.from_numpy(np.stack([q["bias"] for q in f["levels"]])).cuda())
        else:                                        # the oracle's own weight bits
            net.weights[i].copy_(weights_dev(f["w_bits"], "bf16"))
            net.biases[i].copy_(torch.from_numpy(f["bias"]).cuda())
    x = to_dev(synth.to_storage_bits(synth.normal(synth.rng(1), (1, 3, H, W)), "bf16"), "bf16")
    net.frame(x, sparse=False)
    mask = synth.frac_mask(synth.SEED_MASK0 + 1, GH, GW, 0.3)
    assert int(mask.sum()) == 38
    net.set_mask(mask)
    bc.bc_build_block_index(net.mask, 1, net.grid, net.idx, net.count)
    torch.cuda.synchronize()
    _NETS[kind] = (net, folded, x, mask)
    return _NETS[kind]


def _cases():
    out = []
    for kind, table in TABLES.items():
        for li, l in enumerate(table):
            out.append(pytest.param(kind, li, id=f"{kind}-{li:02d}-{l['name']}"))
    return out


def _draw_map(seed, shape):
    return synth.to_storage_bits(synth.normal(synth.rng(seed), shape), "bf16")


def _check_layer(net, table, folded, mask, li, src_bits, res_bits, prev_bits, got):
    l = table[li]
    sel = block_select(mask, got.shape)
    assert np.array_equal(got[~sel], prev_bits[~sel]), "a copied block changed"
    if l["kind"] == "pool":
        z = oracle.maxpool2d_dense(oracle.value(src_bits, "bf16"), l["k"], l["stride"], l["pad"])
        want = oracle.store(z, "bf16")
        assert np.array_equal(got[sel], want[sel])
        return 0.0
    if l["kind"] == "up":
        want = oracle.sparse_upsample_add(src_bits, res_bits, mask, prev_bits, "bf16", relu=l["relu"])
        err = max_abs_rel(oracle.value(got[sel], "bf16"), oracle.value(want[sel], "bf16"))
        assert err <= 2e-2, err
        return err
    if l["kind"] == "spp":
        lv = folded[li]["levels"]
        levels = oracle.spp_levels(src_bits, l["grid"], [q["w_bits"] for q in lv], [q["bias"] for q in lv], "bf16")
        want = oracle.sparse_spp(src_bits, levels, mask, prev_bits, "bf16")
        err = max_abs_rel(oracle.value(got[sel], "bf16"), oracle.value(want[sel], "bf16"))
        assert err <= 2e-2, err
        return err
    act = np.argwhere(sel)
    pick = act[synth.rng(7000 + li).choice(len(act), size=min(SAMPLES, len(act)), replace=False)]
    z = oracle.conv2d_points(oracle.value(src_bits, "bf16"), oracle.value(folded[li]["w_bits"], "bf16"),
                             pick, folded[li]["bias"].astype(np.float64),
                             None if res_bits is None else oracle.value(res_bits, "bf16"),
                             l["stride"], l["pad"], l["relu"])
    want = oracle.value(oracle.store(z, "bf16"), "bf16")
    assert np.count_nonzero(want) >= len(want) // 5       # a live sample, not a dead layer
    g = oracle.value(got[pick[:, 0], pick[:, 1], pick[:, 2], pick[:, 3]], "bf16")
    err = max_abs_rel(g, want)
    assert err <= 2e-2, err
    return err


@pytest.mark.parametrize("kind,li", _cases())
def test_layer_teacher_forced_full_size(R, kind, li):
    bc, resnet = R
    net, folded, x, mask = _net(R, kind)
    table = TABLES[kind]
    sh = onet.shapes(table, H, W)
    # the launch this layer belongs to in the frame: alone, or paired with another layer
    partner = net.pairs.get(li)
    first = next((i for i, j in net.pairs.items() if j == li), None)
    group = [li] if partner is None and first is None else sorted([li, partner if partner is not None else first])
    # every input of the launch: the layers' sources (paired layers may read different
    # buffers, e.g. a decoder lateral beside the pyramid's bottleneck), residuals and
    # previous outputs, drawn on the host and uploaded
    srcs, res, prev = {}, {}, {}
    for i in group:
        si = table[i]["src"]
        if si not in srcs:
            srcs[si] = _draw_map(5000 + (si if si >= 0 else 999), (1, 3, H, W) if si < 0 else (1,) + sh[si])
            (x if si < 0 else net.buffers[si]).copy_(to_dev(srcs[si], "bf16"))
    for i in group:
        l = table[i]
        if l["res"] is not None:
            res[i] = _draw_map(5300 + i, (1,) + sh[l["res"]])
            net.buffers[l["res"]].copy_(to_dev(res[i], "bf16"))
        prev[i] = synth.nan_canaries(synth.rng(5600 + i), (1,) + sh[i], "bf16")
        net.buffers[i].copy_(to_dev(prev[i], "bf16"))
    src_bits = srcs[table[li]["src"]]
    src_shape = src_bits.shape
    print(kind, li, [table[i]["name"] for i in group], src_shape, flush=True)
    if len(group) == 2:
        net.run_pair(group[0], group[1], x, net.idx, net.count)
    else:
        net.run_layer(li, x, net.idx, net.count)
    torch.cuda.synchronize()
    got = from_dev(net.buffers[li])
    err = _check_layer(net, table, folded, mask, li, src_bits, res.get(li), prev[li], got)
    print(f"  max abs-rel {err:.3e}")


@pytest.mark.parametrize("kind", ["resnet50", "swiftnet18"])
def test_paired_and_single_launches_same_bits(R, kind):
    """The frame with independent 1x1 layers paired into one launch and with every layer
    launched alone: every buffer bit for bit after a full frame and a sparse frame."""
    bc, resnet = R
    _NETS.clear()
    torch.cuda.empty_cache()
    if kind == "resnet50":
        net = resnet.SparseResNet(50, H, W, 128, bn_random=True)
    else:
        net = resnet.SparseSwiftNet(18, H, W, 128, bn_random=True)
    assert net.pairs
    x0 = to_dev(synth.to_storage_bits(synth.normal(synth.rng(31), (1, 3, H, W)), "bf16"), "bf16")
    x1 = to_dev(synth.to_storage_bits(synth.normal(synth.rng(32), (1, 3, H, W)), "bf16"), "bf16")
    net.set_mask(synth.frac_mask(33, GH, GW, 0.3))
    snaps = []
    for paired in (True, False):
        net.pair_launches = paired
        net.frame(x0, sparse=False)
        net.frame(x1, sparse=True)
        torch.cuda.synchronize()
        snaps.append([b.view(torch.int16).clone() for b in net.buffers])
    for i, (a, b) in enumerate(zip(*snaps)):
        assert torch.equal(a, b), net.layers[i].name
    del snaps, net
    torch.cuda.empty_cache()


def test_policy_layers_teacher_forced(R):
    """Every layer of the policy network on the dense path at the 2048x1024 workload
    (S_t 512x256), inputs drawn on the host: element-wise within 2e-2 on every output."""
    bc, resnet = R
    _NETS.clear()
    torch.cuda.empty_cache()
    table = onet.policy_table()
    params = onet.make_params(table, seed0=3000)
    folded = onet.fold_params(table, params, "bf16")
    net = resnet.PolicyNet(H, W, params=params)
    sh = onet.shapes(table, H // 4, W // 4)
    for li, l in enumerate(table):
        net.weights[li].copy_(weights_dev(folded[li]["w_bits"], "bf16"))
        net.biases[li].copy_(torch.from_numpy(folded[li]["bias"]).cuda())
        src_shape = (1, 32, H // 4, W // 4) if l["src"] < 0 else (1,) + sh[l["src"]]
        src_bits = _draw_map(6000 + li, src_shape)
        src = net.input if l["src"] < 0 else net.buffers[l["src"]]
        src.copy_(to_dev(src_bits, "bf16"))
        res_bits = None
        if l["res"] is not None:
            res_bits = _draw_map(6100 + li, (1,) + sh[l["res"]])
            net.buffers[l["res"]].copy_(to_dev(res_bits, "bf16"))
        bc.bc_sparse_conv2d((l["k"], l["k"], l["stride"], l["pad"], int(l["relu"])), src, bc.BC_NHWC,
                            net.weights[li], net.biases[li],
                            None if l["res"] is None else net.buffers[l["res"]], net.buffers[li],
                            net.grids[li], None, None)
        torch.cuda.synchronize()
        got = from_dev(net.buffers[li])
        want = oracle.sparse_conv2d(src_bits, folded[li]["w_bits"], np.ones((1, 1, 1), np.uint8),
                                    np.zeros_like(got), "bf16", stride=l["stride"], pad=l["pad"],
                                    bias=folded[li]["bias"], residual_bits=res_bits, relu=l["relu"])
        err = max_abs_rel(oracle.value(got, "bf16"), oracle.value(want, "bf16"))
        print(l["name"], src_shape, f"max abs-rel {err:.3e}", flush=True)
        assert err <= 2e-2, (l["name"], err)
