"""Network-level oracle: a ResNet backbone executed block-sparsely frame by frame.

TEST INFRASTRUCTURE ONLY (see the package docstring).

In single-stage networks every convolution layer is made block-sparse (Section 4,
first paragraph), all layers of a frame share the frame's execution grid A_t
(Section 3.5), each layer keeps its own stored representation (Section 3.1), and
the first frame of a clip is executed completely (Section 4, BlockCopy
configuration). Layers run in network order: layer l reads layer l-1's buffer after
it has been updated for this frame.

The backbones are the standard ResNet-18 / ResNet-50 feature extractors (He et al.,
2016) with the stride of a downsampling bottleneck on its 3x3 convolution (the
torchvision convention), batch normalisation folded into the convolutions, and
no classifier. The layer table below is written here from that definition; the
HIP runner has its own.
"""
from __future__ import annotations

import numpy as np

from . import (fold_bn, sparse_conv2d, sparse_conv2d_active, sparse_maxpool2d, sparse_spp,
               sparse_upsample_add, spp_levels, store)


def resnet_table(depth: int):
    """List of layers. Each is a dict: kind ('conv'|'pool'), name, src (index of the
    input layer, -1 = the frame), res (index of the residual layer or None),
    cin, cout, k, stride, pad, relu."""
    L = []

    def conv(name, src, cin, cout, k, s, relu, res=None):
        L.append(dict(kind="conv", name=name, src=src, res=res, cin=cin, cout=cout,
                      k=k, stride=s, pad=k // 2, relu=relu))
        return len(L) - 1

    x = conv("stem", -1, 3, 64, 7, 2, True)
    L.append(dict(kind="pool", name="maxpool", src=x, res=None, cin=64, cout=64,
                  k=3, stride=2, pad=1, relu=False))
    x = len(L) - 1
    cin = 64
    if depth == 50:
        stages, width, expansion = [3, 4, 6, 3], [64, 128, 256, 512], 4
    elif depth == 18:
        stages, width, expansion = [2, 2, 2, 2], [64, 128, 256, 512], 1
    else:
        raise ValueError(depth)
    for si, (nb, wd) in enumerate(zip(stages, width)):
        for bi in range(nb):
            s = 2 if (si > 0 and bi == 0) else 1
            cout = wd * expansion
            pre = f"layer{si + 1}.{bi}"
            if bi == 0 and (s != 1 or cin != cout):
                ds = conv(pre + ".downsample", x, cin, cout, 1, s, False)
            else:
                ds = x
            if depth == 50:
                a = conv(pre + ".conv1", x, cin, wd, 1, 1, True)
                b = conv(pre + ".conv2", a, wd, wd, 3, s, True)
                x = conv(pre + ".conv3", b, wd, cout, 1, 1, True, res=ds)
            else:
                a = conv(pre + ".conv1", x, cin, wd, 3, s, True)
                x = conv(pre + ".conv2", a, wd, cout, 3, 1, True, res=ds)
            cin = cout
    return L


SPP_GRID = (8, 4, 2, 1)      # rows of the pyramid levels' bin grids


def swiftnet_table(depth: int = 18, classes: int = 19, width: int = 128):
    """A SwiftNet-like single-scale segmentation network (Orsic et al., 2019; the
    paper's semantic segmentation model, Section 4, with a ResNet backbone): the ResNet
    encoder above, a spatial pyramid pooling module on the stride-32 feature, then a
    decoder that runs at strides 32 -> 16 -> 8 -> 4. Pyramid pooling: a 1x1 bottleneck
    to `width` channels; levels with 8, 4, 2 and 1 rows of bins (spp_bins), each the
    bins' means, a 1x1 convolution to width/4 channels and ReLU, upsampled bilinearly
    to the map and concatenated after the bottleneck (kind 'spp', computed densely and
    selected, see oracle.sparse_spp); a 1x1 fuse back to `width`. Each merge upsamples
    the coarser decoder feature by two (bilinear) and adds a 1x1 lateral projection of
    the encoder feature of the finer stride, then blends with a 3x3 convolution; a 1x1
    head gives the class scores at stride 4. Reading: the head computes a multiple of 64
    channels (what the matrix-core layers take) of which the first `classes` are the
    class scores. Layer kind 'up': src = coarse feature, res = lateral (skip)."""
    L = resnet_table(depth)
    ends = {}
    for i, l in enumerate(L):
        if l["name"].startswith("layer") and (i + 1 == len(L) or L[i + 1]["name"].split(".")[0] != l["name"].split(".")[0]):
            ends[int(l["name"][5])] = i          # last layer of stage 1..4
    expansion = 4 if depth == 50 else 1

    def conv(name, src, cin, cout, k, relu):
        L.append(dict(kind="conv", name=name, src=src, res=None, cin=cin, cout=cout,
                      k=k, stride=1, pad=k // 2, relu=relu))
        return len(L) - 1

    b = conv("dec.spp.bottleneck", ends[4], 512 * expansion, width, 1, True)
    cl = width // 4
    cat = width + len(SPP_GRID) * cl
    L.append(dict(kind="spp", name="dec.spp", src=b, res=None, cin=width, cout=cat, k=1, stride=1,
                  pad=0, relu=True, grid=SPP_GRID, cl=cl))
    x = conv("dec.spp.fuse", len(L) - 1, cat, width, 1, True)
    for s in (3, 2, 1):
        lat = conv(f"dec.lat{s}", ends[s], (64 << (s - 1)) * expansion, width, 1, True)
        L.append(dict(kind="up", name=f"dec.up{s}", src=x, res=lat, cin=width, cout=width,
                      k=1, stride=1, pad=0, relu=False))
        x = conv(f"dec.blend{s}", len(L) - 1, width, width, 3, True)
    head = conv("dec.logits", x, width, -(-classes // 64) * 64, 1, False)
    L[head]["classes"] = classes      # the first `classes` channels are the class scores
    return L


def policy_table():
    """The policy network (Section 3.3; reading in policy.py): on S_t (32 channels at a
    quarter of the frame resolution) a 3x3 stride-2 stem to 64 channels, three basic
    residual blocks (64, 128, 256 channels; the second and third stride 2 with a 1x1
    stride-2 projection on the shortcut), then a fully convolutional head of two 3x3
    stride-2 convolutions down to one pixel per 128-pixel block (64 channels, channel 0
    is the block's logit, no ReLU on the last)."""
    L = []

    def conv(name, src, cin, cout, k, s, relu, res=None):
        L.append(dict(kind="conv", name=name, src=src, res=res, cin=cin, cout=cout,
                      k=k, stride=s, pad=k // 2, relu=relu))
        return len(L) - 1

    x = conv("pn.stem", -1, 32, 64, 3, 2, True)
    a = conv("pn.block1.conv1", x, 64, 64, 3, 1, True)
    x = conv("pn.block1.conv2", a, 64, 64, 3, 1, True, res=x)
    cin = 64
    for i, c in ((2, 128), (3, 256)):
        ds = conv(f"pn.block{i}.downsample", x, cin, c, 1, 2, False)
        a = conv(f"pn.block{i}.conv1", x, cin, c, 3, 2, True)
        x = conv(f"pn.block{i}.conv2", a, c, c, 3, 1, True, res=ds)
        cin = c
    x = conv("pn.head1", x, 256, 64, 3, 2, True)
    conv("pn.head2", x, 64, 64, 3, 2, False)
    return L


def dense_frame(table, folded, x_bits, dtype):
    """Every layer on every pixel (a full execution grid)."""
    n = x_bits.shape[0]
    ones = np.ones((n, 1, 1), np.uint8)
    out = []
    for li, l in enumerate(table):
        src = x_bits if l["src"] < 0 else out[l["src"]]
        res = None if l["res"] is None else out[l["res"]]
        oh = (src.shape[2] + 2 * l["pad"] - l["k"]) // l["stride"] + 1
        ow = (src.shape[3] + 2 * l["pad"] - l["k"]) // l["stride"] + 1
        prev = np.zeros((n, l["cout"], oh, ow), np.uint16)
        out.append(sparse_conv2d(src, folded[li]["w_bits"], ones, prev, dtype, stride=l["stride"],
                                 pad=l["pad"], bias=folded[li]["bias"], residual_bits=res,
                                 relu=l["relu"]))
    return out


def make_params(table, seed0=1000, bn_random=False):
    """Per-conv fp32 OIHW weights (He-normal, seed seed0 + layer index) and BN
    parameters; a pyramid pooling layer gets one such set per level (1x1, cl x cin),
    drawn in level order from the layer's seed. Random init uses gamma=1, beta=0,
    mean=0, var=1 unless bn_random."""
    import synth
    params = []

    def one(r, cout, cin, k):
        w = synth.he_normal(r, cout, cin, k, k)
        if bn_random:
            bn = dict(gamma=r.uniform(0.5, 1.5, cout), beta=r.normal(0, 0.1, cout),
                      mean=r.normal(0, 0.1, cout), var=r.uniform(0.5, 1.5, cout))
        else:
            bn = dict(gamma=np.ones(cout), beta=np.zeros(cout), mean=np.zeros(cout), var=np.ones(cout))
        return dict(w=w, **bn)

    for li, l in enumerate(table):
        r = synth.rng(seed0 + li)
        if l["kind"] == "conv":
            params.append(one(r, l["cout"], l["cin"], l["k"]))
        elif l["kind"] == "spp":
            params.append(dict(levels=[one(r, l["cl"], l["cin"], 1) for _ in l["grid"]]))
        else:
            params.append(None)
    return params


def fold_params(table, params, dtype):
    """BN folded in fp64; weights rounded to the storage dtype (bit patterns),
    bias rounded to fp32 (per level for a pyramid pooling layer)."""
    def one(p):
        w2, b2 = fold_bn(p["w"], None, p["gamma"], p["beta"], p["mean"], p["var"], 1e-5)
        return dict(w_bits=store(w2, dtype), bias=b2.astype(np.float32))

    out = []
    for l, p in zip(table, params):
        if p is None:
            out.append(None)
        elif l["kind"] == "spp":
            out.append(dict(levels=[one(q) for q in p["levels"]]))
        else:
            out.append(one(p))
    return out


def shapes(table, h, w):
    """Output (C, H, W) of every layer for an input frame of h x w."""
    out = []
    for l in table:
        ih, iw = (h, w) if l["src"] < 0 else out[l["src"]][1:]
        if l["kind"] == "up":
            out.append((l["cout"], 2 * ih, 2 * iw))
            continue
        oh = (ih + 2 * l["pad"] - l["k"]) // l["stride"] + 1
        ow = (iw + 2 * l["pad"] - l["k"]) // l["stride"] + 1
        out.append((l["cout"], oh, ow))
    return out


def frame(table, folded, x_bits, mask, prev, dtype, only_active=False):
    """One frame through the block-sparse network.

    x_bits: the frame, NCHW bit patterns. mask: uint8 [N, Gh, Gw] execution grid.
    prev: list of previous per-layer buffers (NCHW bit patterns). Returns the new list.
    only_active: convolutions through sparse_conv2d_active (the same bits, inactive
    blocks not computed), for timing the fair sparse CPU comparison.
    """
    conv = sparse_conv2d_active if only_active else sparse_conv2d
    bufs = []
    for li, l in enumerate(table):
        src = x_bits if l["src"] < 0 else bufs[l["src"]]
        if l["kind"] == "pool":
            y = sparse_maxpool2d(src, mask, prev[li], dtype, l["k"], l["stride"], l["pad"])
        elif l["kind"] == "up":
            y = sparse_upsample_add(src, bufs[l["res"]], mask, prev[li], dtype, relu=l["relu"])
        elif l["kind"] == "spp":
            lv = folded[li]["levels"]
            levels = spp_levels(src, l["grid"], [q["w_bits"] for q in lv], [q["bias"] for q in lv], dtype)
            y = sparse_spp(src, levels, mask, prev[li], dtype)
        else:
            res = None if l["res"] is None else bufs[l["res"]]
            y = conv(src, folded[li]["w_bits"], mask, prev[li], dtype,
                              stride=l["stride"], pad=l["pad"], bias=folded[li]["bias"],
                              residual_bits=res, relu=l["relu"])
        bufs.append(y)
    return bufs
