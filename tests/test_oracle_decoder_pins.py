"""Pins of the decoder part of the oracle (bilinear 2x upsampling with a lateral add,
and the SwiftNet-like network table) against a library routine, closed forms and
invariants."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import network as N


def test_upsample_matches_library_interpolate():
    x = synth.normal(synth.rng(300), (2, 5, 7, 9)).astype(np.float64)
    want = torch.nn.functional.interpolate(torch.from_numpy(x), scale_factor=2, mode="bilinear",
                                           align_corners=False).numpy()
    assert np.abs(oracle.upsample2x_bilinear(x) - want).max() < 1e-12


def test_upsample_closed_form_two_pixels():
    """A 1x2 input [a, b]: columns a, 3a/4 + b/4, a/4 + 3b/4, b; both output rows equal
    (the single input row is replicated)."""
    a, b = 2.0, 10.0
    got = oracle.upsample2x_bilinear(np.array([[[[a, b]]]]))
    want = np.array([a, 0.75 * a + 0.25 * b, 0.25 * a + 0.75 * b, b])
    assert got.shape == (1, 1, 2, 4)
    assert np.array_equal(got[0, 0, 0], want) and np.array_equal(got[0, 0, 1], want)


def test_upsample_invariants():
    c = np.full((1, 3, 4, 6), 1.25)
    assert np.array_equal(oracle.upsample2x_bilinear(c), np.full((1, 3, 8, 12), 1.25))
    ramp = np.tile(np.arange(6.0), (1, 1, 4, 1))              # linear in x
    up = oracle.upsample2x_bilinear(ramp)
    xs = (np.arange(12) + 0.5) / 2 - 0.5                      # interior columns stay linear
    assert np.allclose(up[0, 0, 0, 1:11], xs[1:11], atol=1e-15)


def test_sparse_upsample_add_select_rules():
    r = synth.rng(301)
    coarse = synth.to_storage_bits(synth.normal(r, (1, 8, 8, 16)), "bf16")
    skip = synth.to_storage_bits(synth.normal(r, (1, 8, 16, 32)), "bf16")
    prev = synth.nan_canaries(r, (1, 8, 16, 32), "bf16")
    zeros = np.zeros((1, 2, 4), np.uint8)
    assert np.array_equal(oracle.sparse_upsample_add(coarse, skip, zeros, prev, "bf16"), prev)
    full = oracle.sparse_upsample_add(coarse, skip, np.ones_like(zeros), prev, "bf16")
    want = oracle.store(oracle.upsample2x_bilinear(oracle.value(coarse, "bf16")) + oracle.value(skip, "bf16"), "bf16")
    assert np.array_equal(full, want)


def test_swiftnet_table_shapes():
    T = N.swiftnet_table(18, classes=19, width=128)
    S = N.shapes(T, 1024, 2048)
    assert S[-1] == (64, 256, 512) and T[-1]["classes"] == 19          # stride-4 head
    for i, l in enumerate(T):
        if l["kind"] == "up":
            c, h, w = S[l["src"]]
            assert S[i] == (c, 2 * h, 2 * w) == S[l["res"]]             # skip matches
    assert sum(l["kind"] == "up" for l in T) == 3
    spp = [i for i, l in enumerate(T) if l["kind"] == "spp"]
    assert len(spp) == 1 and S[spp[0]] == (128 + 4 * 32, 32, 64)         # stride 32, concat


def test_swiftnet_static_frame_invariance():
    """A sparse frame on the input of a full frame reproduces the full frame's buffers
    bit for bit (every halo is then a valid copy), decoder included."""
    T = N.swiftnet_table(18, classes=19, width=64)
    P = N.fold_params(T, N.make_params(T, seed0=1000), "bf16")
    h, w = 128, 256
    x = synth.to_storage_bits(synth.normal(synth.rng(302), (1, 3, h, w)), "bf16")
    S = N.shapes(T, h, w)
    prev = [np.zeros((1,) + s, np.uint16) for s in S]
    full = N.frame(T, P, x, np.ones((1, 4, 8), np.uint8), prev, "bf16")
    mask = synth.bernoulli_mask(synth.rng(303), 1, 4, 8, 0.4)
    sparse = N.frame(T, P, x, mask, full, "bf16")
    for a, b in zip(full, sparse):
        assert np.array_equal(a, b)


# ------------------------------------------------------------------ pyramid pooling

def _golden_spp():
    path = __import__("os").path.join(__import__("os").path.dirname(__file__), "golden",
                                      "spp_pool2x2_up4x4.txt")
    sec, out = None, {"pooled": [], "upsampled": []}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line in out:
            sec = line
            continue
        out[sec].append([float(v) for v in line.split()])
    return np.array(out["pooled"]), np.array(out["upsampled"])


def test_spp_hand_worked_example():
    pooled, up = _golden_spp()
    x = np.arange(1.0, 17.0).reshape(1, 1, 4, 4)
    p = oracle.adaptive_avg_pool2d(x, 2, 2)
    assert np.array_equal(p[0, 0], pooled)
    assert np.array_equal(oracle.upsample_bilinear(p, 4, 4)[0, 0], up)


@pytest.mark.parametrize("h,w,oh,ow", [(32, 64, 8, 16), (32, 64, 1, 2), (7, 10, 3, 4), (5, 5, 5, 5),
                                       (9, 13, 2, 7)])
def test_adaptive_avg_pool_matches_library(h, w, oh, ow):
    x = synth.normal(synth.rng(310 + h), (2, 3, h, w)).astype(np.float64)
    want = torch.nn.functional.adaptive_avg_pool2d(torch.from_numpy(x), (oh, ow)).numpy()
    assert np.abs(oracle.adaptive_avg_pool2d(x, oh, ow) - want).max() < 1e-12


@pytest.mark.parametrize("h,w,oh,ow", [(1, 2, 32, 64), (2, 4, 32, 64), (8, 16, 32, 64), (3, 5, 7, 11),
                                       (4, 4, 8, 8), (1, 1, 4, 6)])
def test_upsample_bilinear_matches_library(h, w, oh, ow):
    x = synth.normal(synth.rng(320 + oh), (2, 3, h, w)).astype(np.float64)
    want = torch.nn.functional.interpolate(torch.from_numpy(x), size=(oh, ow), mode="bilinear",
                                           align_corners=False).numpy()
    assert np.abs(oracle.upsample_bilinear(x, oh, ow) - want).max() < 1e-12
    if oh == 2 * h and ow == 2 * w:                   # the decoder's x2 form agrees
        assert np.abs(oracle.upsample2x_bilinear(x) - oracle.upsample_bilinear(x, oh, ow)).max() < 1e-15


def test_spp_bins():
    assert [oracle.spp_bins(32, 64, g) for g in (8, 4, 2, 1)] == [(8, 16), (4, 8), (2, 4), (1, 2)]
    assert [oracle.spp_bins(8, 16, g) for g in (8, 4, 2, 1)] == [(8, 16), (4, 8), (2, 4), (1, 2)]
    assert oracle.spp_bins(2, 4, 8) == (2, 4) and oracle.spp_bins(3, 3, 1) == (1, 1)


def test_spp_levels_constant_and_library_conv():
    """A constant map pools to the constant, and a level equals pooling, a library 1x1
    convolution, bias and ReLU (torch, fp64) rounded to bf16."""
    r = synth.rng(330)
    c, cl = 16, 4
    b = synth.to_storage_bits(synth.normal(r, (1, c, 8, 16)), "bf16")
    w = [synth.to_storage_bits(synth.he_normal(r, cl, c, 1, 1), "bf16") for _ in range(2)]
    bias = [synth.normal(r, cl, 0.1).astype(np.float32) for _ in range(2)]
    lv = oracle.spp_levels(b, (4, 1), w, bias, "bf16")
    for g, wl, bl, got in zip((4, 1), w, bias, lv):
        rows, cols = oracle.spp_bins(8, 16, g)
        pooled = torch.nn.functional.adaptive_avg_pool2d(torch.from_numpy(oracle.value(b, "bf16")), (rows, cols))
        z = torch.nn.functional.conv2d(pooled, torch.from_numpy(oracle.value(wl, "bf16")),
                                       torch.from_numpy(bl.astype(np.float64))).clamp_min(0.0)
        assert np.array_equal(got, oracle.store(z.numpy(), "bf16"))
    const = np.full((1, c, 8, 16), 0x3FC0, np.uint16)          # 1.5 in bf16
    wl = synth.to_storage_bits(np.full((cl, c, 1, 1), 0.25), "bf16")
    out = oracle.spp_levels(const, (2,), [wl], [np.zeros(cl, np.float32)], "bf16")[0]
    assert np.array_equal(oracle.value(out, "bf16"), np.full((1, cl, 2, 4), 0.25 * 1.5 * c))


def test_sparse_spp_select_rules():
    """No block executed: the previous bits; every block: the bottleneck's own bits in
    the first channels, then each level upsampled to the map and rounded."""
    r = synth.rng(331)
    b = synth.to_storage_bits(synth.normal(r, (1, 8, 8, 16)), "bf16")
    lv = [synth.to_storage_bits(synth.normal(r, (1, 2, g, 2 * g)), "bf16") for g in (4, 2, 1)]
    prev = synth.nan_canaries(r, (1, 14, 8, 16), "bf16")
    zeros = np.zeros((1, 2, 4), np.uint8)
    assert np.array_equal(oracle.sparse_spp(b, lv, zeros, prev, "bf16"), prev)
    full = oracle.sparse_spp(b, lv, np.ones_like(zeros), prev, "bf16")
    assert np.array_equal(full[:, :8], b)
    for k, l in enumerate(lv):
        up = oracle.store(oracle.upsample_bilinear(oracle.value(l, "bf16"), 8, 16), "bf16")
        assert np.array_equal(full[:, 8 + 2 * k:10 + 2 * k], up)
    part = synth.bernoulli_mask(r, 1, 2, 4, 0.5)
    got = oracle.sparse_spp(b, lv, part, prev, "bf16")
    sel = np.repeat(np.repeat(part != 0, 4, 1), 4, 2)[:, None]
    assert np.array_equal(np.where(sel, full, prev), got)


def test_spp_levels_read_every_block():
    """The levels pool the whole current input buffer, so changing a block that does not
    run this frame still changes the executed blocks' context channels (the dense
    definition the method is held to)."""
    r = synth.rng(332)
    b = synth.to_storage_bits(synth.normal(r, (1, 4, 8, 16)), "bf16")
    w = [synth.to_storage_bits(np.abs(synth.he_normal(r, 2, 4, 1, 1)), "bf16")]
    bias = [np.zeros(2, np.float32)]
    b2 = b.copy()
    b2[:, :, 4:, 8:] = synth.to_storage_bits(np.full((1, 4, 4, 8), 8.0), "bf16")   # one block
    l1 = oracle.spp_levels(b, (1,), w, bias, "bf16")
    l2 = oracle.spp_levels(b2, (1,), w, bias, "bf16")
    assert not np.array_equal(l1[0], l2[0])
    mask = np.zeros((1, 2, 2), np.uint8)
    mask[0, 0, 0] = 1                                       # the changed block does not run
    prev = np.zeros((1, 6, 8, 16), np.uint16)
    y1 = oracle.sparse_spp(b, l1, mask, prev, "bf16")
    y2 = oracle.sparse_spp(b2, l2, mask, prev, "bf16")
    assert not np.array_equal(y1[:, 4:, :4, :8], y2[:, 4:, :4, :8])
