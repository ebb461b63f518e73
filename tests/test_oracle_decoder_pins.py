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
