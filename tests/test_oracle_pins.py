"""Pins of the CPU oracle against things other than itself: library routines
(torch CPU in fp64), brute-force loops on tiny inputs, hand-worked fixtures,
closed forms and invariants. CPU only."""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import network as net

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    on = False
    for line in open(os.path.join(GOLDEN, name)):
        if line.startswith("#") or not line.strip():
            continue
        if line.strip() == "output":
            on = True
            continue
        if on:
            rows.append([float(v) for v in line.split()])
    return np.array(rows)


def _torch_conv(x, w, b, res, s, p, relu):
    y = F.conv2d(torch.from_numpy(x), torch.from_numpy(w),
                 None if b is None else torch.from_numpy(b), stride=s, padding=p)
    if res is not None:
        y = y + torch.from_numpy(res)
    if relu:
        y = torch.relu(y)
    return y.numpy()


# ---------------------------------------------------------------- index

def test_block_index_bruteforce():
    r = synth.rng(11)
    for n, gh, gw, p in [(1, 8, 16, 0.3), (2, 3, 5, 0.5), (1, 1, 1, 1.0), (3, 4, 4, 0.0)]:
        m = synth.bernoulli_mask(r, n, gh, gw, p)
        idx, cnt = oracle.block_index(m)
        want = []
        for a in range(n):
            for y in range(gh):
                for x in range(gw):
                    if m[a, y, x]:
                        want.append((a * gh + y) * gw + x)
        assert cnt == len(want) and idx.tolist() == want and idx.dtype == np.int32


def test_block_index_nonzero_bytes_execute():
    m = np.array([[[0, 3, 255], [1, 0, 0]]], np.uint8)
    idx, cnt = oracle.block_index(m)
    assert cnt == 3 and idx.tolist() == [1, 2, 3]


# ---------------------------------------------------------------- rounding

def test_bf16_rounding_matches_torch():
    r = synth.rng(12)
    x = np.concatenate([
        r.standard_normal(20000).astype(np.float32) * 10.0 ** r.integers(-30, 30, 20000),
        np.array([0.0, -0.0, np.inf, -np.inf, 1.0, 1.00390625, 1.0078125, 1.01171875,
                  3.4e38, -3.4e38, 1e-40, -1e-40, 1.17549435e-38], np.float32),
    ]).astype(np.float32)
    # exact ties (low 16 bits == 0x8000) on both parities of the kept mantissa, both signs
    m7 = r.integers(0, 128, 4000).astype(np.uint32) << 16
    sg = r.integers(0, 2, 4000).astype(np.uint32) << 31
    ex = r.integers(1, 254, 4000).astype(np.uint32) << 23
    ties = (sg | ex | m7 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties])
    got = oracle.f32_to_bf16_bits(x)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    nan = oracle.f32_to_bf16_bits(np.array([np.nan], np.float32))
    assert np.isnan(oracle.value(nan, "bf16")).all()


def test_store_fp64_to_f32_then_bf16():
    r = synth.rng(13)
    z = r.standard_normal(5000) * 100
    got = oracle.store(z, "bf16")
    want = torch.from_numpy(z).to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    got16 = oracle.store(z, "f16")
    want16 = torch.from_numpy(z).to(torch.float32).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got16, want16)


# ---------------------------------------------------------------- dense conv

@pytest.mark.parametrize("cin,cout,h,w,k,s,p", [
    (3, 5, 9, 11, 3, 1, 1), (4, 2, 10, 7, 3, 2, 1), (3, 4, 15, 13, 7, 2, 3),
    (6, 3, 8, 8, 1, 1, 0), (5, 7, 9, 9, 1, 2, 0), (2, 3, 6, 5, 3, 1, 0)])
def test_conv_dense_matches_torch_fp64(cin, cout, h, w, k, s, p):
    r = synth.rng(100 + cin * 7 + k)
    x = r.standard_normal((2, cin, h, w))
    wt = r.standard_normal((cout, cin, k, k))
    b = r.standard_normal(cout)
    ho, wo = oracle.out_size(h, k, s, p), oracle.out_size(w, k, s, p)
    res = r.standard_normal((2, cout, ho, wo))
    for bias, resid, relu in [(None, None, False), (b, None, True), (b, res, True), (None, res, False)]:
        got = oracle.conv2d_dense(x, wt, bias, resid, s, p, relu)
        want = _torch_conv(x, wt, bias, resid, s, p, relu)
        assert got.shape == want.shape
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_conv_tiny_bruteforce_loops():
    r = synth.rng(14)
    for (cin, cout, h, w, k, s, p) in [(2, 3, 4, 4, 3, 1, 1), (3, 2, 4, 3, 3, 2, 1), (1, 1, 4, 4, 1, 2, 0)]:
        x = r.integers(-3, 4, (1, cin, h, w)).astype(np.float64)
        wt = r.integers(-2, 3, (cout, cin, k, k)).astype(np.float64)
        b = r.integers(-5, 6, cout).astype(np.float64)
        ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
        want = np.zeros((1, cout, ho, wo))
        for co in range(cout):
            for y in range(ho):
                for xx in range(wo):
                    t = b[co]
                    for ci in range(cin):
                        for i in range(k):
                            for j in range(k):
                                yy, xj = y * s - p + i, xx * s - p + j
                                if 0 <= yy < h and 0 <= xj < w:
                                    t += wt[co, ci, i, j] * x[0, ci, yy, xj]
                    want[0, co, y, xx] = t
        got = oracle.conv2d_dense(x, wt, b, None, s, p, False)
        assert np.array_equal(got, want)


def test_conv_golden_window_sums():
    x = np.arange(1, 17, dtype=np.float64).reshape(1, 1, 4, 4)
    wt = np.ones((1, 1, 3, 3))
    got = oracle.conv2d_dense(x, wt, None, None, 1, 1, False)[0, 0]
    assert np.array_equal(got, _golden("conv3x3_4x4_ones.txt"))


def test_conv_delta_is_cross_correlation():
    """A unit impulse at (y0, x0) yields out[co, y, x] = W[co, ci, y0 - y*s + p, x0 - x*s + p]
    (no kernel flip), zero elsewhere."""
    r = synth.rng(15)
    cin, cout, k, s, p, h, w = 2, 3, 3, 2, 1, 9, 9
    wt = r.standard_normal((cout, cin, k, k))
    y0, x0, c0 = 4, 5, 1
    x = np.zeros((1, cin, h, w))
    x[0, c0, y0, x0] = 1.0
    got = oracle.conv2d_dense(x, wt, None, None, s, p, False)
    ho = got.shape[2]
    for co in range(cout):
        for y in range(ho):
            for xx in range(got.shape[3]):
                i, j = y0 - y * s + p, x0 - xx * s + p
                want = wt[co, c0, i, j] if (0 <= i < k and 0 <= j < k) else 0.0
                assert got[0, co, y, xx] == want


def test_conv_points_equal_dense():
    r = synth.rng(16)
    x = r.standard_normal((2, 4, 10, 12))
    wt = r.standard_normal((5, 4, 3, 3))
    b = r.standard_normal(5)
    res = r.standard_normal((2, 5, 5, 6))
    dense = oracle.conv2d_dense(x, wt, b, res, 2, 1, True)
    pts = np.stack([r.integers(0, 2, 50), r.integers(0, 5, 50), r.integers(0, 5, 50),
                    r.integers(0, 6, 50)], 1)
    got = oracle.conv2d_points(x, wt, pts, b, res, 2, 1, True)
    assert np.array_equal(got, dense[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]])


# ---------------------------------------------------------------- select

def _layer_inputs(seed, dtype, n=1, cin=4, cout=3, h=16, w=24, k=3):
    r = synth.rng(seed)
    x = synth.to_storage_bits(synth.normal(r, (n, cin, h, w)), dtype)
    wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), dtype)
    b = synth.normal(r, cout)
    prev = synth.nan_canaries(r, (n, cout, h, w), dtype)
    return x, wt, b, prev


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_all_zero_mask_keeps_previous_bits(dtype):
    x, wt, b, prev = _layer_inputs(17, dtype)
    mask = np.zeros((1, 4, 6), np.uint8)
    y = oracle.sparse_conv2d(x, wt, mask, prev, dtype, 1, 1, b, None, True)
    assert y.dtype == prev.dtype and np.array_equal(y, prev)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_ones_mask_equals_dense_library_conv(dtype):
    x, wt, b, prev = _layer_inputs(18, dtype)
    mask = np.ones((1, 4, 6), np.uint8)
    y = oracle.sparse_conv2d(x, wt, mask, prev, dtype, 1, 1, b, None, True)
    xv, wv = synth.storage_to_f64(x, dtype), synth.storage_to_f64(wt, dtype)
    ref = torch.relu(F.conv2d(torch.from_numpy(xv), torch.from_numpy(wv),
                              torch.from_numpy(b.astype(np.float64)), padding=1))
    ref = ref.to(torch.float32)
    if dtype == "bf16":
        ref = ref.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    else:
        ref = ref.numpy().view(np.uint32)
    assert np.array_equal(y, ref)


def test_select_random_mask_per_pixel_loop():
    x, wt, b, prev = _layer_inputs(19, "bf16", n=2, h=8, w=12)
    r = synth.rng(20)
    mask = synth.bernoulli_mask(r, 2, 2, 3, 0.5)
    y = oracle.sparse_conv2d(x, wt, mask, prev, "bf16", 1, 1, b, None, False)
    dense = oracle.sparse_conv2d(x, wt, np.ones_like(mask), prev, "bf16", 1, 1, b, None, False)
    for a in range(2):
        for c in range(3):
            for yy in range(8):
                for xx in range(12):
                    want = dense[a, c, yy, xx] if mask[a, yy // 4, xx // 4] else prev[a, c, yy, xx]
                    assert y[a, c, yy, xx] == want


def test_strided_layer_blocks_index_output():
    """Stride 2: the mask indexes output blocks; input 16x24 -> output 8x12 on a 2x3
    grid gives 4x4 output blocks."""
    x, wt, b, _ = _layer_inputs(21, "f32", h=16, w=24)
    prev = np.zeros((1, 3, 8, 12), np.uint32)
    mask = np.array([[[1, 0, 0], [0, 0, 1]]], np.uint8)
    y = oracle.sparse_conv2d(x, wt, mask, prev, "f32", 2, 1, b, None, False)
    full = oracle.sparse_conv2d(x, wt, np.ones_like(mask), prev, "f32", 2, 1, b, None, False)
    assert np.array_equal(y[..., 0:4, 0:4], full[..., 0:4, 0:4])
    assert np.array_equal(y[..., 4:8, 8:12], full[..., 4:8, 8:12])
    assert not y[..., 0:4, 4:12].any() and not y[..., 4:8, 0:8].any()


# ---------------------------------------------------------------- integer exact

def test_integer_inputs_exact_in_bf16():
    """Small-integer operands: every partial sum is an integer below 2^24, so the
    oracle's bf16 output equals the exact integer result (scipy correlate, int64)."""
    from scipy.signal import correlate
    r = synth.rng(22)
    cin, cout, h, w = 5, 3, 12, 10
    x = synth.small_ints(r, (1, cin, h, w), -2, 2)
    wt = synth.small_ints(r, (cout, cin, 3, 3), -2, 2)
    b = synth.small_ints(r, cout, -3, 3)
    xb, wb = synth.to_storage_bits(x, "bf16"), synth.to_storage_bits(wt, "bf16")
    y = oracle.sparse_conv2d(xb, wb, np.ones((1, 2, 2), np.uint8),
                             np.zeros((1, cout, h, w), np.uint16), "bf16", 1, 1, b, None, False)
    xp = np.pad(x[0].astype(np.int64), ((0, 0), (1, 1), (1, 1)))
    for co in range(cout):
        exact = correlate(xp, wt[co].astype(np.int64), mode="valid")[0] + int(b[co])
        assert np.abs(exact).max() < 256
        assert np.array_equal(oracle.value(y[0, co], "bf16"), exact.astype(np.float64))


# ---------------------------------------------------------------- gather / scatter

def test_gather_matches_padded_slices():
    r = synth.rng(23)
    x = synth.to_storage_bits(synth.normal(r, (2, 3, 16, 24)), "bf16")
    gh, gw = 2, 3
    for (k, s, p) in [(3, 1, 1), (1, 1, 0), (3, 2, 1), (7, 2, 3), (1, 2, 0)]:
        bh, bw = oracle.out_size(16, k, s, p) // gh, oracle.out_size(24, k, s, p) // gw
        idx = np.array([0, 4, 5, 7, 11], np.int32)
        got = oracle.gather_halo(x, idx, gh, gw, bh, bw, k, k, s, p, 0)
        big = 40
        xp = np.pad(x, ((0, 0), (0, 0), (big, big), (big, big)))
        th, tw = (bh - 1) * s + k, (bw - 1) * s + k
        for q, bid in enumerate(idx):
            a, rem = divmod(int(bid), gh * gw)
            gy, gx = divmod(rem, gw)
            y0, x0 = gy * bh * s - p + big, gx * bw * s - p + big
            want = xp[a, :, y0:y0 + th, x0:x0 + tw].transpose(1, 2, 0)
            assert np.array_equal(got[q], want)


def test_scatter_gather_roundtrip_k1():
    r = synth.rng(24)
    x = synth.to_storage_bits(synth.normal(r, (1, 4, 8, 12)), "f32")
    idx = np.array([1, 2, 4], np.int32)
    packed = oracle.gather_halo(x, idx, 2, 3, 4, 4, 1, 1, 1, 0, 0)
    dst = synth.nan_canaries(r, x.shape, "f32")
    y = oracle.scatter_blocks(packed, idx, 2, 3, dst)
    sel = oracle.expand_mask(np.isin(np.arange(6), idx).reshape(1, 2, 3).astype(np.uint8), 4, 4)
    sel = np.broadcast_to(sel, x.shape)
    assert np.array_equal(y[sel], x[sel]) and np.array_equal(y[~sel], dst[~sel])


# ---------------------------------------------------------------- maxpool

def test_maxpool_golden_and_torch():
    x = np.arange(1, 17, dtype=np.float64).reshape(1, 1, 4, 4)
    assert np.array_equal(oracle.maxpool2d_dense(x, 3, 2, 1)[0, 0], _golden("maxpool3x3s2_4x4.txt"))
    r = synth.rng(25)
    x = r.standard_normal((2, 5, 13, 16))
    want = F.max_pool2d(torch.from_numpy(x), 3, 2, 1).numpy()
    assert np.array_equal(oracle.maxpool2d_dense(x, 3, 2, 1), want)


# ---------------------------------------------------------------- BN fold

def test_fold_bn_matches_unfused():
    r = synth.rng(26)
    cin, cout = 4, 6
    x = r.standard_normal((1, cin, 7, 9))
    w = r.standard_normal((cout, cin, 3, 3))
    cb = r.standard_normal(cout)
    g, be = r.uniform(0.5, 2, cout), r.standard_normal(cout)
    mu, var = r.standard_normal(cout), r.uniform(0.2, 3, cout)
    w2, b2 = oracle.fold_bn(w, cb, g, be, mu, var, 1e-5)
    y = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(cb), padding=1)
    y = F.batch_norm(y, torch.from_numpy(mu), torch.from_numpy(var), torch.from_numpy(g),
                     torch.from_numpy(be), training=False, eps=1e-5).numpy()
    got = oracle.conv2d_dense(x, w2, b2, None, 1, 1, False)
    np.testing.assert_allclose(got, y, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- network

def test_resnet_tables_match_torchvision_style_definition():
    t50, t18 = net.resnet_table(50), net.resnet_table(18)
    assert sum(l["kind"] == "conv" for l in t50) == 53
    assert sum(l["kind"] == "conv" for l in t18) == 20
    # MAC count of ResNet-50 at 224x224 is ~4.09 G (the published figure for the backbone,
    # without the classifier's 2 M)
    sh = net.shapes(t50, 224, 224)
    macs = sum(l["cin"] * l["cout"] * l["k"] ** 2 * sh[i][1] * sh[i][2]
               for i, l in enumerate(t50) if l["kind"] == "conv")
    assert abs(macs / 1e9 - 4.09) < 0.02
    sh18 = net.shapes(t18, 224, 224)
    macs18 = sum(l["cin"] * l["cout"] * l["k"] ** 2 * sh18[i][1] * sh18[i][2]
                 for i, l in enumerate(t18) if l["kind"] == "conv")
    assert abs(macs18 / 1e9 - 1.81) < 0.02
    assert sh[-1] == (2048, 7, 7) and sh18[-1] == (512, 7, 7)


def _torch_resnet_dense(table, folded, x_bits):
    """Library-routine reference: torch fp64 conv2d / max_pool2d / relu per layer with
    the storage rounding done by torch's own dtype conversions."""
    def st(t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    outs = []
    x = torch.from_numpy(synth.storage_to_f64(x_bits, "bf16"))
    for li, l in enumerate(table):
        src = x if l["src"] < 0 else outs[l["src"]]
        if l["kind"] == "pool":
            y = F.max_pool2d(src, l["k"], l["stride"], l["pad"])
        else:
            w = torch.from_numpy(synth.storage_to_f64(folded[li]["w_bits"], "bf16"))
            b = torch.from_numpy(folded[li]["bias"].astype(np.float64))
            y = F.conv2d(src, w, b, stride=l["stride"], padding=l["pad"])
            if l["res"] is not None:
                y = y + outs[l["res"]]
            if l["relu"]:
                y = torch.relu(y)
        outs.append(st(y))
    return outs


@pytest.mark.parametrize("depth", [18, 50])
def test_network_all_ones_equals_library_reference(depth):
    table = net.resnet_table(depth)
    folded = net.fold_params(table, net.make_params(table), "bf16")
    h, w = 64, 128
    x = synth.to_storage_bits(synth.normal(synth.rng(1), (1, 3, h, w)), "bf16")
    sh = net.shapes(table, h, w)
    prev = [np.zeros((1,) + s, np.uint16) for s in sh]
    bufs = net.frame(table, folded, x, np.ones((1, 2, 4), np.uint8), prev, "bf16")
    ref = _torch_resnet_dense(table, folded, x)
    for li in range(len(table)):
        got = oracle.value(bufs[li], "bf16")
        want = ref[li].numpy()
        # identical up to fp64 summation order before rounding: bf16 results agree
        # except for values sitting on a rounding boundary (1 ulp)
        bad = got != want
        assert bad.mean() < 1e-3, (li, bad.mean())
        np.testing.assert_allclose(got, want, rtol=2 ** -7, atol=1e-30)


def test_network_static_frame_bit_identical():
    """Frame 0 with the all-ones grid on X, frame 1 with the same X and a random grid:
    every layer's buffer equals frame 0's bit for bit (halos from copied neighbours
    hold exactly the values the dense network would read)."""
    table = net.resnet_table(18)
    folded = net.fold_params(table, net.make_params(table, bn_random=True), "bf16")
    h, w = 64, 128
    x = synth.to_storage_bits(synth.normal(synth.rng(1), (1, 3, h, w)), "bf16")
    sh = net.shapes(table, h, w)
    r = synth.rng(2)
    prev = [synth.nan_canaries(r, (1,) + s, "bf16") for s in sh]
    f0 = net.frame(table, folded, x, np.ones((1, 2, 4), np.uint8), prev, "bf16")
    m = np.array([[[1, 0, 1, 0], [0, 1, 1, 0]]], np.uint8)
    f1 = net.frame(table, folded, x, m, f0, "bf16")
    for a, b in zip(f0, f1):
        assert np.array_equal(a, b)
    # and a changed frame only changes executed blocks
    x2 = synth.to_storage_bits(synth.normal(synth.rng(9), (1, 3, h, w)), "bf16")
    f2 = net.frame(table, folded, x2, m, f0, "bf16")
    for (c, hh, ww), a, b in zip(sh, f0, f2):
        sel = np.broadcast_to(oracle.expand_mask(m, hh // 2, ww // 4), a.shape)
        assert np.array_equal(a[~sel], b[~sel])


@pytest.mark.parametrize("seed,shape,k,s,res,relu,p", [
    (700, (1, 5, 12, 16, 7), 3, 1, True, True, 0.4),
    (701, (2, 3, 16, 24, 4), 3, 2, False, True, 0.5),
    (702, (1, 8, 8, 8, 8), 1, 1, True, False, 0.0),      # no block
    (703, (1, 4, 14, 14, 6), 7, 2, False, True, 1.0),    # every block, stem-like
])
def test_only_active_mode_equals_dense_then_select(seed, shape, k, s, res, relu, p):
    """The only-active mode computes the same points with the same arithmetic and skips
    the rest: bit for bit the dense-then-select result, whatever the mask."""
    n, cin, h, w, cout = shape
    r = synth.rng(seed)
    pad = k // 2
    ho, wo = oracle.out_size(h, k, s, pad), oracle.out_size(w, k, s, pad)
    gh, gw = (2, 2) if ho % 2 == 0 and wo % 2 == 0 else (1, 1)
    x = synth.to_storage_bits(synth.normal(r, (n, cin, h, w)), "bf16")
    wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), "bf16")
    bias = synth.normal(r, cout, 0.1).astype(np.float32)
    rb = synth.to_storage_bits(synth.normal(r, (n, cout, ho, wo)), "bf16") if res else None
    prev = synth.nan_canaries(r, (n, cout, ho, wo), "bf16")
    mask = synth.bernoulli_mask(r, n, gh, gw, p) if p not in (0.0, 1.0) else np.full((n, gh, gw), int(p), np.uint8)
    a = oracle.sparse_conv2d(x, wt, mask, prev, "bf16", s, pad, bias, rb, relu)
    b = oracle.sparse_conv2d_active(x, wt, mask, prev, "bf16", s, pad, bias, rb, relu)
    assert np.array_equal(a, b)
