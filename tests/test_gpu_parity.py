"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same
seeded inputs. Index, copied blocks, gather/scatter and max pooling must match bit for
bit; convolution outputs on active blocks within max abs-rel 1e-4 (fp32) / 2e-2
(bf16, fp16), and bit for bit when every partial sum is exact (small integers)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import TOL, block_select, from_dev, max_abs_rel, to_dev, weights_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B(gpu):
    from paper_2108_09376_amd import bc
    return bc


def _index(B, mask_np, sentinel=-7):
    n, gh, gw = mask_np.shape
    m = torch.from_numpy(mask_np).cuda()
    idx = torch.full((n * gh * gw + 5,), sentinel, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    hc = B.bc_build_block_index(m, n, (gh, gw), idx, cnt, h_count=True)
    return idx, cnt, hc


# ------------------------------------------------------------------ a1: index

@pytest.mark.parametrize("n,gh,gw,p", [(1, 8, 16, 0.3), (1, 8, 16, 0.0), (1, 8, 16, 1.0),
                                       (3, 8, 16, 0.5), (1, 1, 1, 1.0), (1, 37, 29, 0.4),
                                       (2, 512, 1024, 0.3)])
def test_block_index_bit_exact(B, n, gh, gw, p):
    mask = synth.bernoulli_mask(synth.rng(40 + gh), n, gh, gw, p)
    mask[mask != 0] = synth.rng(41).integers(1, 256, int(mask.sum()))  # any nonzero byte executes
    idx, cnt, hc = _index(B, mask)
    want, wc = oracle.block_index(mask)
    got = idx.cpu().numpy()
    assert hc == wc and int(cnt.item()) == wc
    assert np.array_equal(got[:wc], want)
    assert (got[wc:] == -7).all()          # entries at and beyond the count are untouched


# ------------------------------------------------------------------ a2 / a5: gather, scatter

@pytest.mark.parametrize("dtype,nhwc,c", [("bf16", True, 64), ("bf16", True, 12), ("f16", True, 24),
                                          ("f32", True, 8), ("f32", False, 16), ("f32", False, 3),
                                          ("bf16", True, 520)])
@pytest.mark.parametrize("k,s,p", [(3, 1, 1), (1, 1, 0), (3, 2, 1), (7, 2, 3)])
def test_gather_halo_bit_exact(B, dtype, nhwc, c, k, s, p):
    r = synth.rng(50 + c + k)
    h, w, gh, gw = 32, 48, 2, 3
    x = synth.to_storage_bits(synth.normal(r, (2, c, h, w)), dtype)
    mask = synth.bernoulli_mask(r, 2, gh, gw, 0.5)
    idx_np, cnt_np = oracle.block_index(mask)
    bh, bw = oracle.out_size(h, k, s, p) // gh, oracle.out_size(w, k, s, p) // gw
    pad_value = -np.inf if k == 3 else 0.0
    pad_bits = synth.to_storage_bits(np.array([pad_value], np.float32), dtype)[0]
    want = oracle.gather_halo(x, idx_np, gh, gw, bh, bw, k, k, s, p, pad_bits)
    idx, cnt, _ = _index(B, mask)
    th, tw = (bh - 1) * s + k, (bw - 1) * s + k
    cap = idx.numel()
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dtype]
    packed = torch.zeros((cap, th, tw, c), dtype=tdt, device="cuda")
    sent = from_dev(packed[:1].permute(0, 3, 1, 2), nhwc=False)  # all-zero bits
    B.bc_gather_halo(to_dev(x, dtype, nhwc), B.BC_NHWC if nhwc else B.BC_NCHW, (gh, gw),
                     (k, k, s, p, 0), pad_value, idx, cnt, packed)
    got = packed.cpu()
    got = got.view(torch.int16).numpy().view(np.uint16) if dtype != "f32" else got.numpy().view(np.uint32)
    assert np.array_equal(got[:cnt_np], want)
    assert not got[cnt_np:].any() and not sent.any()


@pytest.mark.parametrize("dtype,nhwc,c", [("bf16", True, 64), ("bf16", True, 12), ("f32", False, 16),
                                          ("bf16", True, 520)])
def test_scatter_blocks_bit_exact_and_untouched(B, dtype, nhwc, c):
    r = synth.rng(60 + c)
    h, w, gh, gw = 32, 48, 4, 3
    dst = synth.nan_canaries(r, (2, c, h, w), dtype)
    mask = synth.bernoulli_mask(r, 2, gh, gw, 0.4)
    idx_np, cnt_np = oracle.block_index(mask)
    bh, bw = h // gh, w // gw
    packed_bits = synth.to_storage_bits(synth.normal(r, (cnt_np, bh, bw, c)), dtype)
    want = oracle.scatter_blocks(packed_bits, idx_np, gh, gw, dst)
    idx, cnt, _ = _index(B, mask)
    cap = idx.numel()
    full = np.zeros((cap, bh, bw, c), packed_bits.dtype)
    full[:cnt_np] = packed_bits
    tdt = {"bf16": torch.bfloat16, "f32": torch.float32}[dtype]
    if dtype == "f32":
        pk = torch.from_numpy(full.view(np.float32)).cuda()
    else:
        pk = torch.from_numpy(full.view(np.int16)).view(tdt).cuda()
    d = to_dev(dst, dtype, nhwc)
    B.bc_scatter_blocks(pk, idx, cnt, (gh, gw), d, B.BC_NHWC if nhwc else B.BC_NCHW)
    assert np.array_equal(from_dev(d, nhwc), want)


def test_gather_scatter_roundtrip(B):
    r = synth.rng(70)
    x = synth.to_storage_bits(synth.normal(r, (1, 32, 64, 96)), "bf16")
    mask = synth.bernoulli_mask(r, 1, 4, 6, 0.5)
    idx, cnt, hc = _index(B, mask)
    xd = to_dev(x, "bf16")
    packed = torch.empty((idx.numel(), 16, 16, 32), dtype=torch.bfloat16, device="cuda")
    B.bc_gather_halo(xd, B.BC_NHWC, (4, 6), (1, 1, 1, 0, 0), 0.0, idx, cnt, packed)
    dst_bits = synth.nan_canaries(r, x.shape, "bf16")
    d = to_dev(dst_bits, "bf16")
    B.bc_scatter_blocks(packed, idx, cnt, (4, 6), d, B.BC_NHWC)
    got = from_dev(d)
    sel = block_select(mask, x.shape)
    assert np.array_equal(got[sel], x[sel]) and np.array_equal(got[~sel], dst_bits[~sel])


# ------------------------------------------------------------------ a3/a4: conv, fp32 path

def test_conv_f32_nchw_two_frames(B):
    """Single 3x3 conv, stride 1, pad 1, NCHW fp32, Cin=Cout=16, 64x128 map, 8x8 blocks
    on an 8x16 grid, Bernoulli(0.25) masks; frame 1 runs on frame 0's output."""
    r = synth.rng(synth.SEED_WEIGHT0)
    w = synth.to_storage_bits(synth.he_normal(r, 16, 16, 3, 3), "f32")
    x0 = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_INPUT), (1, 16, 64, 128)), "f32")
    x1 = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_INPUT + 100), (1, 16, 64, 128)), "f32")
    prev = synth.to_storage_bits(synth.normal(synth.rng(synth.SEED_PREV), (1, 16, 64, 128)), "f32")
    bias = synth.normal(synth.rng(7), 16)
    masks = [synth.bernoulli_mask(synth.rng(synth.SEED_MASK0 + t), 1, 8, 16, 0.25) for t in range(2)]
    wd = weights_dev(w, "f32", nhwc=False)
    bd = torch.from_numpy(bias).cuda()
    out = to_dev(prev, "f32", nhwc=False)
    want = prev
    for t, (x, m) in enumerate(zip([x0, x1], masks)):
        idx, cnt, _ = _index(B, m)
        B.bc_sparse_conv2d((3, 3, 1, 1, 1), to_dev(x, "f32", nhwc=False), B.BC_NCHW, wd, bd, None,
                           out, (8, 16), idx, cnt)
        want = oracle.sparse_conv2d(x, w, m, want, "f32", 1, 1, bias, None, True)
        got = from_dev(out, nhwc=False)
        sel = block_select(m, got.shape)
        assert np.array_equal(got[~sel], want[~sel])
        err = max_abs_rel(oracle.value(got[sel], "f32"), oracle.value(want[sel], "f32"))
        assert err <= TOL["f32"], (t, err)
        want = got  # the next frame's previous buffer is what the GPU holds (bitwise checked)


# ------------------------------------------------------------------ a3/a4: conv, matrix cores

CASES = [
    # cin, cout, h(in), w(in), gh, gw, k, s, relu, residual, frac
    (64, 64, 64, 128, 2, 4, 3, 1, True, False, 0.5),     # 32x32 blocks, 3x3
    (64, 128, 64, 128, 8, 16, 3, 1, True, True, 0.4),   # 8x8 blocks, P=2 patches/tile
    (32, 64, 32, 64, 8, 16, 3, 1, False, True, 0.3),    # 4x4 blocks, P=8
    (256, 64, 32, 64, 4, 8, 1, 1, True, False, 0.5),    # 1x1
    (64, 256, 32, 64, 4, 8, 1, 1, True, True, 0.6),     # 1x1 + residual
    (64, 128, 64, 128, 4, 8, 3, 2, True, False, 0.5),   # 3x3/2
    (128, 256, 64, 128, 4, 8, 1, 2, False, False, 0.5), # 1x1/2 downsample
    (3, 64, 128, 256, 2, 4, 7, 2, True, False, 0.5),    # 7x7/2 stem form (Cin=3)
    (8, 64, 64, 64, 2, 2, 7, 2, True, False, 0.75),     # 7x7/2, Cin=8
    (40, 64, 48, 80, 3, 5, 3, 1, True, False, 0.6),     # Cin not a multiple of 32: ragged K chunk
    (64, 192, 64, 64, 4, 4, 5, 1, True, True, 0.5),     # 5x5, Cout=192
    (128, 128, 48, 48, 12, 12, 3, 1, True, True, 0.33), # 4x4 blocks, ragged tail of patches
    (512, 64, 32, 64, 4, 8, 3, 1, True, True, 0.5),     # 16 chunks on 32 tiles: K split in 4
    (3, 64, 32, 64, 2, 4, 1, 1, True, False, 0.5),      # 1x1 with Cin=3 (stem form)
    (5, 64, 32, 64, 2, 4, 3, 1, True, True, 0.5),       # Cin=5: 8 padded channels per pixel
    (3, 64, 64, 64, 2, 2, 7, 1, True, False, 0.5),      # 7x7/1 stem form (unaligned rows)
    (3, 64, 512, 1024, 16, 32, 7, 2, True, False, 0.9), # stem form, more active tiles than
                                                        # resident workgroups: several each
    (3, 64, 64, 63, 2, 4, 7, 2, True, False, 0.5),      # stem form, odd input width: pixels
                                                        # staged one channel at a time
    (1024, 64, 16, 32, 2, 4, 1, 1, True, True, 0.5),    # 1x1, 32 chunks on a few tiles: K split
                                                        # in three (11, 11, 10 chunks)
    (256, 128, 64, 128, 8, 16, 3, 1, True, True, 0.3),  # 3x3, 8 chunks on 256 tiles: K split in
                                                        # two, nine-tap stages
    (520, 64, 16, 32, 2, 4, 1, 1, True, True, 0.5),     # 1x1, 17 chunks on few tiles: K halves
                                                        # over two wave groups (9 and 8 chunks)
    (744, 128, 16, 32, 2, 4, 1, 1, False, False, 0.6),  # 1x1, 24 chunks, the last a quarter
                                                        # full, two wave groups
    (512, 64, 32, 64, 2, 4, 1, 2, True, True, 0.5),     # 1x1/2, 16 chunks on few tiles: two
                                                        # wave groups at stride 2
]


def _conv_case(B, dtype, case, seed, integer=False, mask=None, prev=None, n=1):
    cin, cout, h, w, gh, gw, k, s, relu, has_res, frac = case
    r = synth.rng(seed)
    p = k // 2
    ho, wo = oracle.out_size(h, k, s, p), oracle.out_size(w, k, s, p)
    if integer:
        xv = synth.small_ints(r, (n, cin, h, w), -2, 2)
        wv = synth.small_ints(r, (cout, cin, k, k), -1, 1)
        bias = synth.small_ints(r, cout, -3, 3)
        res = synth.small_ints(r, (n, cout, ho, wo), -4, 4) if has_res else None
    else:
        xv = synth.normal(r, (n, cin, h, w))
        wv = synth.he_normal(r, cout, cin, k, k)
        bias = synth.normal(r, cout, 0.1)
        res = synth.normal(r, (n, cout, ho, wo)) if has_res else None
    x = synth.to_storage_bits(xv, dtype)
    wt = synth.to_storage_bits(wv, dtype)
    rb = None if res is None else synth.to_storage_bits(res, dtype)
    if prev is None:
        prev = synth.nan_canaries(r, (n, cout, ho, wo), dtype)
    if mask is None:
        mask = np.concatenate([synth.frac_mask(seed + 1 + i, gh, gw, frac) for i in range(n)])
    want = oracle.sparse_conv2d(x, wt, mask, prev, dtype, s, p, bias, rb, relu)
    idx, cnt, _ = _index(B, mask)
    out = to_dev(prev, dtype)
    B.bc_sparse_conv2d((k, k, s, p, int(relu)), to_dev(x, dtype), B.BC_NHWC, weights_dev(wt, dtype),
                       torch.from_numpy(bias).cuda(), None if rb is None else to_dev(rb, dtype), out,
                       (gh, gw), idx, cnt)
    got = from_dev(out)
    return got, want, mask, prev


@pytest.mark.parametrize("case", CASES, ids=[f"c{c[0]}-{c[1]}_k{c[6]}s{c[7]}_g{c[4]}x{c[5]}" for c in CASES])
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_conv_mfma_parity(B, dtype, case):
    got, want, mask, prev = _conv_case(B, dtype, case, seed=80)
    sel = block_select(mask, got.shape)
    assert np.array_equal(got[~sel], prev[~sel])          # copied blocks: bit for bit
    err = max_abs_rel(oracle.value(got[sel], dtype), oracle.value(want[sel], dtype))
    assert err <= TOL[dtype], err


@pytest.mark.parametrize("case", CASES, ids=[f"c{c[0]}-{c[1]}_k{c[6]}s{c[7]}_g{c[4]}x{c[5]}" for c in CASES])
def test_conv_mfma_integer_exact(B, case):
    """Small-integer operands: every partial sum is exact in fp32 and every result is
    exact in bf16, so active blocks must match the oracle bit for bit (pins indexing,
    halo, stride, padding, residual and bias wiring with zero tolerance)."""
    got, want, mask, prev = _conv_case(B, "bf16", case, seed=90, integer=True)
    assert np.array_equal(got, want)


def test_conv_all_zero_mask_touches_nothing(B):
    case = (64, 64, 64, 128, 2, 4, 3, 1, True, True, 0.0)
    got, want, mask, prev = _conv_case(B, "bf16", case, seed=91, mask=np.zeros((1, 2, 4), np.uint8))
    assert np.array_equal(got, prev)


def test_conv_all_ones_equals_dense_call(B):
    """A full mask through the index equals the index-free full-frame call bit for bit."""
    case = (64, 128, 64, 128, 8, 16, 3, 1, True, True, 1.0)
    got, want, mask, prev = _conv_case(B, "bf16", case, seed=92, mask=np.ones((1, 8, 16), np.uint8))
    cin, cout, h, w, gh, gw, k, s, relu, _, _ = case
    r = synth.rng(92)
    # same draws as _conv_case
    x = synth.to_storage_bits(synth.normal(r, (1, cin, h, w)), "bf16")
    wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), "bf16")
    bias = synth.normal(r, cout, 0.1)
    rb = synth.to_storage_bits(synth.normal(r, (1, cout, h, w)), "bf16")
    out = torch.empty((1, h, w, cout), dtype=torch.bfloat16, device="cuda")
    B.bc_sparse_conv2d((3, 3, 1, 1, 1), to_dev(x, "bf16"), B.BC_NHWC, weights_dev(wt, "bf16"),
                       torch.from_numpy(bias).cuda(), to_dev(rb, "bf16"), out, (gh, gw), None, None)
    assert np.array_equal(from_dev(out), got)
    assert max_abs_rel(oracle.value(got, "bf16"), oracle.value(want, "bf16")) <= TOL["bf16"]


@pytest.mark.parametrize("case", [CASES[0], CASES[2], CASES[3], CASES[7], CASES[12], CASES[11]],
                         ids=["3x3_32px", "3x3_4px_P8", "1x1_two_chunks", "stem", "split_k", "ragged_tail"])
def test_conv_mfma_batch(B, case):
    """Three images in one call, each with its own execution grid: block ids span the
    images (id = (img * Gh + gy) * Gw + gx)."""
    got, want, mask, prev = _conv_case(B, "bf16", case, seed=95, n=3)
    sel = block_select(mask, got.shape)
    assert np.array_equal(got[~sel], prev[~sel])
    assert max_abs_rel(oracle.value(got[sel], "bf16"), oracle.value(want[sel], "bf16")) <= TOL["bf16"]


@pytest.mark.parametrize("case", [CASES[1], CASES[2], CASES[5], CASES[7], CASES[-1]])
def test_conv_active_bits_independent_of_mask(B, case):
    """An active block's bits do not depend on which other blocks are active."""
    got_sparse, _, mask, _ = _conv_case(B, "bf16", case, seed=93)
    full = np.ones_like(mask)
    got_full, _, _, _ = _conv_case(B, "bf16", case, seed=93, mask=full)
    sel = block_select(mask, got_sparse.shape)
    assert np.array_equal(got_sparse[sel], got_full[sel])


# ------------------------------------------------------------------ a6: max pooling

@pytest.mark.parametrize("dtype,nhwc,k,s,p", [("bf16", True, 3, 2, 1), ("f16", True, 3, 2, 1),
                                               ("f32", False, 3, 2, 1), ("bf16", True, 2, 2, 0),
                                               ("bf16", True, 5, 2, 2)])
def test_maxpool_bit_exact(B, dtype, nhwc, k, s, p):
    """The 3x3 window (every tap requested up front, clamped) and other windows (a loop
    over the taps), border blocks included."""
    r = synth.rng(100)
    c, h, w, gh, gw = 64 if nhwc else 16, 64, 128, 4, 8
    x = synth.to_storage_bits(synth.normal(r, (1, c, h, w)), dtype)
    prev = synth.nan_canaries(r, (1, c, h // 2, w // 2), dtype)
    mask = synth.frac_mask(101, gh, gw, 0.4)
    want = oracle.sparse_maxpool2d(x, mask, prev, dtype, k, s, p)
    idx, cnt, _ = _index(B, mask)
    out = to_dev(prev, dtype, nhwc)
    B.bc_sparse_maxpool2d((k, k, s, p, 0), to_dev(x, dtype, nhwc), B.BC_NHWC if nhwc else B.BC_NCHW,
                          out, (gh, gw), idx, cnt)
    assert np.array_equal(from_dev(out, nhwc), want)


# ------------------------------------------------------------------ error paths with real memory

def test_errors_leave_buffers_untouched(B):
    x = torch.zeros((1, 64, 128, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((64, 3, 3, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.full((1, 64, 128, 64), 3.0, dtype=torch.bfloat16, device="cuda")
    idx = torch.zeros(128, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.BCError) as e:
        B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, out, (7, 16), idx, cnt)
    assert e.value.status == B.BC_ERR_NOT_DIVISIBLE
    with pytest.raises(B.BCError) as e:
        B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, x, (8, 16), idx, cnt)
    assert e.value.status == B.BC_ERR_ALIAS
    with pytest.raises(B.BCError) as e:
        B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, out, (8, 16), idx[:100], cnt)
    assert e.value.status == B.BC_ERR_CAPACITY
    buf = B.Buffer(out, B.BC_NHWC)
    with pytest.raises(B.BCError) as e:
        B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, out, (8, 16), idx, cnt)
    assert e.value.status == B.BC_ERR_UNINITIALIZED
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
    B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, out, (8, 16), None, None)
    assert buf.valid == 1
    B.bc_sparse_conv2d((3, 3, 1, 1, 1), x, B.BC_NHWC, w, None, None, out, (8, 16), idx, cnt)
    torch.cuda.synchronize()
    assert bool((out == 0).all())
    buf.release()


# ------------------------------------------------------------------ a3: seeded random sweep

def _mask_pattern(kind, gh, gw, r):
    """Execution grids of one image: Bernoulli(0.4), none, one block, checkerboard, the
    border ring, every block."""
    y, x = np.mgrid[0:gh, 0:gw]
    m = {"bern": r.random((gh, gw)) < 0.4,
         "empty": np.zeros((gh, gw), bool),
         "one": (y == r.integers(gh)) & (x == r.integers(gw)),
         "checker": (y + x) % 2 == 0,
         "border": (y == 0) | (y == gh - 1) | (x == 0) | (x == gw - 1),
         "full": np.ones((gh, gw), bool)}[kind]
    return m.astype(np.uint8)[None]


def _random_cases(count, seed=2108):
    """Seeded layer configurations inside the supported space (Cout a multiple of 64;
    Cin a multiple of 8, or the few-channel stem form; kernel edge 1, 3, 5 or 7;
    stride 1 or 2; block edges 2-32 px, square or not, whose width divides 64), each
    with a mask pattern and a storage format. The dense oracle's work stays under
    about 1 GFLOP per case."""
    r = np.random.default_rng(seed)
    kinds = ["bern", "empty", "one", "checker", "border", "full"]
    out = []
    while len(out) < count:
        k = int(r.choice([1, 3, 3, 3, 5, 7]))
        s = int(r.choice([1, 2]))
        if k == 7 or (k in (3, 5) and r.random() < 0.2):
            cin = int(r.choice([3, 4]))                          # stem form
        elif k == 1 and r.random() < 0.15:
            cin = int(r.choice([3, 5]))
        else:
            cin = int(8 * r.integers(1, 41)) if r.random() < 0.6 else int(r.choice([64, 128, 256]))
        cout = int(64 * r.integers(1, 4))
        bw = int(r.choice([4, 8, 16, 32] if k <= 3 else [4, 8, 16]))
        bh = int(r.choice([b for b in (bw // 2, bw, 2 * bw) if 2 <= b <= 32]))
        gh, gw = int(r.integers(1, 5)), int(r.integers(1, 6))
        ho, wo = gh * bh, gw * bw
        if ho > 96 or wo > 160:
            continue
        if 2.0 * cin * cout * k * k * ho * wo > 1e9:
            continue
        out.append(dict(cin=cin, cout=cout, h=ho * s, w=wo * s, gh=gh, gw=gw, k=k, s=s,
                        relu=bool(r.random() < 0.5), res=bool(r.random() < 0.5),
                        mask=kinds[len(out) % len(kinds)], dtype=("bf16", "f16")[len(out) % 2],
                        seed=int(r.integers(1 << 30))))
    return out


RANDOM_CASES = _random_cases(36)


@pytest.mark.parametrize("c", RANDOM_CASES,
                         ids=[f"r{i}_c{c['cin']}-{c['cout']}_k{c['k']}s{c['s']}_b{c['h'] // c['s'] // c['gh']}x"
                              f"{c['w'] // c['s'] // c['gw']}_{c['mask']}_{c['dtype']}"
                              for i, c in enumerate(RANDOM_CASES)])
def test_conv_random_shapes_integer_exact(B, c):
    """Small-integer operands on seeded random shapes: every partial sum is an integer
    exact in fp32, so whatever the plan (tile shape, K split, stage grouping, stem or
    general form) the output must equal the oracle's byte for byte, copied blocks
    (NaN canaries) included."""
    r = synth.rng(c["seed"])
    mask = _mask_pattern(c["mask"], c["gh"], c["gw"], r)
    case = (c["cin"], c["cout"], c["h"], c["w"], c["gh"], c["gw"], c["k"], c["s"], c["relu"],
            c["res"], 0.0)
    got, want, _, _ = _conv_case(B, c["dtype"], case, seed=c["seed"], integer=True, mask=mask)
    assert np.array_equal(got, want)


def _random_window_cases(count, seed, pool):
    """Seeded window geometries (edge 1-7, stride 1 or 2, pad up to edge / 2), block
    edges 2-16 px of the output, grids up to 4 x 5, channel counts and storage formats
    (pooling: 16-bit channels-last with C a multiple of 8, or fp32 channels-first; the
    gather takes any element size, layout and C), each with one of the mask patterns."""
    r = np.random.default_rng(seed)
    kinds = ["bern", "empty", "one", "checker", "border", "full"]
    fmts = ([("bf16", True), ("f16", True), ("f32", False)] if pool else
            [("bf16", True), ("f16", True), ("f32", False), ("f32", True)])
    out = []
    while len(out) < count:
        k = int(r.integers(1, 8))
        s = int(r.choice([1, 2]))
        p = int(r.integers(0, k // 2 + 1))
        bh, bw = int(r.choice([2, 4, 8, 16])), int(r.choice([2, 4, 8, 16]))
        gh, gw = int(r.integers(1, 5)), int(r.integers(1, 6))
        ho, wo = gh * bh, gw * bw
        # input size giving exactly this output: (h + 2p - k) // s + 1 == ho
        h, w = (ho - 1) * s + k - 2 * p, (wo - 1) * s + k - 2 * p
        if h < 1 or w < 1:
            continue
        dtype, nhwc = fmts[len(out) % len(fmts)]
        c = int(8 * r.integers(1, 9)) if pool and nhwc else int(r.integers(1, 41))
        out.append(dict(k=k, s=s, p=p, h=h, w=w, gh=gh, gw=gw, c=c, dtype=dtype, nhwc=nhwc,
                        mask=kinds[len(out) % len(kinds)], seed=int(r.integers(1 << 30))))
    return out


POOL_CASES = _random_window_cases(24, 2109, pool=True)


@pytest.mark.parametrize("c", POOL_CASES,
                         ids=[f"r{i}_k{c['k']}s{c['s']}p{c['p']}_{c['h']}x{c['w']}_g{c['gh']}x{c['gw']}_"
                              f"c{c['c']}_{c['dtype']}{'' if c['nhwc'] else '_nchw'}_{c['mask']}"
                              for i, c in enumerate(POOL_CASES)])
def test_maxpool_random_shapes_bit_exact(B, c):
    """Max pooling on seeded random windows and block grids: active blocks equal the
    oracle's dense-then-select maximum, copied blocks keep their NaN canaries."""
    r = synth.rng(c["seed"])
    dtype, nhwc = c["dtype"], c["nhwc"]
    x = synth.to_storage_bits(synth.normal(r, (1, c["c"], c["h"], c["w"])), dtype)
    ho = oracle.out_size(c["h"], c["k"], c["s"], c["p"])
    wo = oracle.out_size(c["w"], c["k"], c["s"], c["p"])
    prev = synth.nan_canaries(r, (1, c["c"], ho, wo), dtype)
    mask = _mask_pattern(c["mask"], c["gh"], c["gw"], r)
    want = oracle.sparse_maxpool2d(x, mask, prev, dtype, c["k"], c["s"], c["p"])
    idx, cnt, _ = _index(B, mask)
    out = to_dev(prev, dtype, nhwc)
    B.bc_sparse_maxpool2d((c["k"], c["k"], c["s"], c["p"], 0), to_dev(x, dtype, nhwc),
                          B.BC_NHWC if nhwc else B.BC_NCHW, out, (c["gh"], c["gw"]), idx, cnt)
    assert np.array_equal(from_dev(out, nhwc), want)


GATHER_CASES = _random_window_cases(24, 2110, pool=False)


@pytest.mark.parametrize("c", GATHER_CASES,
                         ids=[f"r{i}_k{c['k']}s{c['s']}p{c['p']}_{c['h']}x{c['w']}_g{c['gh']}x{c['gw']}_"
                              f"c{c['c']}_{c['dtype']}{'' if c['nhwc'] else '_nchw'}_{c['mask']}"
                              for i, c in enumerate(GATHER_CASES)])
def test_gather_random_shapes_bit_exact(B, c):
    """Standalone halo gather on seeded random windows and block grids: every active
    block's tile equals the oracle's, out-of-image taps carry the pad value, and the
    slots past the active count stay untouched."""
    r = synth.rng(c["seed"])
    dtype, nhwc, k, s, p = c["dtype"], c["nhwc"], c["k"], c["s"], c["p"]
    gh, gw = c["gh"], c["gw"]
    x = synth.to_storage_bits(synth.normal(r, (1, c["c"], c["h"], c["w"])), dtype)
    mask = _mask_pattern(c["mask"], gh, gw, r)
    idx_np, cnt_np = oracle.block_index(mask)
    bh = oracle.out_size(c["h"], k, s, p) // gh
    bw = oracle.out_size(c["w"], k, s, p) // gw
    pad_value = -np.inf if k % 2 else 0.0
    pad_bits = synth.to_storage_bits(np.array([pad_value], np.float32), dtype)[0]
    want = oracle.gather_halo(x, idx_np, gh, gw, bh, bw, k, k, s, p, pad_bits)
    idx, cnt, _ = _index(B, mask)
    th, tw = (bh - 1) * s + k, (bw - 1) * s + k
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dtype]
    packed = torch.zeros((idx.numel(), th, tw, c["c"]), dtype=tdt, device="cuda")
    B.bc_gather_halo(to_dev(x, dtype, nhwc), B.BC_NHWC if nhwc else B.BC_NCHW, (gh, gw),
                     (k, k, s, p, 0), pad_value, idx, cnt, packed)
    got = packed.cpu()
    got = got.view(torch.int16).numpy().view(np.uint16) if dtype != "f32" else got.numpy().view(np.uint32)
    assert np.array_equal(got[:cnt_np], want)
    assert not got[cnt_np:].any()


SCATTER_CASES = _random_window_cases(16, 2111, pool=False)


@pytest.mark.parametrize("c", SCATTER_CASES,
                         ids=[f"r{i}_g{c['gh']}x{c['gw']}_c{c['c']}_{c['dtype']}"
                              f"{'' if c['nhwc'] else '_nchw'}_{c['mask']}"
                              for i, c in enumerate(SCATTER_CASES)])
def test_scatter_random_shapes_bit_exact(B, c):
    """Standalone scatter on seeded random block grids, block edges, channel counts and
    formats: active blocks take the packed tiles, every other element keeps its NaN
    canary bit for bit."""
    r = synth.rng(c["seed"])
    dtype, nhwc, gh, gw = c["dtype"], c["nhwc"], c["gh"], c["gw"]
    h = oracle.out_size(c["h"], c["k"], c["s"], c["p"])
    w = oracle.out_size(c["w"], c["k"], c["s"], c["p"])
    bh, bw = h // gh, w // gw
    dst = synth.nan_canaries(r, (1, c["c"], h, w), dtype)
    mask = _mask_pattern(c["mask"], gh, gw, r)
    idx_np, cnt_np = oracle.block_index(mask)
    packed_bits = synth.to_storage_bits(synth.normal(r, (cnt_np, bh, bw, c["c"])), dtype)
    want = oracle.scatter_blocks(packed_bits, idx_np, gh, gw, dst)
    idx, cnt, _ = _index(B, mask)
    full = np.zeros((idx.numel(), bh, bw, c["c"]), packed_bits.dtype)
    full[:cnt_np] = packed_bits
    if dtype == "f32":
        pk = torch.from_numpy(full.view(np.float32)).cuda()
    else:
        tdt = {"bf16": torch.bfloat16, "f16": torch.float16}[dtype]
        pk = torch.from_numpy(full.view(np.int16)).view(tdt).cuda()
    d = to_dev(dst, dtype, nhwc)
    B.bc_scatter_blocks(pk, idx, cnt, (gh, gw), d, B.BC_NHWC if nhwc else B.BC_NCHW)
    assert np.array_equal(from_dev(d, nhwc), want)
