"""GPU parity of the decoder-side steps of the segmentation network (Section 4, the
SwiftNet-style decoder; Section 3.4, information gain) through the C ABI against the
oracle on the same seeded inputs:

* block-sparse upsample-and-add: copied blocks bit for bit, executed blocks within
  max abs-rel 2e-2 (bf16, fp16) / 1e-4 (fp32) of the fp64 oracle, rounded once;
* information gain on channels-last 16-bit score maps whose first `classes` channels
  are the class scores (the rest padding that must never be read): within 1e-4 of the
  fp64 oracle on the same decoded values."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import policy as P
from tests._util import TOL, block_select, from_dev, max_abs_rel, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B(gpu):
    from paper_2108_09376_amd import bc
    return bc


def _index(B, mask_np):
    n, gh, gw = mask_np.shape
    m = torch.from_numpy(mask_np).cuda()
    idx = torch.full((n * gh * gw + 3,), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    B.bc_build_block_index(m, n, (gh, gw), idx, cnt)
    return idx, cnt


def _check_merge(got, want, mask, dtype):
    sel = block_select(mask, want.shape)
    assert np.array_equal(got[~sel], want[~sel]), "copied blocks changed"
    g, w = oracle.value(got[sel], dtype), oracle.value(want[sel], dtype)
    assert max_abs_rel(g, w) <= TOL[dtype]


# ------------------------------------------------------------------ upsample + add

@pytest.mark.parametrize("dtype,nhwc,n,c,hc,wc,grid,p,skip,relu", [
    ("bf16", True, 1, 128, 32, 64, (8, 16), 0.3, True, False),    # 8x8-pixel blocks
    ("bf16", True, 2, 24, 20, 28, (4, 7), 0.5, True, True),       # 10x8 blocks, 3 vectors/px
    ("f16", True, 1, 8, 15, 21, (3, 7), 0.6, False, False),       # 10x6 blocks, ragged tail
    ("bf16", True, 1, 520, 8, 16, (2, 4), 0.5, True, False),      # 65 vectors per pixel
    ("bf16", True, 1, 64, 1, 1, (1, 1), 1.0, True, True),         # 1x1 coarse: all edges
    ("f32", False, 2, 16, 24, 32, (4, 8), 0.4, True, True),
    ("f32", False, 1, 3, 7, 9, (7, 9), 0.5, False, False),        # 2x2 blocks
])
def test_upsample_add_parity(B, dtype, nhwc, n, c, hc, wc, grid, p, skip, relu):
    r = synth.rng(300 + c + hc)
    gh, gw = grid
    coarse = synth.to_storage_bits(synth.normal(r, (n, c, hc, wc)), dtype)
    sk = synth.to_storage_bits(synth.normal(r, (n, c, 2 * hc, 2 * wc)), dtype) if skip else None
    prev = synth.nan_canaries(r, (n, c, 2 * hc, 2 * wc), dtype)
    mask = synth.bernoulli_mask(r, n, gh, gw, p)
    want = oracle.sparse_upsample_add(coarse, sk, mask, prev, dtype, relu)
    idx, cnt = _index(B, mask)
    out = to_dev(prev, dtype, nhwc)
    lay = B.BC_NHWC if nhwc else B.BC_NCHW
    B.bc_sparse_upsample_add(to_dev(coarse, dtype, nhwc), lay,
                             to_dev(sk, dtype, nhwc) if skip else None, out, grid, int(relu),
                             idx, cnt)
    _check_merge(from_dev(out, nhwc), want, mask, dtype)


def test_upsample_add_full_size(B):
    """The largest merge of the decoder at 2048x1024: 128 channels, 128x256 -> 256x512,
    32x32-pixel blocks of the 8x16 grid, 30 % of them executed."""
    r = synth.rng(310)
    dtype, n, c, hc, wc, gh, gw = "bf16", 1, 128, 128, 256, 8, 16
    coarse = synth.to_storage_bits(synth.normal(r, (n, c, hc, wc)), dtype)
    sk = synth.to_storage_bits(synth.normal(r, (n, c, 2 * hc, 2 * wc)), dtype)
    prev = synth.nan_canaries(r, (n, c, 2 * hc, 2 * wc), dtype)
    mask = synth.frac_mask(311, gh, gw, 0.3)
    want = oracle.sparse_upsample_add(coarse, sk, mask, prev, dtype, True)
    idx, cnt = _index(B, mask)
    out = to_dev(prev, dtype)
    B.bc_sparse_upsample_add(to_dev(coarse, dtype), B.BC_NHWC, to_dev(sk, dtype), out, (gh, gw), 1,
                             idx, cnt)
    _check_merge(from_dev(out), want, mask, dtype)


def test_upsample_add_every_block_and_none(B):
    r = synth.rng(320)
    dtype, c, hc, wc, grid = "bf16", 32, 16, 32, (4, 8)
    coarse = synth.to_storage_bits(synth.normal(r, (1, c, hc, wc)), dtype)
    prev = synth.nan_canaries(r, (1, c, 2 * hc, 2 * wc), dtype)
    full = np.ones((1,) + grid, np.uint8)
    want = oracle.sparse_upsample_add(coarse, None, full, prev, dtype)
    out = to_dev(prev, dtype)
    B.bc_sparse_upsample_add(to_dev(coarse, dtype), B.BC_NHWC, None, out, grid, 0, None, None)
    _check_merge(from_dev(out), want, full, dtype)
    # an empty index leaves every block untouched
    idx, cnt = _index(B, np.zeros((1,) + grid, np.uint8))
    out = to_dev(prev, dtype)
    B.bc_sparse_upsample_add(to_dev(coarse, dtype), B.BC_NHWC, None, out, grid, 0, idx, cnt)
    assert np.array_equal(from_dev(out), prev)


def test_upsample_of_constant_is_constant(B):
    """Bilinear weights sum to one: a constant coarse map stays constant (exact in bf16)."""
    coarse = torch.full((1, 8, 16, 16), 1.5, dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((1, 16, 32, 16), dtype=torch.bfloat16, device="cuda")
    B.bc_sparse_upsample_add(coarse, B.BC_NHWC, None, out, (2, 2), 0, None, None)
    assert bool((out == 1.5).all())


# ------------------------------------------------------------------ information gain, NHWC 16-bit

def _ig_nhwc(B, lt_bits, lp_bits, dtype, classes, grid):
    n = lt_bits.shape[0]
    ig = torch.full((n,) + tuple(grid), -1.0, dtype=torch.float32, device="cuda")
    B.bc_seg_information_gain(to_dev(lt_bits, dtype), to_dev(lp_bits, dtype), grid, ig,
                              classes=classes, layout=B.BC_NHWC)
    return ig.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype,n,classes,c,h,w,grid", [
    ("bf16", 1, 19, 64, 64, 128, (8, 16)),      # a head padded to 64 output channels
    ("bf16", 2, 19, 24, 40, 48, (4, 6)),
    ("f16", 1, 5, 8, 32, 32, (2, 2)),
    ("bf16", 1, 32, 32, 16, 48, (2, 3)),
    ("f16", 1, 9, 16, 24, 24, (3, 3)),
    ("bf16", 1, 1, 8, 16, 16, (2, 2)),          # one class: KL is 0
    ("bf16", 1, 19, 24, 256, 256, (4, 4)),      # 4096-pixel blocks: one workgroup, 16 pixels a thread
    ("bf16", 1, 19, 24, 256, 256, (2, 2)),      # 16384-pixel blocks: several workgroups per block
])
def test_information_gain_nhwc_parity(B, dtype, n, classes, c, h, w, grid):
    r = synth.rng(330 + c + classes)
    lt = synth.to_storage_bits(synth.seg_logits(r, n, classes, h, w, cell=8), dtype)
    lp = synth.to_storage_bits(synth.seg_logits_next(r, synth.storage_to_f64(lt, dtype).astype(np.float32),
                                                     changed=0.3, cell=16), dtype)
    want = P.seg_information_gain(synth.storage_to_f64(lt, dtype), synth.storage_to_f64(lp, dtype), *grid)
    pad = lambda b: np.concatenate([b, synth.nan_canaries(r, (n, c - classes, h, w), dtype)], axis=1)
    got = _ig_nhwc(B, pad(lt), pad(lp), dtype, classes, grid)
    assert max_abs_rel(got, want) <= 1e-4


@pytest.mark.parametrize("layout,grid", [("nchw_f32", (2, 4)), ("nhwc_bf16", (4, 8))])
def test_information_gain_with_execution_grid(B, layout, grid):
    """With the execution grid, blocks that did not run get 0 without their scores being
    read (the previous map holds NaN there), executed blocks their gain: fp32 channels
    first with several workgroups per block (a zero fill first) and bf16 channels last
    (19 classes in 24 channels) with one workgroup per block."""
    r = synth.rng(345)
    n, classes, h, w = 2, 19, 256, 512
    dtype = "f32" if layout == "nchw_f32" else "bf16"
    lt = synth.to_storage_bits(synth.seg_logits(r, n, classes, h, w, cell=8), dtype)
    lp = synth.to_storage_bits(synth.seg_logits_next(r, synth.storage_to_f64(lt, dtype).astype(np.float32),
                                                     0.3), dtype)
    mask = np.concatenate([synth.frac_mask(346, *grid, 0.5), synth.frac_mask(347, *grid, 0.25)])
    want = P.seg_information_gain(synth.storage_to_f64(lt, dtype), synth.storage_to_f64(lp, dtype), *grid)
    want = np.where(mask != 0, want, 0.0)
    nan = synth.to_storage_bits(np.full((1,), np.nan, np.float32), dtype)[0]
    stale = lp.copy()
    sel = np.broadcast_to(oracle.expand_mask(mask, h // grid[0], w // grid[1]), stale.shape)
    stale[~sel] = nan
    ig = torch.full((n,) + grid, -1.0, device="cuda")
    m = torch.from_numpy(mask).cuda()
    if layout == "nchw_f32":
        a, b = (torch.from_numpy(np.ascontiguousarray(x).view(np.float32)).cuda() for x in (lt, stale))
        B.bc_seg_information_gain(a, b, grid, ig, mask=m)
    else:
        pad = lambda x: np.concatenate([x, synth.nan_canaries(r, (n, 24 - classes, h, w), dtype)], axis=1)
        B.bc_seg_information_gain(to_dev(pad(lt), dtype), to_dev(pad(stale), dtype), grid, ig,
                                  classes=classes, layout=B.BC_NHWC, mask=m)
    got = ig.cpu().numpy().astype(np.float64)
    assert (got[mask == 0] == 0.0).all()
    assert max_abs_rel(got[mask != 0], want[mask != 0]) <= 1e-4


def test_information_gain_nhwc_full_size(B):
    """19 classes in 64 channels at a quarter of 2048x1024 (512x256), 8x16 grid."""
    r = synth.rng(340)
    dtype, classes, c, h, w = "bf16", 19, 64, 256, 512
    lt = synth.to_storage_bits(synth.seg_logits(r, 1, classes, h, w), dtype)
    lp = synth.to_storage_bits(synth.seg_logits_next(r, synth.storage_to_f64(lt, dtype).astype(np.float32),
                                                     changed=0.25), dtype)
    want = P.seg_information_gain(synth.storage_to_f64(lt, dtype), synth.storage_to_f64(lp, dtype), 8, 16)
    pad = lambda b: np.concatenate([b, synth.nan_canaries(r, (1, c - classes, h, w), dtype)], axis=1)
    got = _ig_nhwc(B, pad(lt), pad(lp), dtype, classes, (8, 16))
    assert max_abs_rel(got, want) <= 1e-4


def test_information_gain_copied_blocks_are_zero(B):
    """Blocks whose scores were transferred from frame t-1 have exactly zero gain."""
    r = synth.rng(350)
    dtype, classes, c, h, w, grid = "bf16", 19, 32, 64, 128, (4, 8)
    lp = synth.to_storage_bits(synth.seg_logits(r, 1, c, h, w), dtype)
    fresh = synth.to_storage_bits(synth.seg_logits(r, 1, c, h, w), dtype)
    mask = synth.bernoulli_mask(r, 1, *grid, 0.5)
    lt = oracle.select(mask, fresh, lp, h // grid[0], w // grid[1])
    got = _ig_nhwc(B, lt, lp, dtype, classes, grid)
    assert (got[mask == 0] == 0.0).all()
    want = P.seg_information_gain(synth.storage_to_f64(lt[:, :classes], dtype),
                                  synth.storage_to_f64(lp[:, :classes], dtype), *grid)
    assert max_abs_rel(got, want) <= 1e-4


# ------------------------------------------------------------------ pyramid pooling

@pytest.mark.parametrize("dtype,n,c,h,w,grid,rows,cl,p", [
    ("bf16", 1, 128, 32, 64, (8, 16), (8, 4, 2, 1), 32, 0.3),   # the 2048x1024 workload
    ("bf16", 2, 16, 12, 20, (3, 5), (5, 3, 1), 8, 0.5),         # bins of unequal size
    ("f16", 1, 8, 8, 16, (2, 4), (8, 4, 2, 1), 16, 0.6),        # one vector per pixel
    ("bf16", 1, 512, 8, 16, (2, 4), (3, 2), 64, 0.5),           # 64 vectors per pixel
    ("bf16", 1, 2048, 4, 8, (2, 2), (1,), 8, 1.0),              # the widest input
])
def test_spp_parity(B, dtype, n, c, h, w, grid, rows, cl, p):
    r = synth.rng(350 + c + h)
    gh, gw = grid
    bins = [oracle.spp_bins(h, w, g) for g in rows]
    x = synth.to_storage_bits(synth.normal(r, (n, c, h, w)), dtype)
    wts = [synth.to_storage_bits(synth.he_normal(r, cl, c, 1, 1), dtype) for _ in rows]
    bias = [synth.normal(r, cl, 0.1).astype(np.float32) for _ in rows]
    cout = c + len(rows) * cl
    prev = synth.nan_canaries(r, (n, cout, h, w), dtype)
    mask = synth.bernoulli_mask(r, n, gh, gw, p)
    want_lv = oracle.spp_levels(x, rows, wts, bias, dtype)
    want = oracle.sparse_spp(x, want_lv, mask, prev, dtype)
    idx, cnt = _index(B, mask)
    wd = torch.from_numpy(np.stack([wl.reshape(cl, c) for wl in wts]).view(np.int16)).cuda()
    wd = wd.view(torch.bfloat16 if dtype == "bf16" else torch.float16)
    bd = torch.from_numpy(np.stack(bias)).cuda()
    tb = sum(a * b for a, b in bins)
    lv = torch.full((n, tb, cl), float("nan"), device="cuda").to(wd.dtype)
    out = to_dev(prev, dtype)
    B.bc_sparse_spp(to_dev(x, dtype), B.BC_NHWC, [a for a, _ in bins], [b for _, b in bins], cl, wd, bd,
                    lv, out, grid, idx, cnt)
    torch.cuda.synchronize()
    # levels: every bin of every image, [n][bins][cl]
    got_lv = lv.view(torch.int16).cpu().numpy().view(np.uint16)
    o = 0
    for (a, b), wl in zip(bins, want_lv):
        g = got_lv[:, o:o + a * b].reshape(n, a, b, cl).transpose(0, 3, 1, 2)
        assert max_abs_rel(oracle.value(g, dtype), oracle.value(wl, dtype)) <= TOL[dtype]
        o += a * b
    got = from_dev(out)
    sel = block_select(mask, got.shape)
    assert np.array_equal(got[~sel], prev[~sel]), "copied blocks changed"
    assert np.array_equal(got[:, :c][sel[:, :c]], x[sel[:, :c]])      # the input's own bits
    # the context channels against the oracle's resampling of the GPU's own levels (the
    # resampling alone) and of the oracle's levels (the whole layer)
    own = oracle.sparse_spp(x, [got_lv[:, sum(a * b for a, b in bins[:k]):sum(a * b for a, b in bins[:k + 1])]
                                .reshape(n, bins[k][0], bins[k][1], cl).transpose(0, 3, 1, 2).copy()
                                for k in range(len(bins))], mask, prev, dtype)
    # fp32 weights of non-dyadic resampling ratios may put a value on the other side of
    # one rounding boundary: at most one unit in the last place of the storage format
    ulp = {"bf16": 2.0 ** -7, "f16": 2.0 ** -10}[dtype]
    assert max_abs_rel(oracle.value(got[sel], dtype), oracle.value(own[sel], dtype)) <= ulp
    assert max_abs_rel(oracle.value(got[sel], dtype), oracle.value(want[sel], dtype)) <= TOL[dtype]


def test_spp_no_block_and_every_block(B):
    """An empty grid writes no output element (the levels are still recomputed); the
    full call (no index) writes every block."""
    r = synth.rng(360)
    c, h, w, cl = 64, 16, 32, 16
    x = synth.to_storage_bits(synth.normal(r, (1, c, h, w)), "bf16")
    wb = synth.to_storage_bits(synth.he_normal(r, 2 * cl, c, 1, 1), "bf16").reshape(2, cl, c)
    wd = torch.from_numpy(wb.view(np.int16)).view(torch.bfloat16).cuda()
    prev = synth.nan_canaries(r, (1, c + 2 * cl, h, w), "bf16")
    out = to_dev(prev, "bf16")
    lv = torch.empty((1, 4 * 8 + 1 * 2, cl), dtype=torch.bfloat16, device="cuda")
    idx, cnt = _index(B, np.zeros((1, 4, 8), np.uint8))
    B.bc_sparse_spp(to_dev(x, "bf16"), B.BC_NHWC, [4, 1], [8, 2], cl, wd, None, lv, out, (4, 8), idx, cnt)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(out), prev)
    B.bc_sparse_spp(to_dev(x, "bf16"), B.BC_NHWC, [4, 1], [8, 2], cl, wd, None, lv, out, (4, 8), None, None)
    torch.cuda.synchronize()
    got = from_dev(out)
    assert np.array_equal(got[:, :c], x) and not np.isnan(oracle.value(got, "bf16")).any()


def _mask_pattern(kind, n, gh, gw, r):
    """Execution grids: Bernoulli(0.4), none, one block, checkerboard, border ring, all."""
    y, x = np.mgrid[0:gh, 0:gw]
    one = {"bern": lambda: r.random((gh, gw)) < 0.4,
           "empty": lambda: np.zeros((gh, gw), bool),
           "one": lambda: (y == r.integers(gh)) & (x == r.integers(gw)),
           "checker": lambda: (y + x) % 2 == 0,
           "border": lambda: (y == 0) | (y == gh - 1) | (x == 0) | (x == gw - 1),
           "full": lambda: np.ones((gh, gw), bool)}[kind]
    return np.stack([one() for _ in range(n)]).astype(np.uint8)


def _random_upsample_cases(count, seed=2112):
    """Seeded coarse maps (1-24 x 1-24), grids dividing the 2x output, channel counts and
    formats (16-bit channels-last with C a multiple of 8, or fp32 channels-first), skip
    and ReLU on or off, each under one mask pattern."""
    r = np.random.default_rng(seed)
    kinds = ["bern", "empty", "one", "checker", "border", "full"]
    fmts = [("bf16", True), ("f16", True), ("f32", False)]
    out = []
    while len(out) < count:
        hc, wc = int(r.integers(1, 25)), int(r.integers(1, 25))
        gh = int(r.choice([d for d in range(1, 9) if (2 * hc) % d == 0]))
        gw = int(r.choice([d for d in range(1, 9) if (2 * wc) % d == 0]))
        dtype, nhwc = fmts[len(out) % len(fmts)]
        c = int(8 * r.integers(1, 9)) if nhwc else int(r.integers(1, 20))
        out.append(dict(dtype=dtype, nhwc=nhwc, n=int(r.integers(1, 3)), c=c, hc=hc, wc=wc,
                        grid=(gh, gw), skip=bool(r.random() < 0.7), relu=bool(r.random() < 0.5),
                        mask=kinds[len(out) % len(kinds)], seed=int(r.integers(1 << 30))))
    return out


UPSAMPLE_CASES = _random_upsample_cases(18)


@pytest.mark.parametrize("c", UPSAMPLE_CASES,
                         ids=[f"r{i}_{c['dtype']}{'' if c['nhwc'] else '_nchw'}_n{c['n']}_c{c['c']}_"
                              f"{c['hc']}x{c['wc']}_g{c['grid'][0]}x{c['grid'][1]}_{c['mask']}"
                              for i, c in enumerate(UPSAMPLE_CASES)])
def test_upsample_add_random_shapes(B, c):
    """Upsample-and-add on seeded random shapes and grids: copied blocks bit for bit,
    executed blocks within the storage format's bound of the fp64 oracle."""
    r = synth.rng(c["seed"])
    dtype, nhwc, n, ch, hc, wc = c["dtype"], c["nhwc"], c["n"], c["c"], c["hc"], c["wc"]
    gh, gw = c["grid"]
    coarse = synth.to_storage_bits(synth.normal(r, (n, ch, hc, wc)), dtype)
    sk = synth.to_storage_bits(synth.normal(r, (n, ch, 2 * hc, 2 * wc)), dtype) if c["skip"] else None
    prev = synth.nan_canaries(r, (n, ch, 2 * hc, 2 * wc), dtype)
    mask = _mask_pattern(c["mask"], n, gh, gw, r)
    want = oracle.sparse_upsample_add(coarse, sk, mask, prev, dtype, c["relu"])
    idx, cnt = _index(B, mask)
    out = to_dev(prev, dtype, nhwc)
    B.bc_sparse_upsample_add(to_dev(coarse, dtype, nhwc), B.BC_NHWC if nhwc else B.BC_NCHW,
                             to_dev(sk, dtype, nhwc) if c["skip"] else None, out, (gh, gw),
                             int(c["relu"]), idx, cnt)
    _check_merge(from_dev(out, nhwc), want, mask, dtype)
