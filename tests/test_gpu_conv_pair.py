"""GPU: two independent convolutions through bc_sparse_conv2d_pair (one launch when both
are BF16 1x1 layers whose plans pair) against the oracle on active blocks, and bit for
bit against the two single calls; blocks outside the grid keep their previous bits in
both outputs."""
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


# cin, h, w, gh, gw, first (cout, k, s, relu, residual), second (same), active fraction
PAIRS = [
    # 64 -> 256 shortcut (128-wide tiles) with 64 -> 64 (64-wide, two chunks per barrier)
    (64, 64, 128, 2, 4, (256, 1, 1, False, False), (64, 1, 1, True, False), 0.5),
    # stride-2 256 -> 512 shortcut with 256 -> 128 (128-wide tiles both)
    (256, 64, 128, 2, 4, (512, 1, 2, False, False), (128, 1, 1, True, False), 0.5),
    # stride-2 512 -> 1024 with 512 -> 256 (64-wide both), 4x4 and 8x8 output blocks, ragged
    # tail of patches, residual and ReLU on the first
    (512, 48, 48, 6, 6, (1024, 1, 2, True, True), (256, 1, 1, True, False), 0.4),
    # the second splits K (32 chunks on few tiles): two launches
    (1024, 16, 32, 2, 4, (256, 1, 2, False, False), (64, 1, 1, True, True), 0.5),
    # the second is a 3x3 layer: two launches
    (64, 64, 128, 2, 4, (256, 1, 1, False, False), (64, 3, 1, True, False), 0.5),
]
IDS = ["64-256s1_64-64", "256-512s2_256-128", "512-1024s2_512-256_ragged", "second_splits_K",
       "second_3x3"]


def _draw(case, dtype, seed):
    cin, h, w, gh, gw, la, lb, frac = case
    r = synth.rng(seed)
    x = synth.to_storage_bits(synth.normal(r, (1, cin, h, w)), dtype)
    calls = []
    for cout, k, s, relu, has_res in (la, lb):
        p = k // 2
        ho, wo = oracle.out_size(h, k, s, p), oracle.out_size(w, k, s, p)
        wt = synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), dtype)
        bias = synth.normal(r, cout, 0.1)
        res = synth.to_storage_bits(synth.normal(r, (1, cout, ho, wo)), dtype) if has_res else None
        prev = synth.nan_canaries(r, (1, cout, ho, wo), dtype)
        calls.append(dict(cout=cout, k=k, s=s, p=p, relu=relu, wt=wt, bias=bias, res=res, prev=prev))
    mask = synth.frac_mask(seed + 1, gh, gw, frac)
    return x, calls, mask


def _dev_call(B, c, xd, dtype):
    out = to_dev(c["prev"], dtype)
    return ((c["k"], c["k"], c["s"], c["p"], int(c["relu"])), xd, B.BC_NHWC, weights_dev(c["wt"], dtype),
            torch.from_numpy(c["bias"]).cuda(), None if c["res"] is None else to_dev(c["res"], dtype), out)


def _index(B, mask):
    idx = torch.zeros(mask.size, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.bc_build_block_index(torch.from_numpy(mask).cuda(), 1, mask.shape[1:], idx, cnt)
    return idx, cnt


@pytest.mark.parametrize("case", PAIRS, ids=IDS)
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_pair_matches_oracle_and_single_calls(B, case, dtype):
    x, calls, mask = _draw(case, dtype, seed=300)
    gh, gw = mask.shape[1:]
    xd = to_dev(x, dtype)
    idx, cnt = _index(B, mask)
    pa, pb = _dev_call(B, calls[0], xd, dtype), _dev_call(B, calls[1], xd, dtype)
    B.bc_sparse_conv2d_pair(pa, pb, (gh, gw), idx, cnt)
    sa, sb = _dev_call(B, calls[0], xd, dtype), _dev_call(B, calls[1], xd, dtype)
    B.bc_sparse_conv2d(*sa[:6], sa[6], (gh, gw), idx, cnt)
    B.bc_sparse_conv2d(*sb[:6], sb[6], (gh, gw), idx, cnt)
    for c, pc, sc in zip(calls, (pa, pb), (sa, sb)):
        got = from_dev(pc[6])
        assert np.array_equal(got, from_dev(sc[6]))          # same bits as a call of its own
        want = oracle.sparse_conv2d(x, c["wt"], mask, c["prev"], dtype, c["s"], c["p"], c["bias"],
                                    c["res"], c["relu"])
        sel = block_select(mask, got.shape)
        assert np.array_equal(got[~sel], c["prev"][~sel])    # copied blocks: bit for bit
        err = max_abs_rel(oracle.value(got[sel], dtype), oracle.value(want[sel], dtype))
        assert err <= TOL[dtype], err


@pytest.mark.parametrize("case", PAIRS[:3], ids=IDS[:3])
def test_pair_full_frame_and_integer_exact(B, case):
    """Without an index (a full frame) on small-integer operands: every partial sum and
    result is exact, so both outputs match the oracle bit for bit."""
    cin, h, w, gh, gw, la, lb, _ = case
    r = synth.rng(310)
    xb = synth.to_storage_bits(synth.small_ints(r, (1, cin, h, w), -2, 2), "bf16")
    calls, devs = [], []
    xd = to_dev(xb, "bf16")
    for cout, k, s, relu, has_res in (la, lb):
        p = k // 2
        ho, wo = oracle.out_size(h, k, s, p), oracle.out_size(w, k, s, p)
        wt = synth.small_ints(r, (cout, cin, k, k), -1, 1)
        bias = synth.small_ints(r, cout, -3, 3)
        res = synth.small_ints(r, (1, cout, ho, wo), -4, 4) if has_res else None
        wb = synth.to_storage_bits(wt, "bf16")
        rb = None if res is None else synth.to_storage_bits(res, "bf16")
        prev = synth.nan_canaries(r, (1, cout, ho, wo), "bf16")
        c = dict(cout=cout, k=k, s=s, p=p, relu=relu, wt=wb, bias=bias, res=rb, prev=prev)
        calls.append(c)
        devs.append(_dev_call(B, c, xd, "bf16"))
    B.bc_sparse_conv2d_pair(devs[0], devs[1], (gh, gw), None, None)
    full = np.ones((1, gh, gw), np.uint8)
    for c, d in zip(calls, devs):
        want = oracle.sparse_conv2d(xb, c["wt"], full, c["prev"], "bf16", c["s"], c["p"], c["bias"],
                                    c["res"], c["relu"])
        assert np.array_equal(from_dev(d[6]), want)


def test_pair_twice_second_smaller_grid(B):
    """Two frames in a row on the same buffers, the second with fewer active blocks: the
    second frame's inactive blocks keep the first frame's bits."""
    case = PAIRS[1]
    x, calls, mask = _draw(case, "bf16", seed=320)
    gh, gw = mask.shape[1:]
    xd = to_dev(x, "bf16")
    pa, pb = _dev_call(B, calls[0], xd, "bf16"), _dev_call(B, calls[1], xd, "bf16")
    idx, cnt = _index(B, np.ones_like(mask))
    B.bc_sparse_conv2d_pair(pa, pb, (gh, gw), idx, cnt)
    first = [from_dev(pa[6]), from_dev(pb[6])]
    x2 = synth.to_storage_bits(synth.normal(synth.rng(321), x.shape), "bf16")
    xd.copy_(to_dev(x2, "bf16"))
    idx, cnt = _index(B, mask)
    B.bc_sparse_conv2d_pair(pa, pb, (gh, gw), idx, cnt)
    for c, d, f in zip(calls, (pa, pb), first):
        got = from_dev(d[6])
        want = oracle.sparse_conv2d(x2, c["wt"], mask, f, "bf16", c["s"], c["p"], c["bias"], c["res"],
                                    c["relu"])
        sel = block_select(mask, got.shape)
        assert np.array_equal(got[~sel], f[~sel])
        assert max_abs_rel(oracle.value(got[sel], "bf16"), oracle.value(want[sel], "bf16")) <= TOL["bf16"]
