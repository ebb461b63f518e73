"""GPU: bc_sparse_conv2d_noalloc, the convolution entry point that allocates nothing
(split-K partials in the library's fixed scratch array), against bc_sparse_conv2d on
the same inputs: bit for bit on two calls in a row, the second with a smaller input,
both held to the oracle on sampled active outputs, copied blocks untouched; captured in
a HIP graph and replayed with new inputs; a layer whose partials exceed the array is
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import block_select, from_dev, max_abs_rel, to_dev, weights_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B(gpu):
    from paper_2108_09376_amd import bc
    return bc


# cin, cout, h, w (input), gh, gw, k, s, active fraction: layers whose plans split K
BIG = (512, 512, 32, 64, 8, 16, 3, 1, 0.3)     # 256 full-frame tiles, 2 K slices: 8 MiB
SMALL = (512, 512, 16, 32, 4, 8, 3, 1, 0.3)    # 64 tiles, 4 K slices: 4 MiB
ONE = (2048, 512, 32, 64, 8, 16, 1, 1, 0.3)    # 1x1, 256 tiles, 3 K slices: 12 MiB


def _draw(case, seed):
    cin, cout, h, w, gh, gw, k, s, frac = case
    p = k // 2
    ho, wo = oracle.out_size(h, k, s, p), oracle.out_size(w, k, s, p)
    r = synth.rng(seed)
    return dict(case=case, p=p,
                x=synth.to_storage_bits(synth.normal(r, (1, cin, h, w)), "bf16"),
                wt=synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k), "bf16"),
                bias=synth.normal(r, cout, 0.1),
                res=synth.to_storage_bits(synth.normal(r, (1, cout, ho, wo)), "bf16"),
                prev=synth.nan_canaries(r, (1, cout, ho, wo), "bf16"),
                mask=synth.frac_mask(seed + 1, gh, gw, frac))


def _dev(B, d):
    cin, cout, h, w, gh, gw, k, s, _ = d["case"]
    m = torch.from_numpy(d["mask"]).cuda()
    idx = torch.empty(gh * gw, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    B.bc_build_block_index(m, 1, (gh, gw), idx, cnt)
    return dict(conv=(k, k, s, d["p"], 1), x=to_dev(d["x"], "bf16"), w=weights_dev(d["wt"], "bf16"),
                bias=torch.from_numpy(d["bias"]).cuda(), res=to_dev(d["res"], "bf16"),
                grid=(gh, gw), idx=idx, cnt=cnt)


def _run(B, fn, t, out):
    fn(t["conv"], t["x"], B.BC_NHWC, t["w"], t["bias"], t["res"], out, t["grid"], t["idx"], t["cnt"])


def _oracle_check(d, got):
    sel = block_select(d["mask"], got.shape)
    assert np.array_equal(got[~sel], d["prev"][~sel])            # copied blocks: previous bits
    act = np.argwhere(sel)
    pick = act[synth.rng(5).choice(len(act), size=min(1500, len(act)), replace=False)]
    z = oracle.conv2d_points(oracle.value(d["x"], "bf16"), oracle.value(d["wt"], "bf16"), pick,
                             d["bias"].astype(np.float64), oracle.value(d["res"], "bf16"),
                             d["case"][7], d["p"], True)
    want = oracle.value(oracle.store(z, "bf16"), "bf16")
    g = oracle.value(got[pick[:, 0], pick[:, 1], pick[:, 2], pick[:, 3]], "bf16")
    assert max_abs_rel(g, want) <= 2e-2


def test_noalloc_two_calls_match_conv2d(B):
    """Two no-alloc calls in a row (the second smaller, so it reuses the array the first
    filled), then the same two through bc_sparse_conv2d: identical bits."""
    draws = [_draw(BIG, 900), _draw(SMALL, 910), _draw(ONE, 920)]
    devs = [_dev(B, d) for d in draws]
    outs_na = [to_dev(d["prev"], "bf16") for d in draws]
    for t, o in zip(devs, outs_na):
        print("noalloc", t["conv"], tuple(o.shape), flush=True)
        _run(B, B.bc_sparse_conv2d_noalloc, t, o)
    outs_ref = [to_dev(d["prev"], "bf16") for d in draws]
    for t, o in zip(devs, outs_ref):
        _run(B, B.bc_sparse_conv2d, t, o)
    torch.cuda.synchronize()
    for d, a, b in zip(draws, outs_na, outs_ref):
        ga, gb = from_dev(a), from_dev(b)
        assert np.array_equal(ga, gb), d["case"]
        _oracle_check(d, ga)


def test_noalloc_graph_replays(B):
    """A no-alloc call captured once and replayed with new inputs and grids (eager work
    and synchronisation between replays): every replay equals the eager result."""
    d0 = _draw(SMALL, 930)
    t = _dev(B, d0)
    out = to_dev(d0["prev"], "bf16")
    _run(B, B.bc_sparse_conv2d_noalloc, t, out)          # eager first call of this shape
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _run(B, B.bc_sparse_conv2d_noalloc, t, out)
    for r in range(3):
        d = _draw(SMALL, 940 + 10 * r)
        t2 = _dev(B, d)
        for key in ("x", "w", "bias", "res", "idx", "cnt"):
            t[key].copy_(t2[key])
        out.copy_(to_dev(d["prev"], "bf16"))
        ref = to_dev(d["prev"], "bf16")
        _run(B, B.bc_sparse_conv2d, t2, ref)              # eager reference, other buffers
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), r
        _oracle_check(d, from_dev(out))


def test_noalloc_refuses_partials_beyond_scratch(B):
    d = _draw((512, 1024, 64, 128, 8, 16, 3, 1, 0.3), 960)
    t = _dev(B, d)
    out = to_dev(d["prev"], "bf16")
    torch.cuda.synchronize()
    with pytest.raises(B.BCError) as e:
        _run(B, B.bc_sparse_conv2d_noalloc, t, out)
    assert e.value.status == B.BC_ERR_CAPACITY
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(out), d["prev"])        # nothing was enqueued
