"""GPU: a sparse frame captured once in a HIP graph and replayed with a new execution
grid each time (copied into the mask the captured index build reads, with eager work
and synchronisation between replays) leaves every layer buffer bit-identical to the same
frames run eagerly on a twin network with the same weights."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R(gpu):
    from paper_2108_09376_amd import resnet
    return resnet


@pytest.mark.parametrize("kind", ["resnet50", "swiftnet18"])
def test_graph_replays_match_eager_frames(R, kind):
    h, w = 512, 1024

    def make():
        if kind == "resnet50":
            return R.SparseResNet(50, h, w, 128, device="cuda")
        return R.SparseSwiftNet(18, h, w, 128, device="cuda")

    net, twin = make(), make()
    assert net.pairs                     # the frame has paired launches
    x = torch.from_numpy(synth.to_storage_bits(synth.normal(synth.rng(400), (1, h, w, 3)), "bf16")
                         .view(np.int16)).view(torch.bfloat16).cuda()
    for n in (net, twin):
        n.frame(x, sparse=False)
    net.set_mask(synth.frac_mask(401, 4, 8, 0.5))
    net.frame(x, sparse=True)            # eager warm-up: plans and workspaces exist
    twin.set_mask(synth.frac_mask(401, 4, 8, 0.5))
    twin.frame(x, sparse=True)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        net.frame(x, sparse=True)
    for r, frac in enumerate((0.3, 0.6, 0.15)):
        mask = synth.frac_mask(410 + r, 4, 8, frac)
        x2 = synth.to_storage_bits(synth.normal(synth.rng(420 + r), (1, h, w, 3)), "bf16")
        x.copy_(torch.from_numpy(x2.view(np.int16)).view(torch.bfloat16))
        net.set_mask(mask)
        twin.set_mask(mask)
        torch.cuda.synchronize()
        g.replay()
        twin.frame(x, sparse=True)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(net.buffers, twin.buffers)):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (kind, r, net.layers[i].name)


_CAPTURE_SCRIPT = r'''
import sys
import numpy as np
import torch
sys.path.insert(0, sys.argv[1])
import synth
from paper_2108_09376_amd import bc

def t(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()

r = synth.rng(970)
# 3x3 512 -> 512 on a 32x64 map, 8x16 grid: its plan splits K (256 full-frame tiles)
x = t(synth.to_storage_bits(synth.normal(r, (1, 32, 64, 512)), "bf16"))
w = t(synth.to_storage_bits(synth.he_normal(r, 512, 512, 3, 3).transpose(0, 2, 3, 1).copy(), "bf16"))
b = torch.from_numpy(synth.normal(r, 512, 0.1)).cuda()
out = torch.zeros((1, 32, 64, 512), dtype=torch.bfloat16, device="cuda")
idx = torch.arange(128, dtype=torch.int32, device="cuda")
cnt = torch.full((1,), 128, dtype=torch.int32, device="cuda")
args = ((3, 3, 1, 1, 1), x, bc.BC_NHWC, w, b, None)
torch.cuda.synchronize()
status = None
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):
    try:
        bc.bc_sparse_conv2d(*args, out, (8, 16), idx, cnt)
    except bc.BCError as e:
        status = e.status
print("captured-first-call", status, flush=True)
ref = torch.zeros_like(out)
bc.bc_sparse_conv2d(*args, ref, (8, 16), idx, cnt)     # eager: allocates the workspace
torch.cuda.synchronize()
g2 = torch.cuda.CUDAGraph()
with torch.cuda.graph(g2):
    bc.bc_sparse_conv2d(*args, out, (8, 16), idx, cnt)
g2.replay()
torch.cuda.synchronize()
print("replay-equal", bool(torch.equal(out.view(torch.int16), ref.view(torch.int16))), flush=True)
'''


def test_split_workspace_not_allocated_under_capture(R):
    """In a fresh process, the first call that needs the split-K workspace is refused
    with BC_ERR_CAPTURE while its stream captures (nothing allocated, nothing enqueued,
    the capture stays valid); after one eager call the same call captures and replays."""
    import os
    import subprocess
    import sys
    from paper_2108_09376_amd import bc
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", _CAPTURE_SCRIPT, root], capture_output=True,
                       text=True, timeout=110)
    print(r.stdout[-2000:], r.stderr[-2000:])
    assert r.returncode == 0
    assert f"captured-first-call {bc.BC_ERR_CAPTURE}" in r.stdout
    assert "replay-equal True" in r.stdout


def test_captured_split_call_survives_larger_eager_calls(R):
    """A captured split-K call keeps a valid workspace after eager split calls of other,
    larger layers (the workspace is never freed or moved): its replays equal eager runs."""
    from paper_2108_09376_amd import bc

    def dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()

    def layer(seed, cin, cout, h, w, k):
        r = synth.rng(seed)
        x = dev(synth.to_storage_bits(synth.normal(r, (1, h, w, cin)), "bf16"))
        wt = dev(synth.to_storage_bits(synth.he_normal(r, cout, cin, k, k).transpose(0, 2, 3, 1).copy(), "bf16"))
        b = torch.from_numpy(synth.normal(r, cout, 0.1)).cuda()
        return ((k, k, 1, k // 2, 1), x, bc.BC_NHWC, wt, b, None)

    idx = torch.arange(128, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), 128, dtype=torch.int32, device="cuda")
    idx_s = torch.arange(32, dtype=torch.int32, device="cuda")
    cnt_s = torch.full((1,), 32, dtype=torch.int32, device="cuda")
    small = layer(980, 512, 512, 16, 32, 3)          # 4x8 grid below: 64 tiles, 4 slices
    big = layer(981, 1024, 1024, 64, 128, 3)         # 2048 tiles, 2 slices: 64 MiB of partials
    out = torch.zeros((1, 16, 32, 512), dtype=torch.bfloat16, device="cuda")
    bc.bc_sparse_conv2d(*small, out, (4, 8), idx_s, cnt_s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bc.bc_sparse_conv2d(*small, out, (4, 8), idx_s, cnt_s)
    ref = torch.zeros_like(out)
    bc.bc_sparse_conv2d(*small, ref, (4, 8), idx_s, cnt_s)
    big_out = torch.zeros((1, 64, 128, 1024), dtype=torch.bfloat16, device="cuda")
    for rep in range(2):
        bc.bc_sparse_conv2d(*big, big_out, (8, 16), idx, cnt)    # eager, largest partials
        torch.cuda.synchronize()
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), rep
