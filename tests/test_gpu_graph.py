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
