"""GPU parity of the policy network's forward pass (Section 3.3, Eq. 2; architecture
reading in oracle/policy.py) through the C ABI against the oracle on the same seeded
inputs: S_t assembly and the block probabilities within max abs-rel 2e-2 (bf16, fp16
storage) / 1e-4 (the fp32 sigmoid of stored logits), and the whole network end to end
with the norm-wise gate of the other network tests."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import network as onet
from oracle import policy as P
from tests._util import TOL, from_dev, max_abs_rel, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R(gpu):
    from paper_2108_09376_amd import bc, resnet
    return bc, resnet


def _inputs(seed, dtype, n, h, w, c, gh, gw):
    r = synth.rng(seed)
    fr = synth.to_storage_bits(synth.normal(r, (n, 3, h, w)), dtype)
    st = synth.to_storage_bits(synth.normal(r, (n, 3, h, w)), dtype)
    sc = synth.to_storage_bits(synth.normal(r, (n, c, h // 4, w // 4), 3.0), dtype)
    m = synth.bernoulli_mask(r, n, gh, gw, 0.4)
    return fr, st, sc, m


@pytest.mark.parametrize("dtype,n,h,w,c,classes,grid,mask", [
    ("bf16", 1, 1024, 2048, 64, 19, (8, 16), True),     # the workload: 19 classes in 64 channels
    ("bf16", 2, 64, 128, 24, 24, (2, 4), True),
    ("f16", 1, 32, 96, 8, 5, (2, 3), False),            # no previous grid
    ("bf16", 1, 16, 16, 16, 1, (1, 1), True),           # one class: probability 1
])
def test_policy_input_parity(R, dtype, n, h, w, c, classes, grid, mask):
    bc, _ = R
    fr, st, sc, m = _inputs(400 + h, dtype, n, h, w, c, *grid)
    want = P.policy_input(fr, st, sc, classes, m if mask else None, dtype)
    out = torch.full((n, h // 4, w // 4, 32), float("nan"), device="cuda").to(
        torch.bfloat16 if dtype == "bf16" else torch.float16)
    bc.bc_policy_input(to_dev(fr, dtype), to_dev(st, dtype), to_dev(sc, dtype), classes,
                       torch.from_numpy(m).cuda() if mask else None, grid, out)
    got = from_dev(out)
    assert max_abs_rel(oracle.value(got, dtype), oracle.value(want, dtype)) <= TOL[dtype]


def test_policy_probabilities_parity(R):
    bc, _ = R
    r = synth.rng(410)
    lg = synth.to_storage_bits(synth.normal(r, (2, 64, 8, 16), 6.0), "bf16")
    prob = torch.full((2, 8, 16), -1.0, device="cuda")
    bc.bc_policy_probabilities(to_dev(lg, "bf16"), prob)
    assert max_abs_rel(prob.cpu().numpy(), P.policy_probabilities(lg)) <= 1e-4


def test_policy_network_matches_oracle(R):
    """The whole forward pass on a 256x512 frame (S_t 64x128, head 2x4 = the frame's
    128-pixel grid); no GPU value is fed to the oracle."""
    bc, resnet = R
    h, w, classes = 256, 512, 19
    fr, st, sc, m = _inputs(420, "bf16", 1, h, w, 64, 2, 4)
    table = onet.policy_table()
    params = onet.make_params(table, seed0=3000)
    folded = onet.fold_params(table, params, "bf16")
    s_t = P.policy_input(fr, st, sc, classes, m)
    ref = onet.dense_frame(table, folded, s_t, "bf16")
    want_p = P.policy_probabilities(ref[-1])
    net = resnet.PolicyNet(h, w, classes=classes, params=params)
    prob = net.forward(to_dev(fr, "bf16"), to_dev(st, "bf16"), to_dev(sc, "bf16"),
                       torch.from_numpy(m).cuda())
    torch.cuda.synchronize()
    assert max_abs_rel(oracle.value(from_dev(net.input), "bf16"), oracle.value(s_t, "bf16")) <= 2e-2
    for li, (g, r) in enumerate(zip(net.buffers, ref)):
        gv, rv = oracle.value(from_dev(g), "bf16"), oracle.value(r, "bf16")
        assert np.linalg.norm(gv - rv) <= 2e-2 * np.linalg.norm(rv), li
    p = prob.cpu().numpy()
    assert p.shape == (1, 2, 4) and ((p > 0) & (p < 1)).all()
    assert np.abs(p - want_p).max() <= 2e-2
