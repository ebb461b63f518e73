"""GPU parity of the steps around the block-sparse network (Sections 3.3 to 3.5)
through the C ABI against oracle/policy.py on the same seeded inputs: sampled
execution grids and their index bit for bit, frame-state copies bit for bit,
information gain and rewards within max abs-rel 1e-4 (fp32 arithmetic against the
fp64 oracle; the metric of the conv parity tests)."""
import numpy as np
import pytest
import torch

import synth
from oracle import policy as P
from tests._util import from_dev, max_abs_rel, to_dev

pytestmark = pytest.mark.gpu
TOL_F32 = 1e-4


@pytest.fixture(scope="module")
def B(gpu):
    from paper_2108_09376_amd import bc
    return bc


def _sample(B, prob, seed, frame, sentinel=-7):
    n, gh, gw = prob.shape
    p = torch.from_numpy(np.ascontiguousarray(prob, np.float32)).cuda()
    mask = torch.full((n, gh, gw), 9, dtype=torch.uint8, device="cuda")
    idx = torch.full((n * gh * gw + 3,), sentinel, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    hc = B.bc_sample_execution_grid(p, (gh, gw), seed, frame, mask, idx, cnt, h_count=True)
    return mask.cpu().numpy(), idx.cpu().numpy(), int(cnt.item()), hc


# ------------------------------------------------------------------ sampling + index

@pytest.mark.parametrize("n,gh,gw,seed,frame", [(1, 8, 16, 2021, 1), (1, 8, 16, 7, 0), (3, 13, 17, 1, 5),
                                                (2, 64, 64, 123456789012, (1 << 32) + 3),
                                                (1, 1, 1, 0, 0), (4, 256, 256, 99, 17)])
def test_sampling_bit_exact(B, n, gh, gw, seed, frame):
    prob = synth.block_probabilities(synth.rng(70 + gh), n, gh, gw)
    want_mask, want_idx = P.sample_execution_grid(prob, seed, frame)
    mask, idx, cnt, hc = _sample(B, prob, seed, frame)
    assert np.array_equal(mask, want_mask)
    assert cnt == hc == want_idx.size
    assert np.array_equal(idx[:cnt], want_idx) and (idx[cnt:] == -7).all()


def test_sampling_threshold_is_exact(B):
    """p_b = u_b must not execute and p_b = u_b + 2^-24 must: pins the 24-bit uniform
    and the strict comparison. u_b comes from the oracle's generator."""
    n, gh, gw, seed, frame = 2, 32, 32, 555, 12
    u = P.block_uniforms(n, gh, gw, seed, frame)
    mask, _, cnt, _ = _sample(B, u.astype(np.float32), seed, frame)
    assert cnt == 0 and not mask.any()
    mask, _, cnt, _ = _sample(B, (u + 2.0 ** -24).astype(np.float32), seed, frame)
    assert cnt == n * gh * gw and mask.all()


def test_sampling_edges(B):
    z = np.zeros((1, 8, 16), np.float32)
    assert _sample(B, z, 1, 1)[2] == 0
    assert _sample(B, np.ones_like(z), 1, 1)[2] == 128
    nan = np.full_like(z, np.nan)
    mask, _, cnt, _ = _sample(B, nan, 1, 1)
    assert cnt == 0 and not mask.any()                  # a NaN probability never executes


# ------------------------------------------------------------------ frame state

@pytest.mark.parametrize("dtype,nhwc,shape,grid,p", [
    ("bf16", True, (1, 3, 1024, 2048), (8, 16), 0.3),     # the RGB frame of the workload
    ("bf16", True, (2, 3, 64, 96), (4, 6), 0.5),
    ("f32", False, (2, 3, 40, 60), (4, 6), 0.5),          # 10-pixel rows: element path
    ("f32", True, (1, 3, 64, 128), (4, 8), 0.6),
    ("bf16", False, (1, 4, 64, 128), (2, 2), 1.0),
    ("f16", True, (1, 5, 30, 40), (3, 4), 0.4),           # odd channel count: element path
])
def test_frame_state_bit_exact(B, dtype, nhwc, shape, grid, p):
    r = synth.rng(80 + shape[2])
    frame = synth.to_storage_bits(synth.normal(r, shape), dtype)
    state = synth.nan_canaries(r, shape, dtype)
    mask = synth.bernoulli_mask(r, shape[0], grid[0], grid[1], p)
    want = P.update_frame_state(frame, state, mask, "nchw")
    m = torch.from_numpy(mask).cuda()
    idx = torch.empty(mask.size, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    B.bc_build_block_index(m, shape[0], grid, idx, cnt)
    f, s = to_dev(frame, dtype, nhwc), to_dev(state, dtype, nhwc)
    B.bc_update_frame_state(f, s, B.BC_NHWC if nhwc else B.BC_NCHW, grid, idx, cnt)
    assert np.array_equal(from_dev(s, nhwc), want)


def test_frame_state_every_block(B):
    r = synth.rng(90)
    frame = synth.to_storage_bits(synth.normal(r, (1, 3, 128, 256)), "bf16")
    state = synth.nan_canaries(r, (1, 3, 128, 256), "bf16")
    f, s = to_dev(frame, "bf16"), to_dev(state, "bf16")
    B.bc_update_frame_state(f, s, B.BC_NHWC, (8, 16), None, None)
    assert np.array_equal(from_dev(s), frame)


# ------------------------------------------------------------------ information gain

def _ig(B, lt, lp, grid):
    n = lt.shape[0]
    a = torch.from_numpy(lt).cuda()
    b = torch.from_numpy(lp).cuda()
    ig = torch.full((n,) + tuple(grid), -1.0, dtype=torch.float32, device="cuda")
    B.bc_seg_information_gain(a, b, grid, ig)
    return ig.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("n,c,h,w,grid", [(2, 19, 64, 96, (4, 6)), (1, 5, 48, 64, (3, 4)),
                                          (1, 27, 40, 256, (2, 2)), (1, 1, 16, 16, (2, 2)),
                                          (3, 8, 32, 32, (1, 1)), (1, 32, 24, 40, (3, 5))])
def test_information_gain_parity(B, n, c, h, w, grid):
    r = synth.rng(100 + c)
    lt = synth.seg_logits(r, n, c, h, w, cell=8)
    lp = synth.seg_logits_next(r, lt, changed=0.3, cell=16)
    want = P.seg_information_gain(lt, lp, *grid)
    got = _ig(B, lt, lp, grid)
    assert max_abs_rel(got, want) <= TOL_F32


def test_information_gain_no_change_is_zero(B):
    lt = synth.seg_logits(synth.rng(110), 1, 19, 64, 128)
    assert np.abs(_ig(B, lt, lt, (4, 8))).max() <= 1e-5


def test_information_gain_full_size(B):
    """19 classes at 2048x1024, the 8x16 grid of 128-px blocks."""
    r = synth.rng(111)
    lt = synth.seg_logits(r, 1, 19, 1024, 2048)
    lp = synth.seg_logits_next(r, lt, changed=0.25)
    want = P.seg_information_gain(lt, lp, 8, 16)
    got = _ig(B, lt, lp, (8, 16))
    assert max_abs_rel(got, want) <= TOL_F32


# ------------------------------------------------------------------ rewards and loss

@pytest.mark.parametrize("n,gh,gw", [(1, 8, 16), (3, 5, 7), (2, 64, 64)])
def test_rewards_parity_two_frames(B, n, gh, gw):
    r = synth.rng(120 + gh)
    tau, gamma, mu = 0.3, 5.0, 0.9
    m0 = r.uniform(0, 1, n).astype(np.float32)
    mavg = torch.from_numpy(m0.copy()).cuda()
    m_prev = m0.astype(np.float64)
    for t in range(2):                           # M_t feeds the next frame in place
        ig = r.uniform(0, 2, (n, gh, gw)).astype(np.float32)
        prob = synth.block_probabilities(r, n, gh, gw)
        prob = np.clip(prob, 1e-3, 1 - 1e-3).astype(np.float32)
        mask = (r.random((n, gh, gw)) < prob).astype(np.uint8)
        want_r, want_c, want_m = P.block_rewards(ig, mask, tau, gamma, mu, m_prev)
        want_l = P.reinforce_loss(want_r, mask, prob)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        reward = torch.empty((n, gh, gw), dtype=torch.float32, device="cuda")
        cost = torch.empty(n, dtype=torch.float32, device="cuda")
        loss = torch.empty(n, dtype=torch.float32, device="cuda")
        B.bc_block_rewards(dev(ig), dev(mask), dev(prob), (gh, gw), tau, gamma, mu, mavg, reward, cost, loss)
        assert max_abs_rel(reward.cpu().numpy(), want_r) <= TOL_F32
        assert max_abs_rel(cost.cpu().numpy(), want_c) <= 1e-6
        assert max_abs_rel(mavg.cpu().numpy(), want_m) <= 1e-6
        assert max_abs_rel(loss.cpu().numpy(), want_l) <= TOL_F32
        m_prev = want_m


def test_rewards_without_loss(B):
    ig = torch.rand((1, 8, 16), device="cuda")
    mask = (torch.rand((1, 8, 16), device="cuda") < 0.3).to(torch.uint8)
    mavg = torch.full((1,), 0.5, device="cuda")
    reward = torch.empty((1, 8, 16), device="cuda")
    B.bc_block_rewards(ig, mask, None, (8, 16), 0.3, 5.0, 0.9, mavg, reward)
    want, _, m = P.block_rewards(ig.cpu().numpy(), mask.cpu().numpy(), 0.3, 5.0, 0.9, [0.5])
    assert max_abs_rel(reward.cpu().numpy(), want) <= TOL_F32
    assert abs(float(mavg.item()) - m[0]) <= 1e-6


def _random_state_cases(count, seed=2113):
    """Seeded frame-state shapes: batch 1-2, 1-8 channels, block edges 1-12 px on grids up
    to 6 x 7, every storage format in either layout, each under one mask pattern."""
    r = np.random.default_rng(seed)
    kinds = ["bern", "empty", "one", "checker", "border", "full"]
    fmts = [("bf16", True), ("f16", True), ("f32", False), ("f32", True), ("bf16", False), ("f16", False)]
    out = []
    for i in range(count):
        gh, gw = int(r.integers(1, 7)), int(r.integers(1, 8))
        bh, bw = int(r.integers(1, 13)), int(r.integers(1, 13))
        dtype, nhwc = fmts[i % len(fmts)]
        out.append(dict(dtype=dtype, nhwc=nhwc, shape=(int(r.integers(1, 3)), int(r.integers(1, 9)),
                                                      gh * bh, gw * bw),
                        grid=(gh, gw), mask=kinds[i % len(kinds)], seed=int(r.integers(1 << 30))))
    return out


STATE_CASES = _random_state_cases(18)


@pytest.mark.parametrize("c", STATE_CASES,
                         ids=[f"r{i}_{c['dtype']}{'' if c['nhwc'] else '_nchw'}_{'x'.join(map(str, c['shape']))}_"
                              f"g{c['grid'][0]}x{c['grid'][1]}_{c['mask']}" for i, c in enumerate(STATE_CASES)])
def test_frame_state_random_shapes(B, c):
    """Frame state on seeded random shapes, grids and formats: executed blocks take the
    frame's bits, every other element keeps its NaN canary."""
    r = synth.rng(c["seed"])
    dtype, nhwc, shape = c["dtype"], c["nhwc"], c["shape"]
    gh, gw = c["grid"]
    frame = synth.to_storage_bits(synth.normal(r, shape), dtype)
    state = synth.nan_canaries(r, shape, dtype)
    y, x = np.mgrid[0:gh, 0:gw]
    pick = {"bern": lambda: r.random((gh, gw)) < 0.4, "empty": lambda: np.zeros((gh, gw), bool),
            "one": lambda: (y == r.integers(gh)) & (x == r.integers(gw)),
            "checker": lambda: (y + x) % 2 == 0,
            "border": lambda: (y == 0) | (y == gh - 1) | (x == 0) | (x == gw - 1),
            "full": lambda: np.ones((gh, gw), bool)}[c["mask"]]
    mask = np.stack([pick() for _ in range(shape[0])]).astype(np.uint8)
    want = P.update_frame_state(frame, state, mask, "nchw")
    idx = torch.empty(mask.size, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    B.bc_build_block_index(torch.from_numpy(mask).cuda(), shape[0], (gh, gw), idx, cnt)
    f, s = to_dev(frame, dtype, nhwc), to_dev(state, dtype, nhwc)
    B.bc_update_frame_state(f, s, B.BC_NHWC if nhwc else B.BC_NCHW, (gh, gw), idx, cnt)
    assert np.array_equal(from_dev(s, nhwc), want)
