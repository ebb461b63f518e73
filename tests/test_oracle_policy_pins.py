"""Pins of the policy-side oracle (oracle/policy.py) against things other than itself:
published known-answer vectors, closed forms, a library routine, invariants and
hand-worked examples of the paper's equations (Sections 3.3 to 3.5)."""
import math
import os

import numpy as np
import pytest
import scipy.stats

import synth
from oracle import policy as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ Philox (sampling)

def _kat():
    rows = []
    for line in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")):
        if line.startswith("#") or not line.strip():
            continue
        v = [int(t, 16) for t in line.split()]
        rows.append((v[:4], v[4:6], v[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,want", _kat())
def test_philox_known_answers(ctr, key, want):
    got = P.philox4x32_10(np.array(ctr, np.uint64), np.array(key, np.uint64))
    assert [int(x) for x in got] == want


def test_philox_vectorised_matches_scalar():
    ctr = np.array([[i, 7, 0, 3] for i in range(5)], np.uint64)
    many = P.philox4x32_10(ctr, np.array([1, 2], np.uint64))
    for i in range(5):
        assert np.array_equal(many[i], P.philox4x32_10(ctr[i], np.array([1, 2], np.uint64)))


def test_sampling_edges_and_determinism():
    p0 = np.zeros((2, 8, 16), np.float32)
    m, idx = P.sample_execution_grid(p0, 11, 3)
    assert not m.any() and idx.size == 0                      # p = 0: never executed
    m, idx = P.sample_execution_grid(np.ones_like(p0), 11, 3)
    assert m.all() and np.array_equal(idx, np.arange(256))    # p = 1: u < 1 always
    r = synth.rng(4)
    p = r.uniform(0, 1, (2, 8, 16)).astype(np.float32)
    a, _ = P.sample_execution_grid(p, 11, 3)
    b, _ = P.sample_execution_grid(p, 11, 3)
    c, _ = P.sample_execution_grid(p, 11, 4)
    assert np.array_equal(a, b) and not np.array_equal(a, c)  # fixed by (seed, frame)


def test_sampling_is_monotone_in_p():
    """The same uniform u_b decides every probability: raising p never removes a block."""
    r = synth.rng(5)
    p1 = r.uniform(0, 1, (1, 32, 64)).astype(np.float32)
    p2 = np.minimum(p1 + r.uniform(0, 0.3, p1.shape).astype(np.float32), 1).astype(np.float32)
    m1, _ = P.sample_execution_grid(p1, 99, 0)
    m2, _ = P.sample_execution_grid(p2, 99, 0)
    assert not (m1 & ~m2).any()


@pytest.mark.parametrize("p", [0.1, 0.25, 0.5, 0.9])
def test_sampling_frequency(p):
    """Bernoulli(p): the executed fraction over 2^16 blocks is within 5 sigma of p."""
    m, _ = P.sample_execution_grid(np.full((4, 128, 128), p, np.float32), 2021, 17)
    sigma = math.sqrt(p * (1 - p) / m.size)
    assert abs(m.mean() - p) < 5 * sigma


def test_uniforms_are_24_bit_and_in_range():
    u = P.block_uniforms(2, 64, 64, 5, 6)
    assert (u >= 0).all() and (u < 1).all()
    assert np.array_equal(u * 2 ** 24, np.floor(u * 2 ** 24))
    assert scipy.stats.kstest(u.ravel(), "uniform").pvalue > 1e-4


# ------------------------------------------------------------------ frame state

@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_frame_state_select(layout):
    r = synth.rng(6)
    shape = (2, 3, 16, 24) if layout == "nchw" else (2, 16, 24, 3)
    frame = synth.to_storage_bits(synth.normal(r, shape), "bf16")
    state = synth.nan_canaries(r, shape, "bf16")
    zeros = np.zeros((2, 4, 3), np.uint8)
    assert np.array_equal(P.update_frame_state(frame, state, zeros, layout), state)
    assert np.array_equal(P.update_frame_state(frame, state, np.ones_like(zeros), layout), frame)
    mask = synth.bernoulli_mask(r, 2, 4, 3, 0.5)
    got = P.update_frame_state(frame, state, mask, layout)
    for n in range(2):
        for y in range(16):
            for x in range(24):
                src = frame if mask[n, y // 4, x // 8] else state
                if layout == "nchw":
                    assert np.array_equal(got[n, :, y, x], src[n, :, y, x])
                else:
                    assert np.array_equal(got[n, y, x, :], src[n, y, x, :])


# ------------------------------------------------------------------ information gain

def test_kl_two_class_closed_form():
    """p = (1/5, 4/5) against q = (1/2, 1/2): KL = 0.2 ln 0.4 + 0.8 ln 1.6."""
    lt = np.array([0.0, math.log(4.0)]).reshape(1, 2, 1, 1)
    lq = np.zeros((1, 2, 1, 1))
    want = 0.2 * math.log(0.4) + 0.8 * math.log(1.6)
    assert abs(P.pixel_kl(lt, lq)[0, 0, 0] - want) < 1e-14


def test_kl_matches_library_entropy():
    r = synth.rng(7)
    lt = r.normal(0, 2, (1, 19, 4, 5))
    lq = r.normal(0, 2, (1, 19, 4, 5))
    got = P.pixel_kl(lt, lq)
    for y in range(4):
        for x in range(5):
            p = np.exp(lt[0, :, y, x]) / np.exp(lt[0, :, y, x]).sum()
            q = np.exp(lq[0, :, y, x]) / np.exp(lq[0, :, y, x]).sum()
            assert abs(got[0, y, x] - scipy.stats.entropy(p, q)) < 1e-12


def test_kl_invariants():
    r = synth.rng(8)
    lt = r.normal(0, 3, (2, 19, 6, 6))
    lq = r.normal(0, 3, (2, 19, 6, 6))
    kl = P.pixel_kl(lt, lq)
    assert (kl >= -1e-12).all()                                       # Gibbs' inequality
    assert np.abs(P.pixel_kl(lt, lt)).max() < 1e-12                   # no change, no gain
    shift = r.normal(0, 5, (2, 1, 6, 6))                              # softmax shift invariance
    assert np.abs(P.pixel_kl(lt + shift, lq - shift) - kl).max() < 1e-10


def test_information_gain_block_max_brute_force():
    r = synth.rng(9)
    lt = r.normal(0, 1, (2, 5, 8, 12))
    lq = r.normal(0, 1, (2, 5, 8, 12))
    ig = P.seg_information_gain(lt, lq, 2, 3)
    kl = P.pixel_kl(lt, lq)
    for n in range(2):
        for gy in range(2):
            for gx in range(3):
                best = max(kl[n, y, x] for y in range(gy * 4, gy * 4 + 4) for x in range(gx * 4, gx * 4 + 4))
                assert ig[n, gy, gx] == best


# ------------------------------------------------------------------ rewards and loss

def test_rewards_worked_example():
    """gamma = 5 and mu = 0.9 as in the paper's configuration; tau = 0.5. Executed
    blocks (0,0) and (1,1): C_t = 0.5; with M_{t-1} = 0.7, M_t = 0.1*0.5 + 0.9*0.7 =
    0.68, so tau - M_t = -0.18 and gamma * (tau - M_t) = -0.9. R = IG - 0.9 for executed
    blocks, -IG + 0.9 for the others."""
    ig = np.array([[[0.4, 0.1], [0.0, 0.25]]])
    mask = np.array([[[1, 0], [0, 1]]], np.uint8)
    r, c, m = P.block_rewards(ig, mask, tau=0.5, gamma=5.0, mu=0.9, m_prev=[0.7])
    assert c[0] == 0.5 and abs(m[0] - 0.68) < 1e-15
    assert np.abs(r - np.array([[[-0.5, 0.8], [0.9, -0.65]]])).max() < 1e-12
    # L = -(R log pi): pi = 0.8, 1 - 0.25, 1 - 0.5, 0.6 for the four blocks
    prob = np.array([[[0.8, 0.25], [0.5, 0.6]]], np.float32)
    want = -(-0.5 * math.log(0.8) + 0.8 * math.log(0.75) + 0.9 * math.log(0.5) - 0.65 * math.log(0.6))
    assert abs(P.reinforce_loss(r, mask, prob)[0] - want) < 1e-7    # prob is fp32
    assert abs(want - 0.41036968936037666) < 1e-12


def test_rewards_sign_structure():
    """Executed and non-executed copies of one block get opposite rewards."""
    r = synth.rng(10)
    ig = r.uniform(0, 1, (1, 4, 4))
    ones = np.ones((1, 4, 4), np.uint8)
    ra, ca, ma = P.block_rewards(ig, ones, 0.3, 5.0, 0.9, [0.4])
    zeros = np.zeros_like(ones)
    rb, cb, mb = P.block_rewards(ig, zeros, 0.3, 5.0, 0.9, [0.4])
    assert ca[0] == 1 and cb[0] == 0
    assert np.allclose(ra, ig + 5.0 * (0.3 - ma[0])) and np.allclose(rb, -ig - 5.0 * (0.3 - mb[0]))
