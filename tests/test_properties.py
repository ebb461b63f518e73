"""Property tests (CPU, hypothesis) of the oracle and of the C ABI's argument checks
over random shapes and execution grids: empty, single-block, checkerboard, border-only
and random masks.

Oracle (Section 3.1: executed blocks take the layer's result, every other block keeps
the previous execution's bits):
* executed blocks equal the dense layer rounded to the storage format, every other
  element keeps the previous bits (NaN canaries included);
* the only-active mode gives the same bits as dense-then-select;
* the index is the ascending list of nonzero grid entries (Section 3.5);
* a static frame (the same input again, any grid) reproduces the full frame's output.
C ABI: for random geometries the status of bc_sparse_conv2d is the one the documented
rules predict, checked before anything is enqueued (fake device addresses; no GPU).
"""
import ctypes

import numpy as np
import pytest
from hypothesis import HealthCheck, assume, given, settings
from hypothesis import strategies as st

import oracle
import synth

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def make_mask(kind, n, gh, gw, seed):
    m = np.zeros((n, gh, gw), np.uint8)
    if kind == "empty":
        pass
    elif kind == "single":
        r = synth.rng(seed)
        m[r.integers(n), r.integers(gh), r.integers(gw)] = 1
    elif kind == "checker":
        m[:] = (np.add.outer(np.arange(gh), np.arange(gw)) % 2 == 0)[None]
    elif kind == "border":
        m[:, 0, :] = m[:, -1, :] = 1
        m[:, :, 0] = m[:, :, -1] = 1
    elif kind == "full":
        m[:] = 1
    else:
        m = synth.bernoulli_mask(synth.rng(seed), n, gh, gw, 0.4)
    return m


MASKS = st.sampled_from(["empty", "single", "checker", "border", "full", "random"])


@st.composite
def layer_case(draw):
    k = draw(st.sampled_from([1, 3, 5]))
    s = draw(st.sampled_from([1, 2]))
    gh, gw = draw(st.integers(1, 3)), draw(st.integers(1, 4))
    bh, bw = draw(st.integers(1, 4)), draw(st.integers(1, 4))
    ho, wo = gh * bh, gw * bw
    pad = k // 2
    # input size whose conv output is exactly ho x wo
    h, w = (ho - 1) * s + k - 2 * pad, (wo - 1) * s + k - 2 * pad
    h, w = max(h, 1), max(w, 1)
    if oracle.out_size(h, k, s, pad) != ho or oracle.out_size(w, k, s, pad) != wo:
        h, w = ho * s, wo * s
    n = draw(st.integers(1, 2))
    cin, cout = draw(st.integers(1, 4)), draw(st.integers(1, 4))
    return dict(n=n, cin=cin, cout=cout, h=h, w=w, k=k, s=s, pad=pad, gh=gh, gw=gw,
                mask=draw(MASKS), seed=draw(st.integers(0, 10 ** 6)), res=draw(st.booleans()),
                relu=draw(st.booleans()), dtype=draw(st.sampled_from(["bf16", "f16", "f32"])))


@SETTINGS
@given(layer_case())
def test_oracle_select_and_only_active(c):
    r = synth.rng(c["seed"])
    ho = oracle.out_size(c["h"], c["k"], c["s"], c["pad"])
    wo = oracle.out_size(c["w"], c["k"], c["s"], c["pad"])
    assume(ho % c["gh"] == 0 and wo % c["gw"] == 0)   # the ABI rejects other outputs
    dt = c["dtype"]
    x = synth.to_storage_bits(synth.normal(r, (c["n"], c["cin"], c["h"], c["w"])), dt)
    wt = synth.to_storage_bits(synth.he_normal(r, c["cout"], c["cin"], c["k"], c["k"]), dt)
    bias = synth.normal(r, c["cout"], 0.1).astype(np.float32)
    res = synth.to_storage_bits(synth.normal(r, (c["n"], c["cout"], ho, wo)), dt) if c["res"] else None
    prev = synth.nan_canaries(r, (c["n"], c["cout"], ho, wo), dt)
    mask = make_mask(c["mask"], c["n"], c["gh"], c["gw"], c["seed"])
    args = (x, wt, mask, prev, dt, c["s"], c["pad"], bias, res, c["relu"])
    y = oracle.sparse_conv2d(*args)
    assert np.array_equal(y, oracle.sparse_conv2d_active(*args))
    sel = np.broadcast_to(oracle.expand_mask(mask, ho // c["gh"], wo // c["gw"]), y.shape)
    assert np.array_equal(y[~sel], prev[~sel])
    dense = oracle.store(oracle.conv2d_dense(oracle.value(x, dt), oracle.value(wt, dt),
                                             bias.astype(np.float64),
                                             None if res is None else oracle.value(res, dt),
                                             c["s"], c["pad"], c["relu"]), dt)
    assert np.array_equal(y[sel], dense[sel])


@SETTINGS
@given(st.integers(1, 3), st.integers(1, 9), st.integers(1, 17), MASKS, st.integers(0, 10 ** 6))
def test_oracle_index_is_ascending_nonzero(n, gh, gw, kind, seed):
    m = make_mask(kind, n, gh, gw, seed)
    idx, cnt = oracle.block_index(m)
    assert cnt == int((m != 0).sum()) and idx.dtype == np.int32
    assert np.all(np.diff(idx) > 0)
    flat = m.reshape(-1)
    assert all(flat[i] for i in idx)


@SETTINGS
@given(layer_case())
def test_oracle_static_frame(c):
    """Running the same input again with any grid over the full frame's output keeps
    every bit (halos read from copied neighbours hold the dense values)."""
    r = synth.rng(c["seed"])
    ho = oracle.out_size(c["h"], c["k"], c["s"], c["pad"])
    wo = oracle.out_size(c["w"], c["k"], c["s"], c["pad"])
    assume(ho % c["gh"] == 0 and wo % c["gw"] == 0)
    dt = "bf16"
    x = synth.to_storage_bits(synth.normal(r, (c["n"], c["cin"], c["h"], c["w"])), dt)
    wt = synth.to_storage_bits(synth.he_normal(r, c["cout"], c["cin"], c["k"], c["k"]), dt)
    zero = np.zeros((c["n"], c["cout"], ho, wo), np.uint16)
    full = oracle.sparse_conv2d(x, wt, np.ones((c["n"], c["gh"], c["gw"]), np.uint8), zero, dt,
                                c["s"], c["pad"], None, None, c["relu"])
    again = oracle.sparse_conv2d(x, wt, make_mask(c["mask"], c["n"], c["gh"], c["gw"], c["seed"]),
                                 full, dt, c["s"], c["pad"], None, None, c["relu"])
    assert np.array_equal(full, again)


# ------------------------------------------------------------------ C ABI checks

no_gpu = pytest.mark.skipif(__import__("torch").cuda.is_available(),
                            reason="fake device pointers are used only on machines without a GPU")
FAKE_IN, FAKE_W, FAKE_OUT = 0x10000000, 0x20000000, 0x30000000
FAKE_IDX, FAKE_CNT = 0x50000000, 0x60000000


def expected_status(B, c):
    """The status the documented rules of include/bc.h give a bc_sparse_conv2d call."""
    k, s, pad = c["k"], c["s"], c["pad"]
    oh_geom = (c["h"] + 2 * pad - k) // s + 1
    ow_geom = (c["w"] + 2 * pad - k) // s + 1
    if (c["oh"], c["ow"]) != (oh_geom, ow_geom):
        return B.BC_ERR_SHAPE
    if c["oh"] % c["gh"] or c["ow"] % c["gw"]:
        return B.BC_ERR_NOT_DIVISIBLE
    if c["cap"] < c["gh"] * c["gw"]:
        return B.BC_ERR_CAPACITY
    return None                                  # passes the shape checks


@no_gpu
@SETTINGS
@given(st.sampled_from([1, 3, 5, 7]), st.sampled_from([1, 2]), st.integers(1, 6), st.integers(1, 9),
       st.integers(4, 40), st.integers(4, 40), st.integers(-2, 2), st.integers(-2, 2),
       st.integers(0, 200), st.sampled_from([8, 16, 64, 128]), st.sampled_from([64, 128]))
def test_abi_conv_status_matches_the_rules(k, s, gh, gw, h, w, dh, dw, cap, cin, cout):
    from paper_2108_09376_amd import bc as B
    pad = k // 2
    oh, ow = (h + 2 * pad - k) // s + 1 + dh, (w + 2 * pad - k) // s + 1 + dw
    assume(oh > 0 and ow > 0)
    c = dict(k=k, s=s, pad=pad, gh=gh, gw=gw, h=h, w=w, oh=oh, ow=ow, cap=cap)
    lib = B.raw()
    conv = B.bc_conv(k, k, s, pad, 1)
    st_ = lib.bc_sparse_conv2d(ctypes.byref(conv), FAKE_IN, B.bc_tensor(1, cin, h, w, B.BC_BF16, B.BC_NHWC),
                               FAKE_W, None, None, FAKE_OUT, B.bc_tensor(1, cout, oh, ow, B.BC_BF16, B.BC_NHWC),
                               B.bc_grid(gh, gw), FAKE_IDX, FAKE_CNT, cap, None)
    want = expected_status(B, c)
    if want is not None:
        assert st_ == want, (c, B.bc_last_error())
    else:
        # every shape check passed: the call is either unsupported by the kernels (a
        # block too wide for a tile, a halo too large for LDS) or reaches the launch,
        # which fails without a GPU
        assert st_ in (B.BC_ERR_UNSUPPORTED, B.BC_ERR_HIP), (c, st_, B.bc_last_error())
