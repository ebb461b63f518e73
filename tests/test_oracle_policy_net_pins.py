"""Pins of the policy-network part of the oracle (Section 3.3, Eq. 2; the architecture
reading is in oracle/policy.py): the assembly of S_t against per-pixel loops, library
routines and exact constants, the sigmoid against scipy, the network table against the
paper's cost figure, and the dense network against a torch-built reference; for the
online training, the reverse pass against central finite differences of the loss, the
logit gradient against its closed form, and the RMSprop step against torch.optim."""
import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import network as net
from oracle import policy as P


def _inputs(seed, n=1, h=16, w=32, classes=5, c=8, gh=2, gw=4):
    r = synth.rng(seed)
    fr = synth.to_storage_bits(synth.normal(r, (n, 3, h, w)), "bf16")
    st = synth.to_storage_bits(synth.normal(r, (n, 3, h, w)), "bf16")
    sc = synth.to_storage_bits(synth.normal(r, (n, c, h // 4, w // 4), 3.0), "bf16")
    m = synth.bernoulli_mask(r, n, gh, gw, 0.5)
    return fr, st, sc, m


def test_policy_input_brute_force():
    """Every output value by explicit loops over pixels and classes."""
    fr, st, sc, m = _inputs(1, n=2)
    classes = 5
    got = oracle.value(P.policy_input(fr, st, sc, classes, m), "bf16")
    f, s, c = (oracle.value(b, "bf16") for b in (fr, st, sc))
    n, _, h, w = f.shape
    gh, gw = m.shape[1:]
    want = np.zeros((n, 32, h // 4, w // 4))
    for i in range(n):
        for y in range(h // 4):
            for x in range(w // 4):
                for ch in range(3):
                    want[i, ch, y, x] = sum(f[i, ch, 4 * y + dy, 4 * x + dx] for dy in range(4)
                                            for dx in range(4)) / 16.0
                    want[i, 3 + ch, y, x] = sum(s[i, ch, 4 * y + dy, 4 * x + dx] for dy in range(4)
                                                for dx in range(4)) / 16.0
                e = [np.exp(c[i, k, y, x]) for k in range(classes)]
                for k in range(classes):
                    want[i, 6 + k, y, x] = e[k] / sum(e)
                want[i, 6 + classes, y, x] = m[i, y // ((h // 4) // gh), x // ((w // 4) // gw)]
    assert np.array_equal(got, oracle.value(oracle.store(want, "bf16"), "bf16"))


def test_policy_input_constants_and_library_softmax():
    fr, st, sc, _ = _inputs(2)
    fr[:] = synth.to_storage_bits(np.full(fr.shape, 1.5, np.float32), "bf16")
    got = oracle.value(P.policy_input(fr, st, sc, 5, None), "bf16")
    assert (got[:, 0:3] == 1.5).all()                     # the mean of equal values
    assert (got[:, 6 + 5:] == 0.0).all()                  # no previous grid, zero padding
    ref = scipy.special.softmax(oracle.value(sc, "bf16")[:, :5], axis=1)
    np.testing.assert_allclose(got[:, 6:11], ref, rtol=2 ** -7)
    np.testing.assert_allclose(got[:, 6:11].sum(axis=1), 1.0, rtol=2e-2)


def test_policy_probabilities_against_expit():
    r = synth.rng(3)
    lg = synth.to_storage_bits(synth.normal(r, (2, 64, 8, 16), 4.0), "bf16")
    p = P.policy_probabilities(lg)
    v = oracle.value(lg, "bf16")[:, 0]
    np.testing.assert_allclose(p, scipy.special.expit(v), rtol=1e-12)
    zero = synth.to_storage_bits(np.zeros((1, 64, 8, 16), np.float32), "bf16")
    assert (P.policy_probabilities(zero) == 0.5).all()


def test_policy_table_cost_and_output_grid():
    """About the 6.5 GMACs the paper gives for its ResNet-8 policy on a 2048x1024 frame,
    and one output pixel per 128-pixel block (the 8x16 grid)."""
    t = net.policy_table()
    sh = net.shapes(t, 256, 512)                          # S_t of a 2048x1024 frame
    macs = sum(l["cin"] * l["cout"] * l["k"] ** 2 * s[1] * s[2] for l, s in zip(t, sh))
    assert abs(macs / 6.5e9 - 1.0) < 0.1
    assert sh[-1][1:] == (8, 16)
    main = [l for l in t if "downsample" not in l["name"] and "head" not in l["name"]]
    assert len(main) == 7                                 # stem + three blocks of two


def _torch_dense(table, folded, x_bits):
    def st(t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    outs = []
    x = torch.from_numpy(synth.storage_to_f64(x_bits, "bf16"))
    for li, l in enumerate(table):
        src = x if l["src"] < 0 else outs[l["src"]]
        w = torch.from_numpy(synth.storage_to_f64(folded[li]["w_bits"], "bf16"))
        b = torch.from_numpy(folded[li]["bias"].astype(np.float64))
        y = F.conv2d(src, w, b, stride=l["stride"], padding=l["pad"])
        if l["res"] is not None:
            y = y + outs[l["res"]]
        if l["relu"]:
            y = torch.relu(y)
        outs.append(st(y))
    return outs


def test_policy_dense_network_equals_library_reference():
    table = net.policy_table()
    folded = net.fold_params(table, net.make_params(table, seed0=3000), "bf16")
    x = synth.to_storage_bits(synth.normal(synth.rng(4), (1, 32, 64, 128)), "bf16")
    got = net.dense_frame(table, folded, x, "bf16")
    ref = _torch_dense(table, folded, x)
    for li in range(len(table)):
        g, wv = oracle.value(got[li], "bf16"), ref[li].numpy()
        assert (g != wv).mean() < 1e-3, li               # 1-ulp flips on rounding boundaries
        np.testing.assert_allclose(g, wv, rtol=2 ** -7, atol=1e-30)


# ------------------------------------------------------------------ online training

def _tiny_policy():
    """The policy table's layer kinds at a few channels (fast finite differences):
    stride-2 3x3, stride-1 3x3 with a residual, a 1x1/2 projection, a no-ReLU head."""
    def conv(name, src, cin, cout, k, s, relu, res=None):
        return dict(kind="conv", name=name, src=src, res=res, cin=cin, cout=cout, k=k,
                    stride=s, pad=k // 2, relu=relu)
    return [conv("stem", -1, 3, 4, 3, 2, True), conv("c1", 0, 4, 4, 3, 1, True, res=0),
            conv("ds", 1, 4, 6, 1, 2, False), conv("c2", 1, 4, 6, 3, 2, True),
            conv("c3", 3, 6, 6, 3, 1, True, res=2), conv("head", 4, 6, 2, 3, 2, False)]


def _loss(table, ws, bs, x, dz):
    """sum over blocks of dz * z (a linear functional with gradient dz at the logits)."""
    ys = []
    for l, w, b in zip(table, ws, bs):
        src = x if l["src"] < 0 else ys[l["src"]]
        y = F.conv2d(torch.from_numpy(src) if isinstance(src, np.ndarray) else src,
                     torch.from_numpy(w), torch.from_numpy(b), stride=l["stride"], padding=l["pad"])
        if l["res"] is not None:
            y = y + ys[l["res"]]
        ys.append(torch.relu(y) if l["relu"] else y)
    return float((ys[-1][:, 0] * torch.from_numpy(dz)).sum())


def test_policy_backward_finite_differences():
    """Central differences of the loss against the reverse pass, per layer."""
    table = _tiny_policy()
    r = synth.rng(7)
    ws = [r.normal(0, 0.5, (l["cout"], l["cin"], l["k"], l["k"])) for l in table]
    bs = [r.normal(0, 0.1, l["cout"]) for l in table]
    x = r.normal(0, 1, (1, 3, 16, 16))
    dz = r.normal(0, 1, (1, 2, 2))
    dw, db = P.policy_backward(table, ws, bs, x, dz)
    h = 1e-6
    for li in range(len(table)):
        for _ in range(4):
            idx = tuple(int(r.integers(0, s)) for s in ws[li].shape)
            wp = [w.copy() for w in ws]
            wm = [w.copy() for w in ws]
            wp[li][idx] += h
            wm[li][idx] -= h
            fd = (_loss(table, wp, bs, x, dz) - _loss(table, wm, bs, x, dz)) / (2 * h)
            assert abs(fd - dw[li][idx]) <= 1e-6 * max(1.0, abs(fd)), (li, idx)
        c = int(r.integers(0, table[li]["cout"]))
        bp = [b.copy() for b in bs]
        bm = [b.copy() for b in bs]
        bp[li][c] += h
        bm[li][c] -= h
        fd = (_loss(table, ws, bp, x, dz) - _loss(table, ws, bm, x, dz)) / (2 * h)
        assert abs(fd - db[li][c]) <= 1e-6 * max(1.0, abs(fd)), (li, "bias")


def test_policy_backward_with_stored_activations():
    """Handing the reverse pass the exact forward activations changes nothing; handing it
    storage-rounded ones changes the result only through those activations."""
    table = _tiny_policy()
    r = synth.rng(9)
    ws = [r.normal(0, 0.5, (l["cout"], l["cin"], l["k"], l["k"])) for l in table]
    bs = [r.normal(0, 0.1, l["cout"]) for l in table]
    x = r.normal(0, 1, (1, 3, 16, 16))
    dz = r.normal(0, 1, (1, 2, 2))
    ys = []
    for l, w, b in zip(table, ws, bs):
        src = torch.from_numpy(x) if l["src"] < 0 else ys[l["src"]]
        y = F.conv2d(src, torch.from_numpy(w), torch.from_numpy(b), stride=l["stride"], padding=l["pad"])
        if l["res"] is not None:
            y = y + ys[l["res"]]
        ys.append(torch.relu(y) if l["relu"] else y)
    a = P.policy_backward(table, ws, bs, x, dz)
    b = P.policy_backward(table, ws, bs, x, dz, stored=[y.numpy() for y in ys])
    for u, v in zip(a[0] + a[1], b[0] + b[1]):
        assert np.array_equal(u, v)
    c = P.policy_backward(table, ws, bs, x, dz, stored=[oracle.value(oracle.store(y.numpy(), "bf16"), "bf16") for y in ys])
    assert not all(np.array_equal(u, v) for u, v in zip(a[0], c[0]))


def test_logit_grad_closed_form():
    """d/dz of -R log sigmoid(z) is -R (1 - p); of -R log(1 - sigmoid(z)) it is R p."""
    r = np.array([[[2.0, -1.0]]])
    p = np.array([[[0.25, 0.75]]])
    g = P.logit_grad(r, np.array([[[1, 0]]], np.uint8), p)
    np.testing.assert_allclose(g, [[[-2.0 * 0.75, -1.0 * 0.75]]])


def test_rmsprop_matches_torch():
    r = synth.rng(8)
    w0 = r.normal(0, 1, 50)
    grads = [r.normal(0, 1, 50) for _ in range(3)]
    pt = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    opt = torch.optim.RMSprop([pt], lr=1e-4, alpha=0.99, eps=1e-8, weight_decay=1e-3)
    w, v = w0.copy(), np.zeros(50)
    for g in grads:
        pt.grad = torch.from_numpy(g.copy())
        opt.step()
        w, v = P.rmsprop_step(w, v, g)
    np.testing.assert_allclose(w, pt.detach().numpy(), rtol=1e-12, atol=1e-15)
