"""CPU oracle for the steps around the block-sparse network: execution-grid sampling,
frame-state update, information gain for semantic segmentation and the block rewards.

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the CPU baseline leg of ``bench.py`` may use it, and
it shares no code with the HIP library. Plain numpy in float64 (the sampling decision
excepted, see below), written from the paper's definitions:

* Section 3.5: the policy gives an execution probability p_b per block; execution
  decisions a_b in {0, 1} are drawn from them (stochastic sampling, not a threshold).
  The paper does not say which random generator is used. Reading: a_b = 1 when
  u_b < p_b, with u_b uniform in [0, 1) taken from Philox4x32-10 (Salmon, Moraes,
  Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), counter
  (b, frame mod 2^32, frame div 2^32, 0) and key (seed mod 2^32, seed div 2^32), where
  b = (img * Gh + gy) * Gw + gx; u_b = (first output word >> 8) * 2^-24. Both u_b and
  the fp32 probability are exact in float64, so the comparison is the same in any
  precision that holds them.
* Section 3.3: the frame state H_t is an RGB frame in which every block holds the
  image content of the last executed block at that position:
  H_t = select(A_t, I_t, H_{t-1}), bit for bit.
* Section 3.4: information gain per output pixel, semantic segmentation: the KL
  divergence between the output distributions of frame t and frame t-1; per block, the
  maximum over its pixels (Eq. 1). Readings: the direction is KL(O_t || O_{t-1});
  the network hands over per-class scores (logits) and O = softmax over classes.
* Section 3.3 and Eq. 2: the policy network maps S_t = {I_t, H_{t-1}, A_{t-1}, O_{t-1}}
  to one execution probability per block. The architecture is given only as a figure
  (an 8-layer ResNet backbone with a fully convolutional head, about 6.5 GMACs on a
  2048x1024 frame, the extra inputs adding about 0.1 GMAC). Reading: S_t is assembled
  at a quarter of the frame resolution, where O_{t-1} lives, as 32 channels (the
  frame and the frame state averaged over 4x4 pixels, the class probabilities of
  O_{t-1}, A_{t-1} of the pixel's block, zeros); the network ends in a map with one
  pixel per block whose channel 0 is the block's logit, p_b = sigmoid(logit).
* Section 4 (configuration): the policy is trained online with RMSprop (learning rate
  1e-4, weight decay 1e-3), updating every 4 frames. The gradient is that of the
  REINFORCE loss L = -sum_b R_b log pi(a_b) with pi(1) = p_b = sigmoid(z_b): dL/dz_b =
  -R_b (a_b - p_b), back through the network's layers (readings: the batch-norm
  statistics of the random initialisation are folded into the convolutions, which are
  what is trained; RMSprop as PyTorch defines it, smoothing 0.99, eps 1e-8, weight
  decay added to the gradient).
* Section 3.5: rewards. R_IG = IG_b if a_b = 1, else -IG_b. C_t = fraction of executed
  blocks of the frame. M_t = (1 - mu) C_t + mu M_{t-1}, reading the printed C_{t-1} as
  the previous moving average M_{t-1} (the text calls M a moving average with
  momentum). R_cost = tau - M_t if a_b = 1, else -(tau - M_t). R_b = R_IG + gamma
  R_cost. REINFORCE loss L = -sum_b R_b log pi(a_b), pi(1) = p_b, pi(0) = 1 - p_b.
"""
from __future__ import annotations

import numpy as np

# Philox4x32 constants from the published definition (multipliers and Weyl key bumps).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(counter, key):
    """Philox4x32 with 10 rounds. counter: uint array [..., 4], key: uint array [..., 2]
    (broadcast against each other). Returns uint32 [..., 4].

    One round: (hi0, lo0) = M0 * c0 and (hi1, lo1) = M1 * c2 as 64-bit products;
    output (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0). Between rounds the key is bumped
    by the Weyl constants (W0, W1), mod 2^32."""
    c = np.asarray(counter, dtype=np.uint64) & MASK32
    k = np.asarray(key, dtype=np.uint64) & MASK32
    lead = np.broadcast_shapes(c.shape[:-1], k.shape[:-1])
    c = np.broadcast_to(c, lead + (4,))
    k = np.broadcast_to(k, lead + (2,))
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = k[..., 0].copy(), k[..., 1].copy()
    for r in range(10):
        if r:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = c0 * np.uint64(PHILOX_M0)
        p1 = c2 * np.uint64(PHILOX_M1)
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def block_uniforms(n: int, gh: int, gw: int, seed: int, frame: int) -> np.ndarray:
    """u_b in [0, 1) for every block of an [n, gh, gw] grid (float64, exact)."""
    b = np.arange(n * gh * gw, dtype=np.uint64)
    ctr = np.zeros((b.size, 4), np.uint64)
    ctr[:, 0] = b
    ctr[:, 1] = frame & MASK32
    ctr[:, 2] = (frame >> 32) & MASK32
    key = np.zeros((b.size, 2), np.uint64)
    key[:, 0] = seed & MASK32
    key[:, 1] = (seed >> 32) & MASK32
    x0 = philox4x32_10(ctr, key)[:, 0].astype(np.float64)
    return (np.floor(x0 / 256.0) * 2.0 ** -24).reshape(n, gh, gw)


def sample_execution_grid(prob, seed: int, frame: int):
    """Execution decisions A_t (uint8 [n, gh, gw]) sampled from the fp32 block
    probabilities P_t, and the active-block index (ascending raster ids)."""
    p = np.asarray(prob, np.float32).astype(np.float64)
    n, gh, gw = p.shape
    u = block_uniforms(n, gh, gw, seed, frame)
    mask = (u < p).astype(np.uint8)
    idx = np.flatnonzero(mask).astype(np.int32)
    return mask, idx


def update_frame_state(frame_bits, state_bits, mask, layout: str = "nchw"):
    """H_t = select(A_t, I_t, H_{t-1}) on raw bit patterns. frame/state: [n, c, h, w]
    (layout "nchw") or [n, h, w, c] ("nhwc"); mask uint8 [n, gh, gw]."""
    f = np.asarray(frame_bits)
    out = np.array(state_bits, copy=True)
    m = np.asarray(mask)
    n, gh, gw = m.shape
    h, w = (f.shape[2], f.shape[3]) if layout == "nchw" else (f.shape[1], f.shape[2])
    bh, bw = h // gh, w // gw
    for img in range(n):
        for gy in range(gh):
            for gx in range(gw):
                if not m[img, gy, gx]:
                    continue
                ys, xs = slice(gy * bh, gy * bh + bh), slice(gx * bw, gx * bw + bw)
                if layout == "nchw":
                    out[img, :, ys, xs] = f[img, :, ys, xs]
                else:
                    out[img, ys, xs, :] = f[img, ys, xs, :]
    return out


def log_softmax(logits, axis: int = 1):
    """log softmax over the class axis, float64 (max-shifted log-sum-exp)."""
    z = np.asarray(logits, np.float64)
    mx = z.max(axis=axis, keepdims=True)
    return z - (mx + np.log(np.exp(z - mx).sum(axis=axis, keepdims=True)))


def pixel_kl(logits, prev_logits):
    """KL(O_t || O_{t-1}) per pixel: sum_c p_c (log p_c - log q_c), O = softmax of the
    [n, classes, h, w] logits. Returns float64 [n, h, w]."""
    lp = log_softmax(logits)
    lq = log_softmax(prev_logits)
    return (np.exp(lp) * (lp - lq)).sum(axis=1)


def seg_information_gain(logits, prev_logits, gh: int, gw: int):
    """IG_b = max over the pixels of block b of the per-pixel KL (Eq. 1). [n, gh, gw]."""
    kl = pixel_kl(logits, prev_logits)
    n, h, w = kl.shape
    bh, bw = h // gh, w // gw
    return kl.reshape(n, gh, bh, gw, bw).max(axis=(2, 4))


def block_rewards(ig, mask, tau: float, gamma: float, mu: float, m_prev):
    """Rewards of Section 3.5 per block. Returns (R [n, gh, gw], C_t [n], M_t [n])."""
    ig = np.asarray(ig, np.float64)
    a = np.asarray(mask) != 0
    n = ig.shape[0]
    cost = a.reshape(n, -1).mean(axis=1)
    m = (1.0 - mu) * cost + mu * np.asarray(m_prev, np.float64).reshape(n)
    r_ig = np.where(a, ig, -ig)
    slack = (tau - m)[:, None, None]
    r_cost = np.where(a, slack, -slack)
    return r_ig + gamma * r_cost, cost, m


def reinforce_loss(reward, mask, prob):
    """L = -sum_b R_b log pi(a_b) per image, pi(1) = p_b, pi(0) = 1 - p_b. [n]."""
    r = np.asarray(reward, np.float64)
    a = np.asarray(mask) != 0
    p = np.asarray(prob, np.float32).astype(np.float64)
    with np.errstate(divide="ignore"):
        logpi = np.where(a, np.log(p), np.log1p(-p))
    return -(r * logpi).reshape(r.shape[0], -1).sum(axis=1)


POLICY_CHANNELS = 32       # channels of S_t


def policy_input(frame_bits, state_bits, score_bits, classes: int, prev_mask, dtype="bf16"):
    """S_t at a quarter of the frame resolution, as storage bits [n, 32, h/4, w/4].

    frame_bits, state_bits: I_t and H_{t-1}, [n, 3, h, w] bits; score_bits: O_{t-1}'s
    per-class scores [n, C, h/4, w/4] bits (the first `classes` channels are used);
    prev_mask: A_{t-1}, uint8 [n, gh, gw] over the frame's block grid, or None (zeros).
    Channels: 0-2 the mean of I_t over each 4x4 pixel cell, 3-5 the same for H_{t-1},
    6 .. 5+classes the softmax over classes of O_{t-1} (its output probabilities),
    6+classes: a_b of the block the pixel lies in, the rest 0. Values in float64,
    stored once (fp64 -> fp32 -> storage format, round to nearest even)."""
    from . import store, value
    f = value(frame_bits, dtype)
    st = value(state_bits, dtype)
    n, _, h, w = f.shape
    h4, w4 = h // 4, w // 4
    z = np.zeros((n, POLICY_CHANNELS, h4, w4))
    z[:, 0:3] = f.reshape(n, 3, h4, 4, w4, 4).mean(axis=(3, 5))
    z[:, 3:6] = st.reshape(n, 3, h4, 4, w4, 4).mean(axis=(3, 5))
    sc = value(score_bits, dtype)[:, :classes]
    z[:, 6:6 + classes] = np.exp(log_softmax(sc, axis=1))
    if prev_mask is not None:
        m = np.asarray(prev_mask) != 0
        gh, gw = m.shape[1:]
        z[:, 6 + classes] = np.repeat(np.repeat(m, h4 // gh, axis=1), w4 // gw, axis=2)
    return store(z, dtype)


def policy_probabilities(logit_bits, dtype="bf16"):
    """p_b = sigmoid(channel 0) of the head's [n, C, gh, gw] output. float64 [n, gh, gw]."""
    from . import value
    v = value(logit_bits, dtype)[:, 0]
    return 1.0 / (1.0 + np.exp(-v))


def logit_grad(reward, mask, prob):
    """dL/dz_b = -R_b (a_b - p_b) of the REINFORCE loss, p_b = sigmoid(z_b). [n, gh, gw]."""
    a = (np.asarray(mask) != 0).astype(np.float64)
    return -np.asarray(reward, np.float64) * (a - np.asarray(prob, np.float64))


def policy_backward(table, weights, biases, x, dz, stored=None, return_maps=False):
    """Gradients of L with respect to every layer's weights and bias, float64.

    weights[l]: [cout, cin, k, k] (OIHW), biases[l]: [cout], x: S_t [n, 32, h, w] values,
    dz: dL/dz [n, gh, gw] for channel 0 of the last layer. The reverse pass uses the
    forward pass's activations: `stored` (one array of values per layer, e.g. the
    storage-rounded maps a forward pass kept, as the device keeps them), or, if None,
    the forward pass recomputed in float64 without rounding. It visits the layers in reverse
    order: through the ReLU (where the output is > 0), then the weight gradient (the
    correlation of the layer's input with the output gradient), the bias gradient (its
    sum) and the input gradient (the transposed convolution), added to every producer
    that the layer reads (its source, and its residual source as is). torch's conv
    primitives in float64 are the steps (layer_backward). Returns (dW list, db list), and
    with return_maps also each layer's gated output gradient (the gp of layer_backward)."""
    import torch
    import torch.nn.functional as F
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    xs = t(x)
    ys = []
    if stored is not None:
        ys = [t(a) for a in stored]
    else:
        for l, w, b in zip(table, weights, biases):
            src = xs if l["src"] < 0 else ys[l["src"]]
            y = F.conv2d(src, t(w), t(b), stride=l["stride"], padding=l["pad"])
            if l["res"] is not None:
                y = y + ys[l["res"]]
            ys.append(torch.relu(y) if l["relu"] else y)
    g = [torch.zeros_like(y) for y in ys]
    g[-1][:, 0] = t(dz)
    dw, db = [None] * len(table), [None] * len(table)
    gps = [None] * len(table)
    for li in range(len(table) - 1, -1, -1):
        l = table[li]
        gp = g[li] * (ys[li] > 0) if l["relu"] else g[li]
        gps[li] = gp.numpy()
        src = xs if l["src"] < 0 else ys[l["src"]]
        dw[li], db[li], dx = layer_backward(l, weights[li], src.numpy(), gp.numpy())
        if l["src"] >= 0:
            g[l["src"]] += t(dx)
        if l["res"] is not None:
            g[l["res"]] += gp
    if return_maps:
        return dw, db, gps
    return dw, db


def layer_backward(layer, weight, src, gp):
    """One layer's step of the reverse pass, float64: the weight gradient (the correlation
    of the layer's input `src` with its output gradient `gp`, taken after the ReLU gate),
    the bias gradient (the sum of gp over images and pixels) and the input gradient (the
    transposed convolution of gp with the layer's weights). Returns (dW, db, dX)."""
    import torch
    from torch.nn.grad import conv2d_input, conv2d_weight
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    src, gp, w = t(src), t(gp), t(weight)
    dw = conv2d_weight(src, w.shape, gp, stride=layer["stride"], padding=layer["pad"]).numpy()
    db = gp.sum(dim=(0, 2, 3)).numpy()
    dx = conv2d_input(src.shape, w, gp, stride=layer["stride"], padding=layer["pad"]).numpy()
    return dw, db, dx


def rmsprop_step(w, v, grad, lr=1e-4, alpha=0.99, eps=1e-8, weight_decay=1e-3):
    """One RMSprop step as PyTorch defines it (no momentum, not centered):
    g = grad + weight_decay * w; v = alpha v + (1 - alpha) g^2; w = w - lr g / (sqrt(v) + eps).
    float64; returns (w, v)."""
    w = np.asarray(w, np.float64)
    g = np.asarray(grad, np.float64) + weight_decay * w
    v = alpha * np.asarray(v, np.float64) + (1.0 - alpha) * g * g
    return w - lr * g / (np.sqrt(v) + eps), v
