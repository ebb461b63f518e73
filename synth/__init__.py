"""Seeded synthetic inputs for the block-sparse convolution hot path.

This module is input infrastructure only. It is shared by the CPU oracle (tests)
and the HIP path (tests, bench) and holds none of the method's arithmetic: it draws
weights, feature maps, block masks and video clips, and converts drawn fp32 values to
the bf16/fp16 storage formats with torch's own conversion routines.

The inputs stand in for the 2048x1024 Cityscapes / CityPersons video frames that the
paper evaluates on (Section 4, Datasets). Those datasets are not available; only
their shape (2048x1024x3, 20-frame clips) and the structure of block masks
(execution grids, Section 3.1 and Eq. 3) are reproduced.

Seeds follow one convention everywhere: weights ``1000 + layer_idx``, input features
``1``, previous-output buffers ``2``, masks ``3 + frame``. Generators use
``numpy.random.default_rng(seed)`` (PCG64).
"""
from __future__ import annotations

import numpy as np

SEED_INPUT = 1
SEED_PREV = 2
SEED_MASK0 = 3
SEED_WEIGHT0 = 1000


def rng(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- values

def he_normal(r: np.random.Generator, cout: int, cin: int, kh: int, kw: int) -> np.ndarray:
    """He-normal conv weights, fp32, OIHW [cout, cin, kh, kw]; std = sqrt(2 / (cin*kh*kw))."""
    std = np.sqrt(2.0 / float(cin * kh * kw))
    return (r.standard_normal((cout, cin, kh, kw)) * std).astype(np.float32)


def normal(r: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    """N(0, scale^2) fp32 values of the given shape."""
    return (r.standard_normal(shape) * scale).astype(np.float32)


def small_ints(r: np.random.Generator, shape, lo: int = -4, hi: int = 4) -> np.ndarray:
    """Uniform integers in [lo, hi] as fp32 (exact in every storage format used here)."""
    return r.integers(lo, hi + 1, size=shape).astype(np.float32)


def to_storage_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Store fp32 values in ``dtype`` ('f32', 'bf16', 'f16') using torch's conversion.

    Returns the raw bit patterns: uint32 for f32, uint16 for bf16/f16.
    """
    import torch
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x.view(np.uint32).copy()
    t = torch.from_numpy(x)
    if dtype == "bf16":
        return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()
    if dtype == "f16":
        return t.to(torch.float16).view(torch.int16).numpy().view(np.uint16).copy()
    raise ValueError(dtype)


def storage_to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact value of stored bit patterns, as float64 (a decode, no rounding)."""
    bits = np.ascontiguousarray(bits)
    if dtype == "f32":
        return bits.view(np.float32).astype(np.float64)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    raise ValueError(dtype)


def nan_canaries(r: np.random.Generator, shape, dtype: str) -> np.ndarray:
    """Random bit patterns including NaN payloads, for buffers that must stay untouched."""
    if dtype == "f32":
        b = r.integers(0, 2**32, size=shape, dtype=np.uint64).astype(np.uint32)
        flat = b.reshape(-1)
        flat[::7] = 0x7FC00000 | (flat[::7] & 0x3FFFFF)   # quiet NaNs with payloads
        flat[3::11] = 0x7F800001 | (flat[3::11] & 0x3FFFFF)  # signalling NaN patterns
        return b
    b = r.integers(0, 2**16, size=shape, dtype=np.uint32).astype(np.uint16)
    flat = b.reshape(-1)
    nanbase = 0x7FC0 if dtype == "bf16" else 0x7E00
    flat[::7] = nanbase | (flat[::7] & 0x3F)
    return b


# ---------------------------------------------------------------- masks

def bernoulli_mask(r: np.random.Generator, n: int, gh: int, gw: int, p: float) -> np.ndarray:
    """uint8 [n, gh, gw], each block executed with probability p."""
    return (r.random((n, gh, gw)) < p).astype(np.uint8)


def clustered_mask(r: np.random.Generator, gh: int, gw: int, target: int,
                   k_range=(4, 8), h_range=(1, 4), w_range=(1, 8)) -> np.ndarray:
    """uint8 [gh, gw] with exactly ``target`` nonzero blocks, as a union of rectangles.

    Draw k ~ U{k_range} rectangles (height ~ U{h_range}, width ~ U{w_range}, top-left
    uniform, clipped at the grid edge) and take their union; while fewer than
    ``target`` blocks are set, add more rectangles; then clear blocks of the
    last-added rectangles in reverse raster order until the count equals ``target``.
    """
    target = int(target)
    if not 0 <= target <= gh * gw:
        raise ValueError("target out of range")
    m = np.zeros((gh, gw), np.uint8)
    rects = []

    def add():
        h = int(r.integers(h_range[0], h_range[1] + 1))
        w = int(r.integers(w_range[0], w_range[1] + 1))
        y = int(r.integers(0, gh))
        x = int(r.integers(0, gw))
        rects.append((y, min(gh, y + h), x, min(gw, x + w)))
        m[y:y + h, x:x + w] = 1

    for _ in range(int(r.integers(k_range[0], k_range[1] + 1))):
        add()
    while int(m.sum()) < target:
        add()
    while int(m.sum()) > target:
        y0, y1, x0, x1 = rects.pop()
        for y in range(y1 - 1, y0 - 1, -1):
            for x in range(x1 - 1, x0 - 1, -1):
                if int(m.sum()) == target:
                    break
                # keep blocks still covered by an earlier rectangle
                if m[y, x] and not any(a <= y < b and c <= x < d for a, b, c, d in rects):
                    m[y, x] = 0
        if not rects and int(m.sum()) > target:
            # every rectangle consumed: drop remaining blocks in reverse raster order
            for i in np.flatnonzero(m.reshape(-1))[::-1]:
                if int(m.sum()) == target:
                    break
                m.reshape(-1)[i] = 0
    return m


def frac_mask(seed: int, gh: int, gw: int, frac: float) -> np.ndarray:
    """Clustered mask [1, gh, gw] with round(frac * gh * gw) blocks (1.0 -> all ones)."""
    target = int(round(frac * gh * gw))
    if target == gh * gw:
        return np.ones((1, gh, gw), np.uint8)
    return clustered_mask(rng(seed), gh, gw, target)[None]


# ---------------------------------------------------------------- video clips

def _blur_axis(a: np.ndarray, sigma: float, axis: int) -> np.ndarray:
    rad = int(3 * sigma)
    t = np.arange(-rad, rad + 1, dtype=np.float64)
    k = np.exp(-0.5 * (t / sigma) ** 2)
    k /= k.sum()
    a = np.moveaxis(a, axis, -1)
    pad = np.pad(a, [(0, 0)] * (a.ndim - 1) + [(rad, rad)], mode="reflect")
    out = np.zeros_like(a, dtype=np.float64)
    for i, kv in enumerate(k):
        out += kv * pad[..., i:i + a.shape[-1]]
    return np.moveaxis(out, -1, axis)


class SyntheticClip:
    """A video clip of moving textured rectangles over a smooth background.

    Frames are NHWC fp32 [1, H, W, 3]: a Gaussian-blurred N(0,1) background (fixed
    across frames) plus r ~ U{3..10} rectangles of 96..512 px textured with N(0,1),
    each moving at a constant velocity of 8..32 px/frame and reflecting at the
    borders. The execution grid of frame t marks every block touched by a rectangle
    at t or at t-1, following the detection information-gain rule that assigns gain
    to both the current and the previous position of an object (Section 3.4,
    Algorithm 1). Frame 0 uses the all-ones grid (the first frame of a clip is
    executed completely, Section 4, BlockCopy configuration).
    """

    def __init__(self, seed: int, h: int = 1024, w: int = 2048, block: int = 128,
                 size_range=(96, 320), speed_range=(8, 32), nrect_range=(3, 10),
                 blur_sigma: float = 16.0, bg_downsample: int = 8):
        r = rng(seed)
        self.h, self.w, self.block = h, w, block
        self.gh, self.gw = h // block, w // block
        # smooth background: blur at reduced resolution, then nearest upsample
        hs, ws = h // bg_downsample, w // bg_downsample
        bg = r.standard_normal((hs, ws, 3))
        sig = blur_sigma / bg_downsample
        bg = _blur_axis(_blur_axis(bg, sig, 0), sig, 1)
        bg /= bg.std()
        self.bg = np.repeat(np.repeat(bg, bg_downsample, 0), bg_downsample, 1).astype(np.float32)
        nrect = int(r.integers(nrect_range[0], nrect_range[1] + 1))
        self.rects = []
        for _ in range(nrect):
            rh = int(r.integers(size_range[0], size_range[1] + 1))
            rw = int(r.integers(size_range[0], size_range[1] + 1))
            y = float(r.integers(0, h - rh))
            x = float(r.integers(0, w - rw))
            sp = float(r.integers(speed_range[0], speed_range[1] + 1))
            ang = float(r.random() * 2 * np.pi)
            tex = r.standard_normal((rh, rw, 3)).astype(np.float32)
            self.rects.append(dict(h=rh, w=rw, y=y, x=x, vy=sp * np.sin(ang), vx=sp * np.cos(ang), tex=tex))

    def _positions(self, t: int):
        out = []
        for rc in self.rects:
            y, x, vy, vx = rc["y"], rc["x"], rc["vy"], rc["vx"]
            for _ in range(t):
                y += vy
                x += vx
                if y < 0 or y > self.h - rc["h"]:
                    vy = -vy
                    y = min(max(y, 0.0), float(self.h - rc["h"]))
                if x < 0 or x > self.w - rc["w"]:
                    vx = -vx
                    x = min(max(x, 0.0), float(self.w - rc["w"]))
            out.append((int(round(y)), int(round(x)), rc["h"], rc["w"]))
        return out

    def frame(self, t: int) -> np.ndarray:
        img = self.bg.copy()
        for rc, (y, x, rh, rw) in zip(self.rects, self._positions(t)):
            img[y:y + rh, x:x + rw] = rc["tex"]
        return img[None]

    def mask(self, t: int) -> np.ndarray:
        if t == 0:
            return np.ones((1, self.gh, self.gw), np.uint8)
        m = np.zeros((self.gh, self.gw), np.uint8)
        b = self.block
        for pos in (self._positions(t), self._positions(t - 1)):
            for (y, x, rh, rw) in pos:
                m[y // b:(y + rh - 1) // b + 1, x // b:(x + rw - 1) // b + 1] = 1
        return m[None]


# ---------------------------------------------------------------- policy-side inputs

def seg_logits(r: np.random.Generator, n: int, classes: int, h: int, w: int,
               scale: float = 4.0, cell: int = 16) -> np.ndarray:
    """Per-class segmentation scores with spatial structure, standing in for a
    segmentation network's output on a Cityscapes frame (19 classes at full 2048x1024
    resolution): a coarse random field (one value per cell x cell patch) repeated over
    its patch, plus fine N(0, 0.5) noise. float32 [n, classes, h, w]."""
    ch, cw = -(-h // cell), -(-w // cell)
    coarse = r.normal(0.0, scale, (n, classes, ch, cw)).astype(np.float32)
    f = np.repeat(np.repeat(coarse, cell, axis=2), cell, axis=3)[:, :, :h, :w]
    return (f + r.normal(0.0, 0.5, (n, classes, h, w)).astype(np.float32)).astype(np.float32)


def seg_logits_next(r: np.random.Generator, prev: np.ndarray, changed: float = 0.25,
                    cell: int = 64, scale: float = 4.0) -> np.ndarray:
    """The next frame's scores: a random fraction `changed` of the cell x cell patches
    get new scores (moving content), every other pixel keeps its scores plus small
    N(0, 0.05) noise. float32, same shape as prev."""
    n, c, h, w = prev.shape
    out = prev + r.normal(0.0, 0.05, prev.shape).astype(np.float32)
    ch, cw = -(-h // cell), -(-w // cell)
    pick = r.random((n, ch, cw)) < changed
    for img, cy, cx in zip(*np.nonzero(pick)):
        ys, xs = slice(cy * cell, min(h, cy * cell + cell)), slice(cx * cell, min(w, cx * cell + cell))
        out[img, :, ys, xs] = r.normal(0.0, scale, (c, 1, 1)) + r.normal(0.0, 0.5, out[img, :, ys, xs].shape)
    return out.astype(np.float32)


def block_probabilities(r: np.random.Generator, n: int, gh: int, gw: int) -> np.ndarray:
    """Policy outputs p_b in [0, 1] per block: a mix of confident (near 0 or 1) and
    uncertain blocks, as a trained policy produces. float32 [n, gh, gw]."""
    p = r.beta(0.4, 0.8, (n, gh, gw))
    return p.astype(np.float32)
