"""CPU oracle for BlockCopy's block-sparse convolution with temporal feature copying.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package. The product path (the HIP
library and its Python binding) never imports, links or runs it, and the oracle
shares no code with it: no kernels, helpers, tables or pre/post-processing.

What the method computes (Section 3.1 and the caption of Fig. 3): for every
convolution layer and every frame, the blocks selected by the execution grid A_t
(Section 3.5, a_b = 1) are computed, and every other block keeps the layer's
representation from the previous execution (a_b = 0 means "feature transfer").
Blocks are processed with padding taken from their neighbours so that there are no
discontinuities between blocks (the BlockPadding module the paper builds on,
Section 3.1). Evaluated exactly, that is:

    Y_t = select(A_t, conv(X_t), Y_{t-1})

where conv is the ordinary dense layer on the layer's current input buffer X_t
(fresh where the neighbour block was executed this frame, transferred otherwise),
and select keeps Y_{t-1} bit for bit outside the selected blocks. The oracle takes
exactly these steps: a dense convolution everywhere (C, fp64, ``bc_oracle.c``),
rounding to the storage format, then the masked select. Points the paper leaves
open are read as follows:

* the mask indexes *output* blocks; block (gy, gx) of a layer with output block
  edge bh x bw covers output rows gy*bh .. gy*bh+bh-1 (same for columns);
* the halo of a block comes from the layer's current input buffer, zeros outside
  the image (the dense layer's own zero padding; -inf for max pooling);
* rounding: fp64 -> fp32 round-to-nearest-even, then fp32 -> bf16/fp16 RNE;
* active-block index: ascending raster order of nonzero mask entries,
  id = (img * Gh + gy) * Gw + gx;
* BN folding uses eps = 1e-5.

Arrays: feature maps are numpy arrays in NCHW. Stored values are carried as raw
bit patterns (uint32 for f32, uint16 for bf16/f16) so that copied blocks can be
checked byte for byte.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def build() -> str:
    """Compile the C part of the oracle (gcc -O2 -fopenmp). Returns the .so path."""
    subprocess.check_call(["sh", os.path.join(_HERE, "build.sh")])
    return os.path.join(_HERE, "libbc_oracle.so")


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libbc_oracle.so")
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(
                os.path.join(_HERE, "bc_oracle.c")):
            build()
        lib = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        i = ctypes.c_int
        lib.oracle_conv2d_dense.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, dp, dp, i, dp, i, i]
        lib.oracle_conv2d_dense.restype = None
        lib.oracle_conv2d_points.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, dp, dp, i, i, i,
                                             ip, ctypes.c_int64, dp]
        lib.oracle_conv2d_points.restype = None
        lib.oracle_conv2d_blocks.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, dp, dp, i, dp, i, i,
                                             ip, i, i, i]
        lib.oracle_conv2d_blocks.restype = None
        lib.oracle_maxpool2d_dense.argtypes = [dp, i, i, i, i, i, i, i, dp, i, i]
        lib.oracle_maxpool2d_dense.restype = None
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = i
        _LIB = lib
    return _LIB


def num_threads() -> int:
    return int(_lib().oracle_num_threads())


def _dp(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def out_size(h: int, k: int, stride: int, pad: int) -> int:
    """PyTorch convolution output size."""
    return (h + 2 * pad - k) // stride + 1


# ------------------------------------------------------------------ dense layer

def conv2d_dense(x, w, bias=None, residual=None, stride=1, pad=0, relu=False):
    """Dense layer in fp64. x [N,Cin,H,W], w [Cout,Cin,kh,kw], bias [Cout],
    residual [N,Cout,Ho,Wo]. Returns z = conv + bias (+ residual), ReLU'd, in fp64."""
    x = np.ascontiguousarray(x, np.float64)
    w = np.ascontiguousarray(w, np.float64)
    n, cin, h, wd = x.shape
    cout, cin2, kh, kw = w.shape
    assert cin == cin2
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    b = None if bias is None else np.ascontiguousarray(bias, np.float64)
    r = None if residual is None else np.ascontiguousarray(residual, np.float64)
    if r is not None:
        assert r.shape == (n, cout, ho, wo)
    out = np.empty((n, cout, ho, wo), np.float64)
    _lib().oracle_conv2d_dense(_dp(x), n, cin, h, wd, _dp(w), cout, kh, kw, stride, pad,
                               _dp(b), _dp(r), int(bool(relu)), _dp(out), ho, wo)
    return out


def conv2d_points(x, w, pts, bias=None, residual=None, stride=1, pad=0, relu=False):
    """The dense layer's value at output points pts [K,4] = (n, co, y, x), fp64."""
    x = np.ascontiguousarray(x, np.float64)
    w = np.ascontiguousarray(w, np.float64)
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    pts = np.ascontiguousarray(pts, np.int32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float64)
    r = None if residual is None else np.ascontiguousarray(residual, np.float64)
    out = np.empty(len(pts), np.float64)
    _lib().oracle_conv2d_points(_dp(x), n, cin, h, wd, _dp(w), cout, kh, kw, stride, pad,
                                _dp(b), _dp(r), int(bool(relu)), ho, wo,
                                pts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                len(pts), _dp(out))
    return out


def maxpool2d_dense(x, k=3, stride=2, pad=1):
    """Dense max pooling with -inf padding, fp64."""
    x = np.ascontiguousarray(x, np.float64)
    n, c, h, wd = x.shape
    ho, wo = out_size(h, k, stride, pad), out_size(wd, k, stride, pad)
    out = np.empty((n, c, ho, wo), np.float64)
    _lib().oracle_maxpool2d_dense(_dp(x), n, c, h, wd, k, stride, pad, _dp(out), ho, wo)
    return out


# ------------------------------------------------------------------ rounding

def round_to_f32(z):
    """fp64 -> fp32, round to nearest even (IEEE conversion)."""
    return np.asarray(z, np.float64).astype(np.float32)


def f32_to_bf16_bits(z32):
    """fp32 -> bf16 bit pattern, round to nearest even; NaN stays a (quiet) NaN."""
    u = np.ascontiguousarray(z32, np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def f32_to_f16_bits(z32):
    """fp32 -> fp16 bit pattern (IEEE conversion, round to nearest even)."""
    return np.ascontiguousarray(z32, np.float32).astype(np.float16).view(np.uint16)


def store(z, dtype):
    """Round fp64 results to the storage format; returns the bit patterns."""
    z32 = round_to_f32(z)
    if dtype == "f32":
        return z32.view(np.uint32).copy()
    if dtype == "bf16":
        return f32_to_bf16_bits(z32)
    if dtype == "f16":
        return f32_to_f16_bits(z32)
    raise ValueError(dtype)


def value(bits, dtype):
    """Exact fp64 value of stored bit patterns."""
    bits = np.ascontiguousarray(bits)
    if dtype == "f32":
        return bits.view(np.float32).astype(np.float64)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    raise ValueError(dtype)


# ------------------------------------------------------------------ blocks

def block_index(mask):
    """Active-block list: ascending flat ids of the nonzero entries of the execution
    grid (Section 3.5, a_b = 1 executes block b), and their number."""
    idx = np.flatnonzero(np.asarray(mask).reshape(-1) != 0).astype(np.int32)
    return idx, int(idx.size)


def expand_mask(mask, bh, bw):
    """Per-pixel selection [N,1,Gh*bh,Gw*bw] from the block grid [N,Gh,Gw]."""
    m = np.asarray(mask) != 0
    return np.repeat(np.repeat(m, bh, axis=1), bw, axis=2)[:, None]


def select(mask, fresh_bits, prev_bits, bh, bw):
    """Executed blocks take the fresh values; every other element keeps the previous
    execution's bits unchanged (feature transfer, Section 3.1)."""
    assert fresh_bits.shape == prev_bits.shape and fresh_bits.dtype == prev_bits.dtype
    n, c, h, w = fresh_bits.shape
    gh, gw = np.asarray(mask).shape[1:]
    assert h == gh * bh and w == gw * bw
    sel = np.broadcast_to(expand_mask(mask, bh, bw), fresh_bits.shape)
    return np.where(sel, fresh_bits, prev_bits)


def sparse_conv2d(x_bits, w_bits, mask, prev_bits, dtype, stride=1, pad=0, bias=None,
                  residual_bits=None, relu=False):
    """One block-sparse layer: dense conv on the current input, rounded to ``dtype``,
    selected into the previous output by the mask. All tensors NCHW bit patterns;
    bias fp32 values. The block edge is the output size over the grid size."""
    x = value(x_bits, dtype)
    w = value(w_bits, dtype)
    res = None if residual_bits is None else value(residual_bits, dtype)
    b = None if bias is None else np.asarray(bias, np.float32).astype(np.float64)
    z = conv2d_dense(x, w, b, res, stride, pad, relu)
    fresh = store(z, dtype)
    gh, gw = np.asarray(mask).shape[1:]
    return select(mask, fresh, prev_bits, z.shape[2] // gh, z.shape[3] // gw)


def sparse_conv2d_active(x_bits, w_bits, mask, prev_bits, dtype, stride=1, pad=0, bias=None,
                         residual_bits=None, relu=False):
    """sparse_conv2d evaluated only where it is kept: the same per-point definition (C,
    fp64, order ci -> i -> j) at the output points of the executed blocks, nothing
    elsewhere, then the same rounding and select. Bit-identical to sparse_conv2d; the
    fair CPU comparison for a block-sparse execution (it skips what the select would
    discard)."""
    x = np.ascontiguousarray(value(x_bits, dtype), np.float64)
    w = np.ascontiguousarray(value(w_bits, dtype), np.float64)
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    res = None if residual_bits is None else np.ascontiguousarray(value(residual_bits, dtype))
    b = None if bias is None else np.ascontiguousarray(np.asarray(bias, np.float32).astype(np.float64))
    gh, gw = np.asarray(mask).shape[1:]
    blocks, nb = block_index(mask)
    z = np.zeros((n, cout, ho, wo), np.float64)
    if nb:
        _lib().oracle_conv2d_blocks(_dp(x), n, cin, h, wd, _dp(w), cout, kh, kw, stride, pad, _dp(b),
                                    _dp(res), int(bool(relu)), _dp(z), ho, wo,
                                    blocks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), nb, gh, gw)
    return select(mask, store(z, dtype), prev_bits, ho // gh, wo // gw)


def sparse_maxpool2d(x_bits, mask, prev_bits, dtype, k=3, stride=2, pad=1):
    """Block-sparse max pooling (-inf padding), same selection rule as the conv."""
    z = maxpool2d_dense(value(x_bits, dtype), k, stride, pad)
    fresh = store(z, dtype)
    gh, gw = np.asarray(mask).shape[1:]
    return select(mask, fresh, prev_bits, z.shape[2] // gh, z.shape[3] // gw)


def upsample2x_bilinear(x):
    """Bilinear upsampling by two of [n, c, h, w] values (float64), the sampling used by
    SwiftNet-style decoders (pixel centres aligned, borders replicated): output row Y
    samples input row (Y + 1/2) / 2 - 1/2, clamped to [0, h - 1], interpolated linearly
    between its two neighbours; the same for columns. For a factor of two this gives
    out[2i] = 3/4 in[i] + 1/4 in[i-1] and out[2i+1] = 3/4 in[i] + 1/4 in[i+1], with an
    index outside the image replaced by the nearest edge row or column."""
    x = np.asarray(x, np.float64)

    def axis_up(a, axis):
        n = a.shape[axis]
        src = (np.arange(2 * n) + 0.5) / 2.0 - 0.5
        src = np.clip(src, 0.0, n - 1)
        lo = np.floor(src).astype(np.int64)
        hi = np.minimum(lo + 1, n - 1)
        f = src - lo
        shape = [1] * a.ndim
        shape[axis] = 2 * n
        f = f.reshape(shape)
        return np.take(a, lo, axis=axis) * (1.0 - f) + np.take(a, hi, axis=axis) * f

    return axis_up(axis_up(x, 2), 3)


def sparse_upsample_add(coarse_bits, skip_bits, mask, prev_bits, dtype, relu=False):
    """One block-sparse decoder merge: up2(coarse) (+ skip) (ReLU), rounded to dtype,
    selected into the previous output by the mask (the grid indexes output blocks)."""
    z = upsample2x_bilinear(value(coarse_bits, dtype))
    if skip_bits is not None:
        z = z + value(skip_bits, dtype)
    if relu:
        z = np.maximum(z, 0.0)
    fresh = store(z, dtype)
    gh, gw = np.asarray(mask).shape[1:]
    return select(mask, fresh, prev_bits, z.shape[2] // gh, z.shape[3] // gw)


# ------------------------------------------------------------------ pyramid pooling
#
# The segmentation network's context module on the encoder's stride-32 output (the
# spatial pyramid pooling of SwiftNet-style models; the paper makes every layer of such
# single-stage networks block-sparse, Section 4). Each pyramid level averages the whole
# map over a grid of bins, so a level depends on every block of its input: under the
# method's dense-then-select definition the levels are computed densely from the
# layer's current input buffer each frame (fresh where blocks ran, transferred
# elsewhere), and only the concatenated output is selected into the previous output.

def spp_bins(h, w, g):
    """Bin grid of a pyramid level with g rows on an h x w map: g rows (at most h) and
    g * w / h columns rounded to the nearest integer (at least 1, at most w), so bins
    stay about square on maps wider than tall."""
    rows = min(g, h)
    cols = min(w, max(1, int(np.floor(g * w / h + 0.5))))
    return rows, cols


def adaptive_avg_pool2d(x, oh, ow):
    """Mean of each of oh x ow bins of [n, c, h, w] values (float64): bin (i, j) covers
    rows floor(i h / oh) .. ceil((i + 1) h / oh) - 1 and the same for columns."""
    x = np.asarray(x, np.float64)
    n, c, h, w = x.shape
    out = np.empty((n, c, oh, ow), np.float64)
    for i in range(oh):
        r0, r1 = (i * h) // oh, -((-(i + 1) * h) // oh)
        for j in range(ow):
            c0, c1 = (j * w) // ow, -((-(j + 1) * w) // ow)
            out[:, :, i, j] = x[:, :, r0:r1, c0:c1].mean(axis=(2, 3))
    return out


def upsample_bilinear(x, oh, ow):
    """Bilinear resampling of [n, c, h, w] values (float64) to oh x ow with pixel centres
    aligned: output row Y samples input row s = (Y + 1/2) h / oh - 1/2, taken as 0 when
    negative; with i0 = floor(s), i1 = min(i0 + 1, h - 1) and f = s - i0 it is
    (1 - f) x[i0] + f x[i1]. The same along columns."""
    x = np.asarray(x, np.float64)

    def axis_resample(a, axis, n_out):
        n_in = a.shape[axis]
        src = np.maximum((np.arange(n_out) + 0.5) * (n_in / n_out) - 0.5, 0.0)
        i0 = np.floor(src).astype(np.int64)
        i0 = np.minimum(i0, n_in - 1)
        i1 = np.minimum(i0 + 1, n_in - 1)
        f = src - i0
        shape = [1] * a.ndim
        shape[axis] = n_out
        f = f.reshape(shape)
        return np.take(a, i0, axis=axis) * (1.0 - f) + np.take(a, i1, axis=axis) * f

    return axis_resample(axis_resample(x, 2, oh), 3, ow)


def spp_levels(b_bits, grid_rows, w_bits, bias, dtype):
    """The pyramid levels of the bottleneck map b ([n, c, h, w] bit patterns), every
    pixel: per level l with grid_rows[l] rows, the bins' means (spp_bins), a 1x1
    convolution with weights w_bits[l] ([cl, c] bit patterns) plus bias[l] (fp32
    values), ReLU, rounded to dtype. Returns a list of [n, cl, rows, cols] bit patterns."""
    b = value(b_bits, dtype)
    n, c, h, w = b.shape
    out = []
    for g, wl, bl in zip(grid_rows, w_bits, bias):
        rows, cols = spp_bins(h, w, g)
        pooled = adaptive_avg_pool2d(b, rows, cols)
        wv = value(wl, dtype).reshape(wl.shape[0], c)
        z = np.einsum("oc,nchw->nohw", wv, pooled) + np.asarray(bl, np.float32).astype(np.float64)[None, :, None, None]
        out.append(store(np.maximum(z, 0.0), dtype))
    return out


def sparse_spp(b_bits, level_bits, mask, prev_bits, dtype):
    """The pyramid pooling's concatenated output, block-sparse: channels 0..c-1 are the
    bottleneck map itself (its stored bits), then each level upsampled bilinearly to the
    map's size (upsample_bilinear) and rounded to dtype; executed blocks take these
    values, every other element keeps prev_bits."""
    n, c, h, w = b_bits.shape
    parts = [b_bits]
    for lb in level_bits:
        parts.append(store(upsample_bilinear(value(lb, dtype), h, w), dtype))
    fresh = np.concatenate(parts, axis=1)
    gh, gw = np.asarray(mask).shape[1:]
    return select(mask, fresh, prev_bits, h // gh, w // gw)


def gather_halo(x_bits, idx, gh, gw, bh, bw, kh, kw, stride, pad, pad_bits):
    """Halo tiles of the listed output blocks, packed [K, th, tw, C] (channels last):
    packed[k, i, j, c] = X[n, c, gy*bh*s - pad + i, gx*bw*s - pad + j], with
    ``pad_bits`` outside the image. th = (bh-1)*s + kh, tw = (bw-1)*s + kw."""
    n, c, h, w = x_bits.shape
    th, tw = (bh - 1) * stride + kh, (bw - 1) * stride + kw
    out = np.empty((len(idx), th, tw, c), x_bits.dtype)
    for k, bid in enumerate(np.asarray(idx)):
        img, rem = divmod(int(bid), gh * gw)
        gy, gx = divmod(rem, gw)
        y0, x0 = gy * bh * stride - pad, gx * bw * stride - pad
        for i in range(th):
            for j in range(tw):
                y, xx = y0 + i, x0 + j
                if 0 <= y < h and 0 <= xx < w:
                    out[k, i, j, :] = x_bits[img, :, y, xx]
                else:
                    out[k, i, j, :] = pad_bits
    return out


def scatter_blocks(packed, idx, gh, gw, dst_bits):
    """Write packed [K, bh, bw, C] blocks to their positions of dst (NCHW); every
    other element of dst is returned unchanged."""
    out = dst_bits.copy()
    _, bh, bw, _ = packed.shape
    for k, bid in enumerate(np.asarray(idx)):
        img, rem = divmod(int(bid), gh * gw)
        gy, gx = divmod(rem, gw)
        out[img, :, gy * bh:(gy + 1) * bh, gx * bw:(gx + 1) * bw] = packed[k].transpose(2, 0, 1)
    return out


# ------------------------------------------------------------------ batch norm

def fold_bn(w, conv_bias, gamma, beta, mean, var, eps=1e-5):
    """Fold inference-mode batch normalisation into the preceding conv, in fp64:
    w' = w * g / sqrt(var + eps), b' = beta + (b - mean) * g / sqrt(var + eps)."""
    w = np.asarray(w, np.float64)
    scale = np.asarray(gamma, np.float64) / np.sqrt(np.asarray(var, np.float64) + eps)
    b = np.zeros(w.shape[0]) if conv_bias is None else np.asarray(conv_bias, np.float64)
    w2 = w * scale.reshape((-1,) + (1,) * (w.ndim - 1))
    b2 = np.asarray(beta, np.float64) + (b - np.asarray(mean, np.float64)) * scale
    return w2, b2


from . import network  # noqa: E402,F401
