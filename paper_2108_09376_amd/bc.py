"""Python binding of libblockcopy (the C ABI declared in include/bc.h).

Argument marshalling only: every function here has the name of the C entry point it
calls, takes torch tensors (device memory) or numpy arrays (host memory), and
passes raw pointers, sizes and the current HIP stream. All computation happens in
the HIP kernels of the library. There is no fallback: if the library is missing
or fails to load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libblockcopy.so")

BC_OK, BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT = 0, 1, 2, 3, 4
BC_ERR_NOT_DIVISIBLE, BC_ERR_CAPACITY, BC_ERR_ALIAS, BC_ERR_UNINITIALIZED = 5, 6, 7, 8
BC_ERR_UNSUPPORTED, BC_ERR_HIP, BC_ERR_CAPTURE = 9, 10, 11
BC_F32, BC_BF16, BC_F16 = 0, 1, 2
BC_NCHW, BC_NHWC = 0, 1


class BCError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: status {status} ({status_name(status)}): {detail}")


class bc_tensor(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("c", ctypes.c_int32), ("h", ctypes.c_int32),
                ("w", ctypes.c_int32), ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32)]


class bc_grid(ctypes.Structure):
    _fields_ = [("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32)]


class bc_param(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("v", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("w16", ctypes.c_void_p), ("count", ctypes.c_int64)]


class bc_conv(ctypes.Structure):
    _fields_ = [("kh", ctypes.c_int32), ("kw", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("relu", ctypes.c_int32)]


class bc_spp_geom(ctypes.Structure):
    _fields_ = [("levels", ctypes.c_int32), ("cl", ctypes.c_int32), ("rows", ctypes.c_int32 * 8),
                ("cols", ctypes.c_int32 * 8)]


class bc_conv_call(ctypes.Structure):
    _fields_ = [("conv", bc_conv), ("d_in", ctypes.c_void_p), ("in_", bc_tensor),
                ("d_w", ctypes.c_void_p), ("d_bias", ctypes.c_void_p),
                ("d_residual", ctypes.c_void_p), ("d_out", ctypes.c_void_p), ("out", bc_tensor)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2108_09376_amd.build` "
                      "(there is no fallback path)")
_lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
_sigs = {
    "bc_abi_version": ([], _i32),
    "bc_status_str": ([_i32], ctypes.c_char_p),
    "bc_last_error": ([], ctypes.c_char_p),
    "bc_build_block_index": ([_vp, _i32, bc_grid, _vp, _i32, _vp, _vp, _vp], _i32),
    "bc_gather_halo": ([_vp, bc_tensor, bc_grid, ctypes.POINTER(bc_conv), _f32, _vp, _vp, _i32, _vp,
                        _vp], _i32),
    "bc_scatter_blocks": ([_vp, _vp, _vp, _i32, bc_grid, _vp, bc_tensor, _vp], _i32),
    "bc_sparse_conv2d": ([ctypes.POINTER(bc_conv), _vp, bc_tensor, _vp, _vp, _vp, _vp, bc_tensor,
                          bc_grid, _vp, _vp, _i32, _vp], _i32),
    "bc_sparse_conv2d_noalloc": ([ctypes.POINTER(bc_conv), _vp, bc_tensor, _vp, _vp, _vp, _vp,
                                  bc_tensor, bc_grid, _vp, _vp, _i32, _vp], _i32),
    "bc_sparse_conv2d_pair": ([ctypes.POINTER(bc_conv_call), ctypes.POINTER(bc_conv_call), bc_grid,
                               _vp, _vp, _i32, _vp], _i32),
    "bc_sparse_spp": ([_vp, bc_tensor, ctypes.POINTER(bc_spp_geom), _vp, _vp, _vp, _vp, bc_tensor, bc_grid,
                       _vp, _vp, _i32, _vp], _i32),
    "bc_sparse_maxpool2d": ([ctypes.POINTER(bc_conv), _vp, bc_tensor, _vp, bc_tensor, bc_grid, _vp,
                             _vp, _i32, _vp], _i32),
    "bc_fold_bn": ([_vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp], _i32),
    "bc_repack_weights": ([_vp, _i32, _i32, _i32, _i32, _i32, _vp], _i32),
    "bc_buffer_register": ([_vp, bc_tensor, ctypes.POINTER(_vp)], _i32),
    "bc_buffer_release": ([_vp], _i32),
    "bc_buffer_invalidate": ([_vp], _i32),
    "bc_buffer_mark_written": ([_vp, _i32], _i32),
    "bc_buffer_is_valid": ([_vp], _i32),
    "bc_sample_execution_grid": ([_vp, _i32, bc_grid, ctypes.c_uint64, ctypes.c_uint64, _vp, _vp, _i32,
                                  _vp, _vp, _vp], _i32),
    "bc_update_frame_state": ([_vp, _vp, bc_tensor, bc_grid, _vp, _vp, _i32, _vp], _i32),
    "bc_sparse_upsample_add": ([_vp, bc_tensor, _vp, _vp, bc_tensor, bc_grid, _i32, _vp, _vp, _i32,
                                _vp], _i32),
    "bc_seg_information_gain": ([_vp, _vp, bc_tensor, _i32, bc_grid, _vp, _vp, _vp], _i32),
    "bc_policy_input": ([_vp, _vp, bc_tensor, _vp, bc_tensor, _i32, _vp, bc_grid, _vp, bc_tensor, _vp], _i32),
    "bc_policy_probabilities": ([_vp, bc_tensor, _vp, _vp], _i32),
    "bc_policy_logit_grad": ([_vp, _vp, _vp, _vp, bc_tensor, _vp], _i32),
    "bc_grad_combine": ([_vp, _vp, _vp, bc_tensor, _vp, _vp], _i32),
    "bc_conv2d_input_grad": ([ctypes.POINTER(bc_conv), _vp, bc_tensor, _vp, _vp, _vp, bc_tensor, _vp], _i32),
    "bc_conv2d_weight_grad": ([ctypes.POINTER(bc_conv), _vp, bc_tensor, _vp, bc_tensor, _vp, _vp, _vp], _i32),
    "bc_rmsprop_step": ([_vp, _vp, _vp, ctypes.c_int64, _f32, _f32, _f32, _f32, _vp, _i32, _vp], _i32),
    "bc_rmsprop_step_many": ([ctypes.POINTER(bc_param), _i32, _f32, _f32, _f32, _f32, _i32, _vp], _i32),
    "bc_block_rewards": ([_vp, _vp, _vp, _i32, bc_grid, _f32, _f32, _f32, _vp, _vp, _vp, _vp, _vp], _i32),
}
for _name, (_args, _res) in _sigs.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res

EXPORTED = tuple(_sigs)

# The ABI these bindings marshal for (BC_ABI_VERSION of include/bc.h); a library built
# from other sources is refused rather than called with mismatched arguments.
ABI_VERSION = 10
if _lib.bc_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} has ABI {_lib.bc_abi_version()}, the bindings expect "
                      f"{ABI_VERSION}: rebuild with `python -m paper_2108_09376_amd.build`")


def status_name(s: int) -> str:
    return _lib.bc_status_str(int(s)).decode()


def _check(status: int, func: str):
    if status != BC_OK:
        raise BCError(status, func, _lib.bc_last_error().decode())


def bc_abi_version() -> int:
    return int(_lib.bc_abi_version())


def bc_last_error() -> str:
    return _lib.bc_last_error().decode()


# ------------------------------------------------------------------ marshalling helpers

_TORCH_DT = {}


def _dtype_code(t) -> int:
    import torch
    if not _TORCH_DT:
        _TORCH_DT.update({torch.float32: BC_F32, torch.bfloat16: BC_BF16, torch.float16: BC_F16})
    return _TORCH_DT[t.dtype]


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def desc(t, layout: int) -> bc_tensor:
    """bc_tensor of a contiguous 4-D tensor stored NHWC ([N,H,W,C]) or NCHW ([N,C,H,W])."""
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    if t.dim() != 4:
        raise ValueError("feature maps are 4-D")
    if layout == BC_NHWC:
        n, h, w, c = t.shape
    else:
        n, c, h, w = t.shape
    return bc_tensor(n, c, h, w, _dtype_code(t), layout)


def _grid(g) -> bc_grid:
    return g if isinstance(g, bc_grid) else bc_grid(int(g[0]), int(g[1]))


def _conv(c) -> bc_conv:
    return c if isinstance(c, bc_conv) else bc_conv(*[int(v) for v in c])


# ------------------------------------------------------------------ entry points

def bc_build_block_index(mask, n, grid, idx, count, h_count=None, stream=None):
    """mask uint8 [n, gh, gw] (device) -> idx int32 [capacity], count int32 [1] (device).
    With h_count=True the count is also returned to the host (synchronising)."""
    hc = ctypes.c_int32(0) if h_count else None
    st = _lib.bc_build_block_index(_ptr(mask), int(n), _grid(grid), _ptr(idx), int(idx.numel()),
                                   _ptr(count), ctypes.byref(hc) if hc is not None else None,
                                   _stream(stream))
    _check(st, "bc_build_block_index")
    return hc.value if hc is not None else None


def bc_gather_halo(src, layout, grid, geom, pad_value, idx, count, packed, stream=None):
    cap = 0 if idx is None else int(idx.numel())
    c = _conv(geom)
    st = _lib.bc_gather_halo(_ptr(src), desc(src, layout), _grid(grid), ctypes.byref(c),
                             float(pad_value), _ptr(idx), _ptr(count), cap, _ptr(packed),
                             _stream(stream))
    _check(st, "bc_gather_halo")


def bc_scatter_blocks(packed, idx, count, grid, dst, layout, stream=None):
    cap = 0 if idx is None else int(idx.numel())
    st = _lib.bc_scatter_blocks(_ptr(packed), _ptr(idx), _ptr(count), cap, _grid(grid), _ptr(dst),
                                desc(dst, layout), _stream(stream))
    _check(st, "bc_scatter_blocks")


def bc_sparse_conv2d(conv, x, layout, w, bias, residual, out, grid, idx, count, stream=None):
    cap = 0 if idx is None else int(idx.numel())
    c = _conv(conv)
    st = _lib.bc_sparse_conv2d(ctypes.byref(c), _ptr(x), desc(x, layout), _ptr(w), _ptr(bias),
                               _ptr(residual), _ptr(out), desc(out, layout), _grid(grid), _ptr(idx),
                               _ptr(count), cap, _stream(stream))
    _check(st, "bc_sparse_conv2d")


def bc_sparse_conv2d_noalloc(conv, x, layout, w, bias, residual, out, grid, idx, count, stream=None):
    cap = 0 if idx is None else int(idx.numel())
    c = _conv(conv)
    st = _lib.bc_sparse_conv2d_noalloc(ctypes.byref(c), _ptr(x), desc(x, layout), _ptr(w), _ptr(bias),
                                       _ptr(residual), _ptr(out), desc(out, layout), _grid(grid),
                                       _ptr(idx), _ptr(count), cap, _stream(stream))
    _check(st, "bc_sparse_conv2d_noalloc")


def _call(conv, x, layout, w, bias, residual, out) -> bc_conv_call:
    def addr(t):
        return None if t is None else t.data_ptr()
    return bc_conv_call(_conv(conv), addr(x), desc(x, layout), addr(w), addr(bias), addr(residual),
                        addr(out), desc(out, layout))


def bc_sparse_conv2d_pair(a, b, grid, idx, count, stream=None):
    """Two independent convolutions on one grid and index; a and b are each the tuple
    (conv, x, layout, w, bias, residual, out) of a bc_sparse_conv2d call."""
    cap = 0 if idx is None else int(idx.numel())
    ca, cb = _call(*a), _call(*b)
    st = _lib.bc_sparse_conv2d_pair(ctypes.byref(ca), ctypes.byref(cb), _grid(grid), _ptr(idx),
                                    _ptr(count), cap, _stream(stream))
    _check(st, "bc_sparse_conv2d_pair")


def bc_sparse_spp(x, layout, rows, cols, cl, w, bias, levels, out, grid, idx, count, stream=None):
    """rows, cols: the bin grid of each level (host sequences of equal length)."""
    cap = 0 if idx is None else int(idx.numel())
    g = bc_spp_geom()
    g.levels, g.cl = len(rows), int(cl)
    for i, (r, c) in enumerate(zip(rows, cols)):
        g.rows[i], g.cols[i] = int(r), int(c)
    st = _lib.bc_sparse_spp(_ptr(x), desc(x, layout), ctypes.byref(g), _ptr(w), _ptr(bias), _ptr(levels),
                            _ptr(out), desc(out, layout), _grid(grid), _ptr(idx), _ptr(count), cap,
                            _stream(stream))
    _check(st, "bc_sparse_spp")


def bc_sparse_maxpool2d(geom, x, layout, out, grid, idx, count, stream=None):
    cap = 0 if idx is None else int(idx.numel())
    c = _conv(geom)
    st = _lib.bc_sparse_maxpool2d(ctypes.byref(c), _ptr(x), desc(x, layout), _ptr(out),
                                  desc(out, layout), _grid(grid), _ptr(idx), _ptr(count), cap,
                                  _stream(stream))
    _check(st, "bc_sparse_maxpool2d")


def bc_sparse_upsample_add(coarse, layout, skip, out, grid, relu, idx, count, stream=None):
    """out[active blocks] = relu?(up2(coarse) + skip); out is [n, c, 2h, 2w] of coarse
    (NHWC or NCHW order per layout), skip shaped like out or None."""
    cap = 0 if idx is None else int(idx.numel())
    if skip is not None and (skip.shape != out.shape or skip.dtype != out.dtype):
        raise ValueError("skip must be shaped and typed like out")
    if skip is not None and not skip.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    st = _lib.bc_sparse_upsample_add(_ptr(coarse), desc(coarse, layout), _ptr(skip), _ptr(out),
                                     desc(out, layout), _grid(grid), int(relu), _ptr(idx),
                                     _ptr(count), cap, _stream(stream))
    _check(st, "bc_sparse_upsample_add")


def bc_sample_execution_grid(prob, grid, seed, frame, mask, idx, count, h_count=None, stream=None):
    """prob float32 [n, gh, gw] (device) -> mask uint8 [n, gh, gw], idx int32 [capacity],
    count int32 [1] (device). With h_count=True the count is also returned (synchronising)."""
    hc = ctypes.c_int32(0) if h_count else None
    st = _lib.bc_sample_execution_grid(_ptr(prob), int(prob.shape[0]), _grid(grid),
                                       ctypes.c_uint64(int(seed)), ctypes.c_uint64(int(frame)),
                                       _ptr(mask), _ptr(idx), int(idx.numel()), _ptr(count),
                                       ctypes.byref(hc) if hc is not None else None, _stream(stream))
    _check(st, "bc_sample_execution_grid")
    return hc.value if hc is not None else None


def bc_update_frame_state(frame, state, layout, grid, idx, count, stream=None):
    """state[active blocks] = frame[active blocks]; frame/state same shape and dtype."""
    if frame.shape != state.shape or frame.dtype != state.dtype:
        raise ValueError("frame and state must have the same shape and dtype")
    cap = 0 if idx is None else int(idx.numel())
    st = _lib.bc_update_frame_state(_ptr(frame), _ptr(state), desc(state, layout), _grid(grid),
                                    _ptr(idx), _ptr(count), cap, _stream(stream))
    _check(st, "bc_update_frame_state")


def bc_seg_information_gain(logits, prev_logits, grid, ig, classes=None, layout=BC_NCHW,
                            mask=None, stream=None):
    """Score maps of frames t and t-1 (float32 [n, c, h, w], or bf16/f16 [n, h, w, c] with
    layout=BC_NHWC) -> ig float32 [n, gh, gw]; the first `classes` channels (default all)
    are the class scores. With the execution grid `mask` (uint8 [n, gh, gw]) blocks that
    did not run get 0 without their scores being read."""
    if logits.shape != prev_logits.shape or logits.dtype != prev_logits.dtype:
        raise ValueError("score maps must have the same shape and dtype")
    d = desc(logits, layout)
    st = _lib.bc_seg_information_gain(_ptr(logits), _ptr(prev_logits), d,
                                      int(d.c if classes is None else classes), _grid(grid),
                                      _ptr(mask), _ptr(ig), _stream(stream))
    _check(st, "bc_seg_information_gain")


def bc_policy_input(frame, state, scores, classes, prev_mask, grid, out, stream=None):
    """S_t [n, h/4, w/4, 32] (NHWC) from the frame and frame state [n, h, w, 3], the
    previous scores [n, h/4, w/4, c] and the previous grid (uint8 [n, gh, gw] or None)."""
    st = _lib.bc_policy_input(_ptr(frame), _ptr(state), desc(frame, BC_NHWC), _ptr(scores),
                              desc(scores, BC_NHWC), int(classes), _ptr(prev_mask), _grid(grid),
                              _ptr(out), desc(out, BC_NHWC), _stream(stream))
    _check(st, "bc_policy_input")


def bc_policy_probabilities(logits, prob, stream=None):
    """prob float32 [n, gh, gw] = sigmoid(logits[..., 0]), logits [n, gh, gw, c] NHWC."""
    st = _lib.bc_policy_probabilities(_ptr(logits), desc(logits, BC_NHWC), _ptr(prob), _stream(stream))
    _check(st, "bc_policy_probabilities")


def bc_policy_logit_grad(reward, mask, prob, grad, stream=None):
    """grad [n, gh, gw, c] NHWC: channel 0 = -R (a - p), the rest 0."""
    st = _lib.bc_policy_logit_grad(_ptr(reward), _ptr(mask), _ptr(prob), _ptr(grad),
                                   desc(grad, BC_NHWC), _stream(stream))
    _check(st, "bc_policy_logit_grad")


def bc_grad_combine(a, b, y, out, stream=None):
    """out = (a + b) * [y > 0] (b, y may be None); NHWC 16-bit, all alike."""
    st = _lib.bc_grad_combine(_ptr(a), _ptr(b), _ptr(y), desc(a, BC_NHWC), _ptr(out), _stream(stream))
    _check(st, "bc_grad_combine")


def bc_conv2d_input_grad(geom, grad_out, w, accum, grad_in, stream=None):
    """grad_in = transposed conv of grad_out with w (+ accum), NHWC."""
    c = _conv(geom)
    st = _lib.bc_conv2d_input_grad(ctypes.byref(c), _ptr(grad_out), desc(grad_out, BC_NHWC), _ptr(w),
                                   _ptr(accum), _ptr(grad_in), desc(grad_in, BC_NHWC), _stream(stream))
    _check(st, "bc_conv2d_input_grad")


def bc_conv2d_weight_grad(geom, x, grad_out, dw, db=None, stream=None):
    """dw float32 [cout, k, k, cin] += weight gradient; db float32 [cout] += bias gradient."""
    c = _conv(geom)
    st = _lib.bc_conv2d_weight_grad(ctypes.byref(c), _ptr(x), desc(x, BC_NHWC), _ptr(grad_out),
                                    desc(grad_out, BC_NHWC), _ptr(dw), _ptr(db), _stream(stream))
    _check(st, "bc_conv2d_weight_grad")


def bc_rmsprop_step(w, v, grad, lr, alpha, eps, weight_decay, w16=None, stream=None):
    """One RMSprop step on float32 tensors w, v, grad (grad reset to 0), and the 16-bit
    copy w16 (same element count) if given."""
    dt = _dtype_code(w16) if w16 is not None else BC_BF16
    st = _lib.bc_rmsprop_step(_ptr(w), _ptr(v), _ptr(grad), ctypes.c_int64(int(w.numel())), float(lr),
                              float(alpha), float(eps), float(weight_decay), _ptr(w16), dt, _stream(stream))
    _check(st, "bc_rmsprop_step")


def bc_rmsprop_step_many(params, lr, alpha, eps, weight_decay, stream=None):
    """bc_rmsprop_step on every (w, v, grad, w16 or None) of `params` in one launch; the
    16-bit copies share one dtype."""
    arr = (bc_param * len(params))()
    dt = BC_BF16
    for i, (w, v, grad, w16) in enumerate(params):
        arr[i] = bc_param(_ptr(w), _ptr(v), _ptr(grad), _ptr(w16), int(w.numel()))
        if w16 is not None:
            dt = _dtype_code(w16)
    st = _lib.bc_rmsprop_step_many(arr, len(params), float(lr), float(alpha), float(eps),
                                   float(weight_decay), dt, _stream(stream))
    _check(st, "bc_rmsprop_step_many")


def bc_block_rewards(ig, mask, prob, grid, tau, gamma, mu, mavg, reward, cost=None, loss=None,
                     stream=None):
    """Rewards per block (reward [n, gh, gw]), C_t (cost [n]), M_t (mavg [n], in/out) and
    the REINFORCE loss (loss [n], needs prob). All float32 device tensors, mask uint8."""
    st = _lib.bc_block_rewards(_ptr(ig), _ptr(mask), _ptr(prob), int(ig.shape[0]), _grid(grid),
                               float(tau), float(gamma), float(mu), _ptr(mavg), _ptr(reward),
                               _ptr(cost), _ptr(loss), _stream(stream))
    _check(st, "bc_block_rewards")


def _np_ptr(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def bc_fold_bn(w, conv_bias, gamma, beta, mean, var, eps=1e-5):
    """Host: fold inference batch norm into fp32 weights [cout, ...]; returns (w', b')."""
    w = np.ascontiguousarray(w, np.float32)
    cout = w.shape[0]
    f = lambda a: None if a is None else np.ascontiguousarray(a, np.float32)
    cb, g, b, m, v = f(conv_bias), f(gamma), f(beta), f(mean), f(var)
    w_out = np.empty_like(w)
    b_out = np.empty(cout, np.float32)
    st = _lib.bc_fold_bn(_np_ptr(w), cout, int(w.size // cout), _np_ptr(cb), _np_ptr(g), _np_ptr(b),
                         _np_ptr(m), _np_ptr(v), float(eps), _np_ptr(w_out), _np_ptr(b_out))
    _check(st, "bc_fold_bn")
    return w_out, b_out


def bc_repack_weights(w_oihw, dtype_code):
    """Host: fp32 OIHW -> [cout][kh][kw][cin] in the given dtype (numpy, raw bits for 16-bit)."""
    w = np.ascontiguousarray(w_oihw, np.float32)
    co, ci, kh, kw = w.shape
    out = np.empty((co, kh, kw, ci), np.float32 if dtype_code == BC_F32 else np.uint16)
    st = _lib.bc_repack_weights(_np_ptr(w), co, ci, kh, kw, int(dtype_code), _np_ptr(out))
    _check(st, "bc_repack_weights")
    return out


class Buffer:
    """A registered persistent buffer (wraps caller memory; see bc_buffer_* in bc.h)."""

    def __init__(self, t, layout):
        self.t = t
        self.layout = layout
        h = ctypes.c_void_p()
        _check(_lib.bc_buffer_register(_ptr(t), desc(t, layout), ctypes.byref(h)), "bc_buffer_register")
        self.handle = h

    def release(self):
        if self.handle is not None:
            _check(_lib.bc_buffer_release(self.handle), "bc_buffer_release")
            self.handle = None

    def invalidate(self):
        _check(_lib.bc_buffer_invalidate(self.handle), "bc_buffer_invalidate")

    def mark_written(self, full_mask: bool):
        _check(_lib.bc_buffer_mark_written(self.handle, int(bool(full_mask))), "bc_buffer_mark_written")

    @property
    def valid(self) -> int:
        return int(_lib.bc_buffer_is_valid(self.handle))

    def __del__(self):
        try:
            self.release()
        except Exception:
            pass


def bc_buffer_register(t, layout) -> Buffer:
    return Buffer(t, layout)


def raw():
    """The ctypes library object (for tests that call entry points with raw pointers)."""
    return _lib
