"""Helpers for GPU tests: moving seeded inputs (bit patterns) between numpy NCHW and
device tensors, and the tolerance metric. No method arithmetic lives here."""
import numpy as np
import torch

TORCH = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}
TOL = {"f32": 1e-4, "bf16": 2e-2, "f16": 2e-2}


def to_dev(bits, dtype, nhwc=True, device="cuda"):
    """NCHW bit patterns -> device tensor (NHWC if nhwc)."""
    b = np.ascontiguousarray(bits)
    if dtype == "f32":
        t = torch.from_numpy(b.view(np.float32).copy())
    else:
        t = torch.from_numpy(b.view(np.int16).copy()).view(TORCH[dtype])
    if nhwc:
        t = t.permute(0, 2, 3, 1)
    return t.contiguous().to(device)


def from_dev(t, nhwc=True):
    """Device tensor -> NCHW bit patterns (uint16 / uint32)."""
    t = t.detach().cpu()
    if nhwc:
        t = t.permute(0, 3, 1, 2)
    t = t.contiguous()
    if t.dtype == torch.float32:
        return t.numpy().view(np.uint32).copy()
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def weights_dev(w_bits_oihw, dtype, nhwc=True, device="cuda"):
    """OIHW bit patterns -> device weights ([Cout][kh][kw][Cin] if nhwc else OIHW)."""
    b = np.ascontiguousarray(w_bits_oihw)
    if nhwc:
        b = np.ascontiguousarray(b.transpose(0, 2, 3, 1))
    if dtype == "f32":
        t = torch.from_numpy(b.view(np.float32).copy())
    else:
        t = torch.from_numpy(b.view(np.int16).copy()).view(TORCH[dtype])
    return t.to(device)


def max_abs_rel(got, want):
    """max |y - y_ref| / max(1, |y_ref|) (the stated tolerance metric)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if got.size == 0:
        return 0.0
    return float(np.max(np.abs(got - want) / np.maximum(1.0, np.abs(want))))


def block_select(mask, shape_nchw):
    n, c, h, w = shape_nchw
    gh, gw = mask.shape[1:]
    m = np.repeat(np.repeat(np.asarray(mask) != 0, h // gh, 1), w // gw, 2)[:, None]
    return np.broadcast_to(m, shape_nchw)
