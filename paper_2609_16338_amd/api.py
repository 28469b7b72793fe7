"""Python binding of libbitcos: the C ABI's functions under the same names.

Argument marshalling only -- every step of the GEMV runs in the HIP kernels of
libbitcos.so; packing runs in its C++ host code.  Host arrays are numpy;
device buffers are torch tensors (torch supplies device memory and streams).
Sizes of device buffers are checked here, before the call, because the C ABI
takes plain pointers.
"""

from __future__ import annotations

import ctypes

import numpy as np

from . import _native as N
from ._native import (FMT_BIT2, FMT_BITCOS, FMT_TRIT5, LaunchInfo, Layout, X_BF16, X_I8,  # noqa: F401
                      Y_F32, Y_F32_ADD, Y_I32_RAW, Y_I32_RAW_ADD)


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


def _w(w) -> np.ndarray:
    w = np.ascontiguousarray(w)
    if w.dtype != np.int8 or w.ndim != 2:
        raise ValueError("W must be a 2-D int8 array")
    return w


def _scales(s) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(s).view(np.uint16) if np.asarray(s).dtype == np.float16
                                else np.asarray(s, dtype=np.uint16)).reshape(-1)


def num_scales(L: Layout) -> int:
    return L.n * (L.k // 128) if L.group == 128 else 1


# ---------------------------------------------------------------------------
# plan / pack / unpack (host)
# ---------------------------------------------------------------------------

def bitcos_plan(w, group: int = 128, unit_rows: int = 0) -> Layout:
    w = _w(w)
    L = Layout()
    N.check(N.lib().bitcos_plan(_ptr(w), w.shape[0], w.shape[1], group, unit_rows, ctypes.byref(L)),
            "bitcos_plan")
    return L


def trit5_plan(w, group: int = 128) -> Layout:
    w = _w(w)
    L = Layout()
    N.check(N.lib().trit5_plan(_ptr(w), w.shape[0], w.shape[1], group, ctypes.byref(L)), "trit5_plan")
    return L


def bit2_plan(w, group: int = 128) -> Layout:
    w = _w(w)
    L = Layout()
    N.check(N.lib().bit2_plan(_ptr(w), w.shape[0], w.shape[1], group, ctypes.byref(L)), "bit2_plan")
    return L


def _pack(fn: str, w, scales, L: Layout) -> np.ndarray:
    w = _w(w)
    s = _scales(scales)
    if w.shape != (L.n, L.k) or s.size != num_scales(L):
        raise ValueError("W or scales do not match the layout")
    out = np.empty(L.total_bytes, dtype=np.uint8)
    N.check(getattr(N.lib(), fn)(_ptr(w), _ptr(s), ctypes.byref(L), _ptr(out), out.nbytes), fn)
    return out


def bitcos_pack(w, scales, L: Layout) -> np.ndarray:
    return _pack("bitcos_pack", w, scales, L)


def trit5_pack(w, scales, L: Layout) -> np.ndarray:
    return _pack("trit5_pack", w, scales, L)


def bit2_pack(w, scales, L: Layout) -> np.ndarray:
    return _pack("bit2_pack", w, scales, L)


def _unpack(fn: str, L: Layout, blob) -> tuple[np.ndarray, np.ndarray]:
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    w = np.empty((L.n, L.k), dtype=np.int8)
    s = np.empty(num_scales(L), dtype=np.uint16)
    N.check(getattr(N.lib(), fn)(ctypes.byref(L), _ptr(blob), blob.nbytes, _ptr(w), _ptr(s)), fn)
    return w, s


def bitcos_unpack(L: Layout, blob):
    return _unpack("bitcos_unpack", L, blob)


def trit5_unpack(L: Layout, blob):
    return _unpack("trit5_unpack", L, blob)


def bit2_unpack(L: Layout, blob):
    return _unpack("bit2_unpack", L, blob)


def plan_and_pack(fmt: int, w, scales, group: int = 128, unit_rows: int = 0):
    """(layout, host blob) for one of the three formats."""
    if fmt == FMT_BITCOS:
        L = bitcos_plan(w, group, unit_rows)
        return L, bitcos_pack(w, scales, L)
    if fmt == FMT_TRIT5:
        L = trit5_plan(w, group)
        return L, trit5_pack(w, scales, L)
    if fmt == FMT_BIT2:
        L = bit2_plan(w, group)
        return L, bit2_pack(w, scales, L)
    raise ValueError(f"unknown format {fmt}")


def bitcos_pack_device(w_dev, scales_dev, group: int = 128, unit_rows: int = 0, stream=None):
    """(layout, device blob) packed on the GPU from device tensors: W int8 [n][k]
    and fp16 scales ([n][k/128] or [1]).  Same bytes as the host packer."""
    import torch
    if w_dev.dtype != torch.int8 or w_dev.dim() != 2 or not w_dev.is_cuda or not w_dev.is_contiguous():
        raise ValueError("w_dev must be a contiguous 2-D int8 CUDA tensor")
    if scales_dev.dtype not in (torch.float16, torch.int16) or not scales_dev.is_cuda or not scales_dev.is_contiguous():
        raise ValueError("scales_dev must be a contiguous fp16 CUDA tensor")
    n, k = w_dev.shape
    ws_bytes = N.lib().bitcos_plan_device_workspace(n)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=w_dev.device)
    L = Layout()
    h = _stream_handle(stream)
    N.check(N.lib().bitcos_plan_device(ctypes.c_void_p(w_dev.data_ptr()), n, k, group, unit_rows,
                                       ctypes.c_void_p(ws.data_ptr()), ws_bytes, ctypes.byref(L), h),
            "bitcos_plan_device")
    if scales_dev.numel() != num_scales(L):
        raise ValueError(f"scales_dev has {scales_dev.numel()} values, layout needs {num_scales(L)}")
    blob = torch.empty(L.total_bytes, dtype=torch.uint8, device=w_dev.device)
    N.check(N.lib().bitcos_pack_device(ctypes.c_void_p(w_dev.data_ptr()), ctypes.c_void_p(scales_dev.data_ptr()),
                                       ctypes.byref(L), ctypes.c_void_p(ws.data_ptr()), ws_bytes,
                                       ctypes.c_void_p(blob.data_ptr()), L.total_bytes, h),
            "bitcos_pack_device")
    return L, blob


def bitcos_pack_device_noalloc(w_dev, scales_dev, dst_dev, group: int = 128, unit_rows: int = 0, stream=None):
    """Layout of W packed on the GPU into the caller's dst_dev (a uint8 cuda
    tensor), with the library's fixed per-GPU workspace: no device memory is
    allocated by the call.  Raises BitcosError(E_SPACE) if dst_dev is too
    small (its .status tells; the layout needed is in the exception's
    `layout`)."""
    import torch
    if w_dev.dtype != torch.int8 or w_dev.dim() != 2 or not w_dev.is_cuda or not w_dev.is_contiguous():
        raise ValueError("w_dev must be a contiguous 2-D int8 CUDA tensor")
    if scales_dev.dtype not in (torch.float16, torch.int16) or not scales_dev.is_cuda or not scales_dev.is_contiguous():
        raise ValueError("scales_dev must be a contiguous fp16 CUDA tensor")
    if dst_dev.dtype != torch.uint8 or not dst_dev.is_cuda or not dst_dev.is_contiguous():
        raise ValueError("dst_dev must be a contiguous uint8 CUDA tensor")
    n, k = w_dev.shape
    ns = n * (k // 128) if group == 128 else 1
    if scales_dev.numel() != ns:
        raise ValueError(f"scales_dev has {scales_dev.numel()} values, the layout needs {ns}")
    L = Layout()
    st = N.lib().bitcos_pack_device_noalloc(ctypes.c_void_p(w_dev.data_ptr()), ctypes.c_void_p(scales_dev.data_ptr()),
                                            n, k, group, unit_rows, ctypes.byref(L),
                                            ctypes.c_void_p(dst_dev.data_ptr()), dst_dev.numel(),
                                            _stream_handle(stream))
    if st:
        err = N.BitcosError(st, "bitcos_pack_device_noalloc")
        err.layout = L
        raise err
    return L


# ---------------------------------------------------------------------------
# GEMV (device)
# ---------------------------------------------------------------------------

_GEMV = {FMT_BITCOS: "bitcos_gemv", FMT_TRIT5: "trit5_gemv", FMT_BIT2: "bit2_gemv"}


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def gemv(L: Layout, blob_dev, x, y, xscale=None, y_mode: int = Y_F32, stream=None):
    """Enqueue y = (S (.) W) x for the layout's format on `stream`.

    blob_dev: uint8 cuda tensor of >= L.total_bytes; x: int8 or bfloat16 cuda
    tensor [m, k] (or [k]); y: float32 (Y_F32, Y_F32_ADD) or int32 (Y_I32_RAW,
    Y_I32_RAW_ADD) cuda tensor [m, n] (or [n]), overwritten or (the _ADD modes)
    added onto; xscale: None or float32 cuda tensor [m, k/128].
    """
    import torch
    m = x.shape[0] if x.dim() == 2 else 1
    if x.dtype == torch.int8:
        xd = X_I8
    elif x.dtype == torch.bfloat16:
        xd = X_BF16
    else:
        raise TypeError("x must be int8 or bfloat16")
    for t, nm in ((blob_dev, "blob"), (x, "x"), (y, "y")):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{nm} must be a contiguous cuda tensor")
    if blob_dev.dtype != torch.uint8 or blob_dev.numel() < L.total_bytes:
        raise ValueError("blob_dev must be uint8 with at least total_bytes elements")
    if x.numel() != m * L.k:
        raise ValueError("x has the wrong size")
    want_y = torch.int32 if y_mode in (Y_I32_RAW, Y_I32_RAW_ADD) else torch.float32
    if y.dtype != want_y or y.numel() != m * L.n:
        raise ValueError("y has the wrong dtype or size")
    xs_ptr = None
    if xscale is not None:
        if (not xscale.is_cuda or xscale.dtype != torch.float32 or not xscale.is_contiguous()
                or xscale.numel() != m * (L.k // 128) or L.k % 128):
            raise ValueError("xscale must be a contiguous float32 cuda tensor [m, k/128]")
        xs_ptr = ctypes.c_void_p(xscale.data_ptr())
    fn = getattr(N.lib(), _GEMV[L.format])
    st = fn(ctypes.byref(L), ctypes.c_void_p(blob_dev.data_ptr()), m, ctypes.c_void_p(x.data_ptr()), xd,
            xs_ptr, ctypes.c_void_p(y.data_ptr()), y_mode, _stream_handle(stream))
    N.check(st, _GEMV[L.format])
    return y


def bitcos_gemv(L, blob_dev, x, y, xscale=None, y_mode=Y_F32, stream=None):
    assert L.format == FMT_BITCOS
    return gemv(L, blob_dev, x, y, xscale, y_mode, stream)


def trit5_gemv(L, blob_dev, x, y, xscale=None, y_mode=Y_F32, stream=None):
    assert L.format == FMT_TRIT5
    return gemv(L, blob_dev, x, y, xscale, y_mode, stream)


def bit2_gemv(L, blob_dev, x, y, xscale=None, y_mode=Y_F32, stream=None):
    assert L.format == FMT_BIT2
    return gemv(L, blob_dev, x, y, xscale, y_mode, stream)


def describe(L: Layout, m: int = 1, x_dtype: int = X_I8) -> LaunchInfo:
    info = LaunchInfo()
    N.check(N.lib().bitcos_describe(ctypes.byref(L), m, x_dtype, ctypes.byref(info)), "bitcos_describe")
    return info


def add_partials(y, parts, stream=None):
    """Enqueue y += parts[0] + parts[1] + ... (fp32, in that order) on
    `stream`: the partial outputs of a split row's later column blocks.
    y: contiguous float32 cuda tensor of n elements; parts: contiguous float32
    cuda tensor [nparts, ...] of nparts * n elements."""
    import torch
    for t, nm in ((y, "y"), (parts, "parts")):
        if not t.is_cuda or not t.is_contiguous() or t.dtype != torch.float32:
            raise ValueError(f"{nm} must be a contiguous float32 cuda tensor")
    n = y.numel()
    if parts.dim() < 1 or parts.shape[0] < 1 or parts.numel() != parts.shape[0] * n:
        raise ValueError("parts must hold nparts slices of y's size")
    N.check(N.lib().bitcos_add_partials(ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(parts.data_ptr()),
                                        int(parts.shape[0]), n, _stream_handle(stream)), "bitcos_add_partials")
    return y


def quantize_activations(x, q, scale, stream=None):
    """Device int8 quantisation of bf16 activations per group of 128 (see bitcos.h)."""
    import torch
    if x.dtype != torch.bfloat16 or q.dtype != torch.int8 or scale.dtype != torch.float32:
        raise TypeError("x bfloat16, q int8, scale float32")
    for t in (x, q, scale):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("contiguous cuda tensors required")
    m = x.shape[0] if x.dim() == 2 else 1
    k = x.numel() // m
    if q.numel() != m * k or scale.numel() != m * (k // 128) or k % 128:
        raise ValueError("q must be [m, k] and scale [m, k/128], k % 128 == 0")
    N.check(N.lib().bitcos_quantize_act(ctypes.c_void_p(x.data_ptr()), m, k, ctypes.c_void_p(q.data_ptr()),
                                        ctypes.c_void_p(scale.data_ptr()), _stream_handle(stream)),
            "bitcos_quantize_act")
    return q, scale


class Batch:
    """A list of GEMVs of one format and tile, run as one persistent launch.

    Holds the host table and its device copy; the device buffers it points to
    (blobs, activations, outputs) must outlive it.  Every GEMV takes the same
    number m of activation rows: xs[i] is [m, k] (or [k] for m = 1) and ys[i]
    [m, n]; m > 1 runs the small-batch kernel.
    """

    def __init__(self, layouts, blobs_dev, xs, ys, xscales=None, y_mode: int = Y_F32):
        import torch
        count = len(layouts)
        if not (count == len(blobs_dev) == len(xs) == len(ys)) or count < 1:
            raise ValueError("layouts, blobs, xs and ys must have the same non-zero length")
        x_dtype = X_I8 if xs[0].dtype == torch.int8 else X_BF16
        m = xs[0].shape[0] if xs[0].dim() == 2 else 1
        arr = (Layout * count)(*layouts)
        for L, b, x, y in zip(layouts, blobs_dev, xs, ys):
            _check_gemv_buffers(L, b, x, y, None, y_mode, m)
        if xscales is not None:
            for L, xs_ in zip(layouts, xscales):
                if xs_ is not None:
                    _check_xscale(L, xs_, m)
        P = ctypes.c_void_p
        blobs = (P * count)(*[b.data_ptr() for b in blobs_dev])
        xp = (P * count)(*[x.data_ptr() for x in xs])
        yp = (P * count)(*[y.data_ptr() for y in ys])
        sp = None if xscales is None else (P * count)(*[0 if s is None else s.data_ptr() for s in xscales])
        nbytes = N.lib().bitcos_batch_bytes(count)
        self.host = np.zeros(nbytes, dtype=np.uint8)
        N.check(N.lib().bitcos_batch_build(count, m, arr, blobs, xp, sp, yp, x_dtype, y_mode,
                                           _ptr(self.host), nbytes), "bitcos_batch_build")
        self.dev = torch.from_numpy(self.host).cuda()
        self.count = count
        self.m = m
        self._keep = (layouts, blobs_dev, xs, ys, xscales)

    def run(self, stream=None):
        N.check(N.lib().bitcos_gemv_batch(_ptr(self.host), ctypes.c_void_p(self.dev.data_ptr()),
                                          _stream_handle(stream)), "bitcos_gemv_batch")


def _check_gemv_buffers(L, blob_dev, x, y, xscale, y_mode, m=1):
    import torch
    for t, nm in ((blob_dev, "blob"), (x, "x"), (y, "y")):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{nm} must be a contiguous cuda tensor")
    if blob_dev.dtype != torch.uint8 or blob_dev.numel() < L.total_bytes:
        raise ValueError("blob_dev must be uint8 with at least total_bytes elements")
    if x.numel() != m * L.k or x.dtype not in (torch.int8, torch.bfloat16):
        raise ValueError("x must be int8 or bfloat16 with m * k elements")
    want_y = torch.int32 if y_mode in (Y_I32_RAW, Y_I32_RAW_ADD) else torch.float32
    if y.dtype != want_y or y.numel() != m * L.n:
        raise ValueError("y has the wrong dtype or size")


def _check_xscale(L, xscale, m):
    import torch
    if (not xscale.is_cuda or xscale.dtype != torch.float32 or not xscale.is_contiguous()
            or xscale.numel() != m * (L.k // 128) or L.k % 128):
        raise ValueError("xscale must be a contiguous float32 cuda tensor [m, k/128]")
