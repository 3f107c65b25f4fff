"""Ternary-weight x int8-activation mpGEMM for AMD MI355X (gfx950), after Bitnet.cpp (arXiv 2502.11880).

This package is a thin ctypes binding over the C ABI in ``include/bitnet_mi355x.h``: each function
below has the name of the C entry point it calls, checks and marshals its torch arguments (device,
dtype, contiguity) and raises ``BitnetError`` on a non-OK status.  All arithmetic runs in the HIP
kernels of ``libbitnet_mi355x.so``; if that library has not been built, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

LIB_NAME = "libbitnet_mi355x.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

BITNET_LAYOUT_I2S = 0
BITNET_LAYOUT_TL2 = 1
BITNET_LAYOUT_TL1 = 2
BITNET_LAYOUT_C4G2 = 3
BITNET_LAYOUT_C5G2 = 4
BITNET_LAYOUT_C3G5 = 5
BITNET_LAYOUT_TL2_0 = 6
BITNET_LAYOUT_TL1_0 = 7
LAYOUTS = {"i2s": BITNET_LAYOUT_I2S, "tl2": BITNET_LAYOUT_TL2, "tl1": BITNET_LAYOUT_TL1, "c4g2": BITNET_LAYOUT_C4G2,
           "c5g2": BITNET_LAYOUT_C5G2, "c3g5": BITNET_LAYOUT_C3G5, "tl2_0": BITNET_LAYOUT_TL2_0,
           "tl1_0": BITNET_LAYOUT_TL1_0}
INT_LAYOUTS = ("c4g2", "c5g2", "c3g5")

BITNET_OK = 0
STATUS_NAMES = {0: "BITNET_OK", 1: "BITNET_E_INVALID", 2: "BITNET_E_SHAPE", 3: "BITNET_E_ALIGN",
                4: "BITNET_E_LAYOUT", 5: "BITNET_E_WORKSPACE", 6: "BITNET_E_HIP"}

# (name, restype, argtypes) of every exported entry point, in header order
_SIGNATURES = [
    ("bitnet_packed_bytes", ctypes.c_size_t, [ctypes.c_int, ctypes.c_int64, ctypes.c_int64]),
    ("bitnet_pack_workspace_bytes", ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64]),
    ("bitnet_pack_weights", ctypes.c_int,
     [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t,
      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    ("bitnet_pack_int_weights", ctypes.c_int,
     [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    ("bitnet_quantize_act", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
      ctypes.c_void_p]),
    ("bitnet_mpgemm_workspace_bytes", ctypes.c_size_t, [ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]),
    ("bitnet_mpgemm", ctypes.c_int,
     [ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    ("bitnet_mpgemm_noalloc", ctypes.c_int,
     [ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
      ctypes.c_void_p]),
    ("bitnet_mpgemm_fused_workspace_bytes", ctypes.c_size_t,
     [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]),
    ("bitnet_mpgemm_fused", ctypes.c_int,
     [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
      ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    ("bitnet_elut_tables", ctypes.c_int,
     [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    ("bitnet_status_string", ctypes.c_char_p, [ctypes.c_int]),
    ("bitnet_last_error", ctypes.c_char_p, []),
]

_lock = threading.Lock()
_handle = None


class BitnetError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        self.status = status
        super().__init__(f"{fn} failed: {STATUS_NAMES.get(status, status)}: {detail}")


def lib():
    """The loaded C library (loads it on first use; raises if it is not built)."""
    global _handle
    with _lock:
        if _handle is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_NAME} is not built; run `python -m paper_2502_11880_amd.build` "
                                   "(or __graft_entry__.build()) first")
            h = ctypes.CDLL(LIB_PATH)
            for name, res, args in _SIGNATURES:
                fn = getattr(h, name)
                fn.restype = res
                fn.argtypes = args
            _handle = h
        return _handle


def _check(fn: str, status: int) -> None:
    if status != BITNET_OK:
        detail = lib().bitnet_last_error().decode(errors="replace")
        raise BitnetError(fn, status, detail)


def _layout(layout) -> int:
    if isinstance(layout, str):
        return LAYOUTS[layout.lower()]
    return int(layout)


def _ptr(t, name, dtype=None, device=True):
    if t is None:
        return None
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if device and not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------------------------------------
# Size queries (pure host functions)
# ------------------------------------------------------------------------------------------------
def bitnet_packed_bytes(layout, N: int, K: int) -> int:
    return int(lib().bitnet_packed_bytes(_layout(layout), N, K))


def bitnet_pack_workspace_bytes(N: int, K: int) -> int:
    return int(lib().bitnet_pack_workspace_bytes(N, K))


def bitnet_mpgemm_workspace_bytes(layout, M: int, N: int, K: int) -> int:
    return int(lib().bitnet_mpgemm_workspace_bytes(_layout(layout), M, N, K))


# ------------------------------------------------------------------------------------------------
# Entry points
# ------------------------------------------------------------------------------------------------
def bitnet_pack_weights(layout, W, packed, w_scale, ws, stream=None) -> None:
    """Ternarise and pack W (fp32 [N, K], device) into `packed` (uint8) and `w_scale` (fp32 [1])."""
    import torch
    N, K = W.shape
    st = lib().bitnet_pack_weights(_layout(layout), _ptr(W, "W", torch.float32), N, K,
                                   _ptr(packed, "packed", torch.uint8), packed.numel(),
                                   _ptr(w_scale, "w_scale", torch.float32), _ptr(ws, "ws"),
                                   ws.numel() * ws.element_size(), _stream(stream))
    _check("bitnet_pack_weights", st)


def bitnet_pack_int_weights(layout, Wq, packed, stream=None) -> None:
    """Pack integer weights Wq (int8 [N, K], device) for an integer-weight layout (c4g2, c5g2, c3g5)."""
    import torch
    N, K = Wq.shape
    st = lib().bitnet_pack_int_weights(_layout(layout), _ptr(Wq, "Wq", torch.int8), N, K,
                                       _ptr(packed, "packed", torch.uint8), packed.numel(), _stream(stream))
    _check("bitnet_pack_int_weights", st)


def bitnet_quantize_act(x, xq, x_scale, x_rowsum=None, stream=None) -> None:
    """Per-token absmax int8 quantisation of x (fp32 [M, K], device) into xq (int8), x_scale (fp32 [M]) and,
    optionally, x_rowsum (int32 [M])."""
    import torch
    M, K = x.shape
    st = lib().bitnet_quantize_act(_ptr(x, "x", torch.float32), M, K, _ptr(xq, "xq", torch.int8),
                                   _ptr(x_scale, "x_scale", torch.float32), _ptr(x_rowsum, "x_rowsum", torch.int32),
                                   _stream(stream))
    _check("bitnet_quantize_act", st)


def bitnet_mpgemm(layout, packed, w_scale, N: int, K: int, xq, x_scale, y, acc=None, ws=None, stream=None,
                  x_rowsum=None) -> None:
    """y = dequant(xq @ t^T) for the packed ternary weight; optionally the exact int32 accumulators."""
    import torch
    M = xq.shape[0]
    ws_ptr = _ptr(ws, "ws") if ws is not None else None
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    st = lib().bitnet_mpgemm(_layout(layout), _ptr(packed, "packed", torch.uint8), packed.numel(),
                             _ptr(w_scale, "w_scale", torch.float32), N, K, _ptr(xq, "xq", torch.int8),
                             _ptr(x_scale, "x_scale", torch.float32), _ptr(x_rowsum, "x_rowsum", torch.int32), M,
                             _ptr(y, "y", torch.float32),
                             _ptr(acc, "acc", torch.int32), ws_ptr, ws_bytes, _stream(stream))
    _check("bitnet_mpgemm", st)


NOALLOC_SCRATCH_BYTES = 32 << 20     # BITNET_NOALLOC_SCRATCH_BYTES


def bitnet_mpgemm_noalloc(layout, packed, w_scale, N: int, K: int, xq, x_scale, y, acc=None, stream=None,
                          x_rowsum=None) -> None:
    """bitnet_mpgemm with its workspace taken from the library's static per-GPU scratch (no allocation)."""
    import torch
    M = xq.shape[0]
    st = lib().bitnet_mpgemm_noalloc(_layout(layout), _ptr(packed, "packed", torch.uint8), packed.numel(),
                                     _ptr(w_scale, "w_scale", torch.float32), N, K, _ptr(xq, "xq", torch.int8),
                                     _ptr(x_scale, "x_scale", torch.float32),
                                     _ptr(x_rowsum, "x_rowsum", torch.int32), M, _ptr(y, "y", torch.float32),
                                     _ptr(acc, "acc", torch.int32), _stream(stream))
    _check("bitnet_mpgemm_noalloc", st)


def bitnet_mpgemm_fused_workspace_bytes(layout, Ns, K: int, M: int) -> int:
    """Workspace bytes with which bitnet_mpgemm_fused runs every K split it can use for weights of rows Ns (a list)
    at M tokens: at least the largest single-weight workspace."""
    arr = (ctypes.c_int64 * len(Ns))(*Ns)
    return int(lib().bitnet_mpgemm_fused_workspace_bytes(_layout(layout), len(Ns), arr, K, M))


class FusedArgs:
    """Host arrays for bitnet_mpgemm_fused, built once so repeated calls only pass pointers."""

    def __init__(self, packed, w_scales, ys):
        import torch
        n = len(packed)
        self.n = n
        self.packed = (ctypes.c_void_p * n)(*[_ptr(p, "packed", torch.uint8) for p in packed])
        self.packed_bytes = (ctypes.c_size_t * n)(*[p.numel() for p in packed])
        self.w_scale = (ctypes.c_void_p * n)(*[_ptr(w, "w_scale", torch.float32) for w in w_scales])
        self.N = (ctypes.c_int64 * n)(*[y.shape[1] for y in ys])
        self.y = (ctypes.c_void_p * n)(*[_ptr(y, "y", torch.float32) for y in ys])
        self._keep = (list(packed), list(w_scales), list(ys))


def bitnet_mpgemm_fused(layout, packed, w_scales, x, xq, x_scale, x_rowsum, ys, ws=None, stream=None,
                        args: FusedArgs = None) -> None:
    """Quantise x (fp32 [M, K]) and multiply it by every packed weight (lists of equal length) in one call.
    With x None, xq / x_scale / x_rowsum already hold the quantised activation and only the products run."""
    import torch
    M, K = (x if x is not None else xq).shape
    a = args if args is not None else FusedArgs(packed, w_scales, ys)
    if a.n < 1:
        raise ValueError("bitnet_mpgemm_fused needs at least one weight")
    ws_ptr = _ptr(ws, "ws") if ws is not None else None
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    st = lib().bitnet_mpgemm_fused(_layout(layout), a.n, a.packed, a.packed_bytes, a.w_scale, a.N, K,
                                   _ptr(x, "x", torch.float32) if x is not None else None, M,
                                   _ptr(xq, "xq", torch.int8),
                                   _ptr(x_scale, "x_scale", torch.float32), _ptr(x_rowsum, "x_rowsum", torch.int32),
                                   a.y, ws_ptr, ws_bytes, _stream(stream))
    _check("bitnet_mpgemm_fused", st)


def bitnet_elut_tables(xq, lut, lut1=None, stream=None) -> None:
    """TL2 activation tables of xq (int8 [M, K], device) into lut (int16 [M, ThreeK/3, 16]) and lut1."""
    import torch
    M, K = xq.shape
    st = lib().bitnet_elut_tables(_ptr(xq, "xq", torch.int8), M, K, _ptr(lut, "lut", torch.int16),
                                  _ptr(lut1, "lut1", torch.int16), _stream(stream))
    _check("bitnet_elut_tables", st)


def bitnet_status_string(status: int) -> str:
    return lib().bitnet_status_string(status).decode()


def bitnet_last_error() -> str:
    return lib().bitnet_last_error().decode(errors="replace")
