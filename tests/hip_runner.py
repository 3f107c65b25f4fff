"""Helpers that drive the HIP library through its C ABI (via the ctypes binding) and return numpy arrays."""
from __future__ import annotations

import numpy as np
import torch

import paper_2502_11880_amd as B

DEV = "cuda:0"


def pack(W: torch.Tensor, layout="i2s"):
    """Pack an fp32 [N, K] tensor on the GPU; returns (packed uint8 device tensor, w_scale device tensor)."""
    W = W.to(DEV).contiguous()
    N, K = W.shape
    packed = torch.empty(B.bitnet_packed_bytes(layout, N, K), dtype=torch.uint8, device=DEV)
    w_scale = torch.empty(1, dtype=torch.float32, device=DEV)
    ws = torch.empty(B.bitnet_pack_workspace_bytes(N, K), dtype=torch.uint8, device=DEV)
    B.bitnet_pack_weights(layout, W, packed, w_scale, ws)
    return packed, w_scale


def quantize(x: torch.Tensor, with_rowsum=False):
    x = x.to(DEV).contiguous()
    M, K = x.shape
    xq = torch.empty((M, K), dtype=torch.int8, device=DEV)
    s = torch.empty(M, dtype=torch.float32, device=DEV)
    rs = torch.empty(M, dtype=torch.int32, device=DEV) if with_rowsum else None
    B.bitnet_quantize_act(x, xq, s, rs)
    return (xq, s, rs) if with_rowsum else (xq, s)


def workspace(layout, M, N, K):
    nbytes = B.bitnet_mpgemm_workspace_bytes(layout, M, N, K)
    return torch.zeros(max(nbytes, 16), dtype=torch.uint8, device=DEV)


def mpgemm(layout, packed, w_scale, N, K, xq, s, ws=None, want_acc=True, x_rowsum=None):
    M = xq.shape[0]
    y = torch.empty((M, N), dtype=torch.float32, device=DEV)
    acc = torch.empty((M, N), dtype=torch.int32, device=DEV) if want_acc else None
    if ws is None:
        ws = workspace(layout, M, N, K)
    B.bitnet_mpgemm(layout, packed, w_scale, N, K, xq, s, y, acc, ws, x_rowsum=x_rowsum)
    return y, acc


def to_np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def check_y(y_gpu: np.ndarray, y_ref: np.ndarray, acc: np.ndarray, rtol=1e-5):
    """fp32 outputs within rtol of the float64 reference; exact zeros where acc == 0."""
    y_gpu = y_gpu.astype(np.float64)
    err = np.abs(y_gpu - y_ref)
    bad = err > rtol * np.abs(y_ref)
    assert not bad.any(), f"{int(bad.sum())} outputs outside {rtol} relative; worst {float((err / np.maximum(np.abs(y_ref), 1e-30)).max())}"
    assert np.all(y_gpu[acc == 0] == 0.0)
