"""Torch-tensor front end of the C ABI.

PyTorch supplies device memory and the current stream; these functions only
check tensor metadata, allocate outputs and pass raw pointers to
libhscale.so.  All arithmetic happens in the library's HIP kernels.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import HScaleError


def _check(status: int, where: str) -> None:
    if status != _lib.HSCALE_OK:
        raise HScaleError(status, where)


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _bf16_matrix(t: torch.Tensor, name: str) -> None:
    if t.dtype != torch.bfloat16 or t.dim() != 2 or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous 2-D bf16 CUDA tensor")


def hdiag_workspace_bytes(tokens: int, in_features: int) -> int:
    """Bytes of scratch hdiag needs for a [tokens, in_features] X."""
    return _lib.hscale_hdiag_workspace_bytes(tokens, in_features)


def hdiag(X: torch.Tensor, h: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
          stream=None) -> torch.Tensor:
    """h = diag(X^T X) (Sec. 3.2, Eq. 4) of bf16 X [tokens, in] as fp32 [in]."""
    _bf16_matrix(X, "X")
    T, n = X.shape
    if h is None:
        h = torch.empty(n, dtype=torch.float32, device=X.device)
    need = hdiag_workspace_bytes(T, n)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.hscale_hdiag(X.data_ptr(), T, n, h.data_ptr(), ws_ptr, ws_bytes, _stream(stream)),
           "hscale_hdiag")
    return h


def search(W: torch.Tensor, h: torch.Tensor, global_scale: float, window: int | None = None,
           down: int | None = None, up: int | None = None, scale_codes: torch.Tensor | None = None,
           packed_e2m1: torch.Tensor | None = None, stream=None):
    """The per-group NVFP4 scale search (Sec. 3.3).  Returns
    (scale_codes uint8 [out, in/16], packed_e2m1 uint8 [out, in/2])."""
    _bf16_matrix(W, "W")
    m, n = W.shape
    if h.dtype != torch.float32 or h.shape != (n,) or not h.is_contiguous():
        raise ValueError("h must be a contiguous fp32 tensor of shape [in]")
    if scale_codes is None:
        scale_codes = torch.empty((m, n // 16), dtype=torch.uint8, device=W.device)
    if packed_e2m1 is None:
        packed_e2m1 = torch.empty((m, n // 2), dtype=torch.uint8, device=W.device)
    s = _stream(stream)
    if window is not None:
        if down is not None or up is not None:
            raise ValueError("give either window or down/up")
        st = _lib.hscale_search(W.data_ptr(), m, n, h.data_ptr(), int(window), float(global_scale),
                                scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search")
    else:
        st = _lib.hscale_search_du(W.data_ptr(), m, n, h.data_ptr(), int(down), int(up),
                                   float(global_scale), scale_codes.data_ptr(),
                                   packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_du")
    return scale_codes, packed_e2m1


def quantize(W: torch.Tensor, global_scale: float, scale_codes: torch.Tensor,
             packed_e2m1: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Packed E2M1 codes of W at the given scale codes (final re-quantization)."""
    _bf16_matrix(W, "W")
    m, n = W.shape
    if scale_codes.dtype != torch.uint8 or scale_codes.shape != (m, n // 16) or not scale_codes.is_contiguous():
        raise ValueError("scale_codes must be a contiguous uint8 tensor [out, in/16]")
    if packed_e2m1 is None:
        packed_e2m1 = torch.empty((m, n // 2), dtype=torch.uint8, device=W.device)
    _check(_lib.hscale_quantize(W.data_ptr(), m, n, float(global_scale), scale_codes.data_ptr(),
                                packed_e2m1.data_ptr(), _stream(stream)), "hscale_quantize")
    return packed_e2m1
