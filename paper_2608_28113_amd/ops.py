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


def _init_mode(init):
    if isinstance(init, str):
        return {"maxabs": _lib.HSCALE_INIT_MAXABS, "rtn": _lib.HSCALE_INIT_MAXABS,
                "4over6": _lib.HSCALE_INIT_4OVER6}[init], None
    if isinstance(init, torch.Tensor):
        if init.dtype != torch.uint8 or not init.is_cuda:
            raise ValueError("initial codes must be a uint8 CUDA tensor")
        return _lib.HSCALE_INIT_GIVEN, init
    raise ValueError("init must be 'maxabs', '4over6' or a uint8 tensor of codes")


def search(W: torch.Tensor, h: torch.Tensor, global_scale: float, window: int | None = None,
           down: int | None = None, up: int | None = None, init="maxabs",
           scale_codes: torch.Tensor | None = None, packed_e2m1: torch.Tensor | None = None, stream=None):
    """The per-group NVFP4 scale search (Sec. 3.3).  Returns
    (scale_codes uint8 [out, in/16], packed_e2m1 uint8 [out, in/2]).

    ``window`` gives the symmetric shift set -window..+window; ``down``/``up``
    the paper's asymmetric one.  ``init`` is "maxabs" (Eq. 7), "4over6", or a
    uint8 tensor [out, in/16] of initial codes (it may be ``scale_codes``
    itself, to refine in place).
    """
    _bf16_matrix(W, "W")
    m, n = W.shape
    if h.dtype != torch.float32 or h.shape != (n,) or not h.is_contiguous():
        raise ValueError("h must be a contiguous fp32 tensor of shape [in]")
    if window is not None:
        if down is not None or up is not None:
            raise ValueError("give either window or down/up")
        down = up = int(window)
    if down is None or up is None:
        raise ValueError("give window or both down and up")
    mode, init_t = _init_mode(init)
    if scale_codes is None:
        scale_codes = torch.empty((m, n // 16), dtype=torch.uint8, device=W.device)
    if packed_e2m1 is None:
        packed_e2m1 = torch.empty((m, n // 2), dtype=torch.uint8, device=W.device)
    s = _stream(stream)
    if mode == _lib.HSCALE_INIT_MAXABS:
        st = _lib.hscale_search_du(W.data_ptr(), m, n, h.data_ptr(), int(down), int(up), float(global_scale),
                                   scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_du")
    elif mode == _lib.HSCALE_INIT_4OVER6:
        st = _lib.hscale_search_4over6(W.data_ptr(), m, n, h.data_ptr(), int(down), int(up),
                                       float(global_scale), scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_4over6")
    else:
        if init_t.shape != (m, n // 16) or not init_t.is_contiguous():
            raise ValueError("initial codes must be a contiguous uint8 tensor [out, in/16]")
        st = _lib.hscale_search_from(W.data_ptr(), m, n, h.data_ptr(), int(down), int(up), float(global_scale),
                                     init_t.data_ptr(), scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_from")
    return scale_codes, packed_e2m1


def _row_view(t: torch.Tensor, dtype, name: str):
    if t.dtype != dtype or t.dim() != 2 or not t.is_cuda or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be a 2-D {dtype} CUDA tensor (view) with unit column stride")
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def search_block(W: torch.Tensor, h: torch.Tensor, global_scale: float, down: int, up: int,
                 scale_codes: torch.Tensor, packed_e2m1: torch.Tensor, init="maxabs", stream=None):
    """The search on a column block given as strided views: W = Wfull[:, a:b]
    (bf16), h = hfull[a:b], scale_codes = codes[:, a/16:b/16] and
    packed_e2m1 = packed[:, a/2:b/2] (uint8), as in the paper's GPTQ
    combination (App. B).  Outputs are written in place."""
    m, cols = W.shape
    ldw = _row_view(W, torch.bfloat16, "W")
    ldc = _row_view(scale_codes, torch.uint8, "scale_codes")
    ldp = _row_view(packed_e2m1, torch.uint8, "packed_e2m1")
    if scale_codes.shape != (m, cols // 16) or packed_e2m1.shape != (m, cols // 2):
        raise ValueError("output views do not match the block")
    if h.dtype != torch.float32 or h.shape != (cols,) or not h.is_contiguous():
        raise ValueError("h must be a contiguous fp32 slice of shape [cols]")
    mode, init_t = _init_mode(init)
    ldi = 0
    iptr = 0
    if init_t is not None:
        ldi = _row_view(init_t, torch.uint8, "init codes")
        if init_t.shape != (m, cols // 16):
            raise ValueError("initial codes do not match the block")
        iptr = init_t.data_ptr()
    st = _lib.hscale_search_block(W.data_ptr(), ldw, m, cols, h.data_ptr(), int(down), int(up),
                                  float(global_scale), mode, iptr, ldi, scale_codes.data_ptr(), ldc,
                                  packed_e2m1.data_ptr(), ldp, _stream(stream))
    _check(st, "hscale_search_block")
    return scale_codes, packed_e2m1


def hdiag_accumulate(X: torch.Tensor, h64: torch.Tensor, workspace: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """h64 += diag(X^T X) for one calibration batch (fp64 accumulator)."""
    _bf16_matrix(X, "X")
    T, n = X.shape
    if h64.dtype != torch.float64 or h64.shape != (n,) or not h64.is_contiguous():
        raise ValueError("h64 must be a contiguous fp64 tensor of shape [in]")
    need = hdiag_workspace_bytes(T, n)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.hscale_hdiag_accumulate(X.data_ptr(), T, n, h64.data_ptr(), ws_ptr, ws_bytes,
                                        _stream(stream)), "hscale_hdiag_accumulate")
    return h64


def hdiag_finalize(h64: torch.Tensor, h: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """h = fp32(h64)."""
    n = h64.shape[0]
    if h is None:
        h = torch.empty(n, dtype=torch.float32, device=h64.device)
    _check(_lib.hscale_hdiag_finalize(h64.data_ptr(), n, h.data_ptr(), _stream(stream)), "hscale_hdiag_finalize")
    return h


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


def search_stats(W: torch.Tensor, h: torch.Tensor, global_scale: float, down: int, up: int, init="maxabs",
                 stream=None):
    """The search with per-group statistics.  Returns a dict of
    scale_codes, packed_e2m1, shift (int8 [out, in/16], the chosen shift),
    err_best and err_init (fp32 [out, in/16], the score at the chosen shift
    and at shift 0)."""
    _bf16_matrix(W, "W")
    m, n = W.shape
    if h.dtype != torch.float32 or h.shape != (n,) or not h.is_contiguous():
        raise ValueError("h must be a contiguous fp32 tensor of shape [in]")
    mode, init_t = _init_mode(init)
    iptr = 0
    if init_t is not None:
        if init_t.shape != (m, n // 16) or not init_t.is_contiguous():
            raise ValueError("initial codes must be a contiguous uint8 tensor [out, in/16]")
        iptr = init_t.data_ptr()
    G = (m, n // 16)
    out = dict(scale_codes=torch.empty(G, dtype=torch.uint8, device=W.device),
               packed_e2m1=torch.empty((m, n // 2), dtype=torch.uint8, device=W.device),
               shift=torch.empty(G, dtype=torch.int8, device=W.device),
               err_best=torch.empty(G, dtype=torch.float32, device=W.device),
               err_init=torch.empty(G, dtype=torch.float32, device=W.device))
    st = _lib.hscale_search_stats(W.data_ptr(), m, n, h.data_ptr(), int(down), int(up), float(global_scale), mode,
                                  iptr, out["scale_codes"].data_ptr(), out["packed_e2m1"].data_ptr(),
                                  out["shift"].data_ptr(), out["err_best"].data_ptr(), out["err_init"].data_ptr(),
                                  _stream(stream))
    _check(st, "hscale_search_stats")
    return out


def shift_summary(shift: torch.Tensor, err_best: torch.Tensor, err_init: torch.Tensor, down: int, up: int,
                  stream=None) -> dict:
    """Per-shift counts and fp64 sums of initial errors, chosen errors and
    relative reductions over the groups (bins d = -down..up), as tensors of
    length down + up + 1 on the device."""
    groups = shift.numel()
    for t, dt, name in ((shift, torch.int8, "shift"), (err_best, torch.float32, "err_best"),
                        (err_init, torch.float32, "err_init")):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous() or t.numel() != groups:
            raise ValueError(f"{name} must be a contiguous {dt} CUDA tensor with one entry per group")
    K = int(down) + int(up) + 1
    dev = shift.device
    # counts are uint64 in the C ABI; int64 holds them (< 2^63) with full torch support
    out = dict(count=torch.empty(K, dtype=torch.int64, device=dev),
               sum_init=torch.empty(K, dtype=torch.float64, device=dev),
               sum_best=torch.empty(K, dtype=torch.float64, device=dev),
               sum_rel=torch.empty(K, dtype=torch.float64, device=dev))
    need = _lib.hscale_shift_summary_workspace_bytes(groups, int(down), int(up))
    ws = torch.empty(max(need, 8), dtype=torch.uint8, device=dev)
    st = _lib.hscale_shift_summary(shift.data_ptr(), err_best.data_ptr(), err_init.data_ptr(), groups, int(down),
                                   int(up), out["count"].data_ptr(), out["sum_init"].data_ptr(),
                                   out["sum_best"].data_ptr(), out["sum_rel"].data_ptr(), ws.data_ptr(), need,
                                   _stream(stream))
    _check(st, "hscale_shift_summary")
    return out


def output_error_workspace_bytes(tokens: int, in_features: int, out_features: int) -> int:
    """Bytes of scratch output_error needs."""
    return _lib.hscale_output_error_workspace_bytes(tokens, in_features, out_features)


def output_error(X: torch.Tensor, W: torch.Tensor, global_scale: float, scale_codes: torch.Tensor,
                 packed_e2m1: torch.Tensor, row_err: torch.Tensor | None = None,
                 workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Eq. 3 per output row: row_err[r] += sum_t (X dW^T)_tr^2 with dW = W - W^
    the rounding error of the stored NVFP4 tensor (scale_codes, packed_e2m1).
    row_err is fp64 [out] (zeros when not given); the layer's L_full is its
    sum."""
    _bf16_matrix(X, "X")
    _bf16_matrix(W, "W")
    T, n = X.shape
    m = W.shape[0]
    if W.shape[1] != n:
        raise ValueError("X and W disagree on in_features")
    if scale_codes.dtype != torch.uint8 or scale_codes.shape != (m, n // 16) or not scale_codes.is_contiguous():
        raise ValueError("scale_codes must be a contiguous uint8 tensor [out, in/16]")
    if packed_e2m1.dtype != torch.uint8 or packed_e2m1.shape != (m, n // 2) or not packed_e2m1.is_contiguous():
        raise ValueError("packed_e2m1 must be a contiguous uint8 tensor [out, in/2]")
    if row_err is None:
        row_err = torch.zeros(m, dtype=torch.float64, device=X.device)
    if row_err.dtype != torch.float64 or row_err.shape != (m,) or not row_err.is_contiguous():
        raise ValueError("row_err must be a contiguous fp64 tensor [out]")
    need = output_error_workspace_bytes(T, n, m)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.hscale_output_error(X.data_ptr(), T, n, W.data_ptr(), m, float(global_scale),
                                    scale_codes.data_ptr(), packed_e2m1.data_ptr(), row_err.data_ptr(), ws_ptr,
                                    ws_bytes, _stream(stream)), "hscale_output_error")
    return row_err
