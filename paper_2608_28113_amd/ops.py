"""Torch-tensor front end of the C ABI.

PyTorch supplies device memory and the current stream; these functions only
check tensor metadata, allocate outputs and pass raw pointers to
libhscale.so.  All arithmetic happens in the library's HIP kernels.

The C ABI cannot see buffer sizes or devices, so every tensor handed to it
here (inputs, caller-provided outputs and workspaces) is checked for dtype,
shape, contiguity and device first: a wrong buffer raises ValueError and
nothing is launched.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import HScaleError


def _check(status: int, where: str) -> None:
    if status != _lib.HSCALE_OK:
        raise HScaleError(status, where)


def _stream(stream, device) -> int:
    """Handle of `stream`, or of `device`'s current stream when None.  A
    torch stream must belong to `device`, the device the operands are on."""
    if stream is None:
        stream = torch.cuda.current_stream(device)
    elif isinstance(stream, torch.cuda.Stream) and stream.device != device:
        raise ValueError(f"stream is on {stream.device}, the operands on {device}")
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _call(device, fn, *args) -> int:
    """Calls the library with `device` current, so that its launches go to
    the device that holds the operands."""
    with torch.cuda.device(device):
        return fn(*args)


def _on_device(t) -> bool:
    """t is a tensor in GPU memory (the only memory the kernels may touch)."""
    return isinstance(t, torch.Tensor) and t.is_cuda


def _bf16_matrix(t, name: str) -> None:
    if (not _on_device(t) or t.dtype != torch.bfloat16 or t.dim() != 2 or not t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous 2-D bf16 CUDA tensor")


def _tensor(t, name: str, dtype, shape, device) -> torch.Tensor:
    """t must be a contiguous tensor of this dtype and shape on `device`."""
    if (not isinstance(t, torch.Tensor) or t.dtype != dtype or tuple(t.shape) != tuple(shape)
            or t.device != device or not t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")
    return t


def _out(t, name: str, dtype, shape, device) -> torch.Tensor:
    """A caller-provided output (checked) or a new one."""
    if t is None:
        return torch.empty(tuple(shape), dtype=dtype, device=device)
    return _tensor(t, name, dtype, shape, device)


def _workspace(ws, need: int, device) -> tuple[int, int]:
    """(pointer, bytes) of a caller-provided scratch tensor (any dtype,
    contiguous, on `device`) or of a new one; the library checks the size."""
    if ws is None:
        if need <= 0:
            return 0, 0
        ws = torch.empty(need, dtype=torch.uint8, device=device)
    elif not isinstance(ws, torch.Tensor) or ws.device != device or not ws.is_contiguous():
        raise ValueError(f"workspace must be a contiguous tensor on {device}")
    return ws.data_ptr(), ws.numel() * ws.element_size()


def _row_view(t, dtype, shape, device, name: str) -> int:
    """A 2-D view with unit column stride; returns its row stride."""
    if (not isinstance(t, torch.Tensor) or t.dtype != dtype or t.dim() != 2 or tuple(t.shape) != tuple(shape)
            or t.device != device or (t.shape[1] > 1 and t.stride(1) != 1)):
        raise ValueError(f"{name} must be a 2-D {dtype} view of shape {tuple(shape)} on {device} "
                         "with unit column stride")
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def _init_mode(init, shape, device):
    """(init_mode, initial-code tensor or None) of an `init` argument."""
    if isinstance(init, str):
        modes = {"maxabs": _lib.HSCALE_INIT_MAXABS, "rtn": _lib.HSCALE_INIT_MAXABS,
                 "4over6": _lib.HSCALE_INIT_4OVER6}
        if init not in modes:
            raise ValueError("init must be 'maxabs', '4over6' or a uint8 tensor of codes")
        return modes[init], None
    if isinstance(init, torch.Tensor):
        return _lib.HSCALE_INIT_GIVEN, _tensor(init, "initial codes", torch.uint8, shape, device)
    raise ValueError("init must be 'maxabs', '4over6' or a uint8 tensor of codes")


def _window(window, down, up) -> tuple[int, int]:
    if window is not None:
        if down is not None or up is not None:
            raise ValueError("give either window or down/up")
        return int(window), int(window)
    if down is None or up is None:
        raise ValueError("give window or both down and up")
    return int(down), int(up)


def hdiag_workspace_bytes(tokens: int, in_features: int) -> int:
    """Bytes of scratch hdiag needs for a [tokens, in_features] X."""
    return _lib.hscale_hdiag_workspace_bytes(tokens, in_features)


def hdiag(X: torch.Tensor, h: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
          stream=None) -> torch.Tensor:
    """h = diag(X^T X) (Sec. 3.2, Eq. 4) of bf16 X [tokens, in] as fp32 [in]."""
    _bf16_matrix(X, "X")
    T, n = X.shape
    dev = X.device
    h = _out(h, "h", torch.float32, (n,), dev)
    ws_ptr, ws_bytes = _workspace(workspace, hdiag_workspace_bytes(T, n), dev)
    _check(_call(dev, _lib.hscale_hdiag, X.data_ptr(), T, n, h.data_ptr(), ws_ptr, ws_bytes,
                 _stream(stream, dev)), "hscale_hdiag")
    return h


def hdiag_noalloc(X: torch.Tensor, h: torch.Tensor, stream=None) -> torch.Tensor:
    """hdiag into a caller-provided fp32 h [in] with the library's static
    scratch instead of a workspace: the call allocates no device memory
    (problems up to 2^20 columns; calls that may overlap on one GPU race)."""
    _bf16_matrix(X, "X")
    T, n = X.shape
    dev = X.device
    _tensor(h, "h", torch.float32, (n,), dev)
    _check(_call(dev, _lib.hscale_hdiag_noalloc, X.data_ptr(), T, n, h.data_ptr(), _stream(stream, dev)),
           "hscale_hdiag_noalloc")
    return h


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
    dev = W.device
    _tensor(h, "h", torch.float32, (n,), dev)
    down, up = _window(window, down, up)
    mode, init_t = _init_mode(init, (m, n // 16), dev)
    scale_codes = _out(scale_codes, "scale_codes", torch.uint8, (m, n // 16), dev)
    packed_e2m1 = _out(packed_e2m1, "packed_e2m1", torch.uint8, (m, n // 2), dev)
    s = _stream(stream, dev)
    if mode == _lib.HSCALE_INIT_MAXABS:
        st = _call(dev, _lib.hscale_search_du, W.data_ptr(), m, n, h.data_ptr(), down, up, float(global_scale),
                   scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_du")
    elif mode == _lib.HSCALE_INIT_4OVER6:
        st = _call(dev, _lib.hscale_search_4over6, W.data_ptr(), m, n, h.data_ptr(), down, up, float(global_scale),
                   scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_4over6")
    else:
        st = _call(dev, _lib.hscale_search_from, W.data_ptr(), m, n, h.data_ptr(), down, up, float(global_scale),
                   init_t.data_ptr(), scale_codes.data_ptr(), packed_e2m1.data_ptr(), s)
        _check(st, "hscale_search_from")
    return scale_codes, packed_e2m1


def search_layers(layers, window: int | None = None, down: int | None = None, up: int | None = None,
                  init="maxabs", outputs=None, stream=None):
    """The search of several layers in one launch (per up to 32 layers):
    ``layers`` is a sequence of (W, h, global_scale), all on one device;
    ``init`` is "maxabs", "4over6" or a sequence of per-layer uint8 code
    tensors; ``outputs`` optionally a sequence of (scale_codes, packed_e2m1)
    to write.  Returns the list of (scale_codes, packed_e2m1), each equal to
    what ``search`` returns for that layer alone."""
    layers = list(layers)
    down, up = _window(window, down, up)
    if outputs is not None:
        outputs = list(outputs)
        if len(outputs) != len(layers):
            raise ValueError("give one (scale_codes, packed_e2m1) pair per layer")
    given = None
    if isinstance(init, str):
        mode, _ = _init_mode(init, None, None)
    else:
        given = list(init)
        if len(given) != len(layers):
            raise ValueError("give one initial-code tensor per layer")
        mode = _lib.HSCALE_INIT_GIVEN
    dev = None
    args, result = [], []
    for k, layer in enumerate(layers):
        if len(layer) != 3:
            raise ValueError("each layer is (W, h, global_scale)")
        W, h, s_g = layer
        _bf16_matrix(W, f"W of layer {k}")
        if dev is None:
            dev = W.device
        elif W.device != dev:
            raise ValueError("all layers must be on one device")
        m, n = W.shape
        _tensor(h, f"h of layer {k}", torch.float32, (n,), dev)
        codes, packed = (None, None) if outputs is None else outputs[k]
        codes = _out(codes, f"scale_codes of layer {k}", torch.uint8, (m, n // 16), dev)
        packed = _out(packed, f"packed_e2m1 of layer {k}", torch.uint8, (m, n // 2), dev)
        iptr = 0
        if given is not None:
            iptr = _tensor(given[k], f"initial codes of layer {k}", torch.uint8, (m, n // 16), dev).data_ptr()
        args.append((W.data_ptr(), m, n, h.data_ptr(), float(s_g), iptr, codes.data_ptr(), packed.data_ptr()))
        result.append((codes, packed))
    if not layers:
        return result
    _check(_call(dev, _lib.hscale_search_layers, args, down, up, mode, _stream(stream, dev)), "hscale_search_layers")
    return result


def search_block(W: torch.Tensor, h: torch.Tensor, global_scale: float, down: int, up: int,
                 scale_codes: torch.Tensor, packed_e2m1: torch.Tensor, init="maxabs", stream=None):
    """The search on a column block given as strided views: W = Wfull[:, a:b]
    (bf16), h = hfull[a:b], scale_codes = codes[:, a/16:b/16] and
    packed_e2m1 = packed[:, a/2:b/2] (uint8), as in the paper's GPTQ
    combination (App. B).  Outputs are written in place."""
    if not _on_device(W) or W.dim() != 2:
        raise ValueError("W must be a 2-D bf16 CUDA view")
    m, cols = W.shape
    dev = W.device
    ldw = _row_view(W, torch.bfloat16, (m, cols), dev, "W")
    ldc = _row_view(scale_codes, torch.uint8, (m, cols // 16), dev, "scale_codes")
    ldp = _row_view(packed_e2m1, torch.uint8, (m, cols // 2), dev, "packed_e2m1")
    _tensor(h, "h", torch.float32, (cols,), dev)
    if isinstance(init, torch.Tensor):
        ldi = _row_view(init, torch.uint8, (m, cols // 16), dev, "initial codes")
        mode, iptr = _lib.HSCALE_INIT_GIVEN, init.data_ptr()
    else:
        mode, _ = _init_mode(init, None, dev)
        iptr, ldi = 0, 0
    st = _call(dev, _lib.hscale_search_block, W.data_ptr(), ldw, m, cols, h.data_ptr(), int(down), int(up),
               float(global_scale), mode, iptr, ldi, scale_codes.data_ptr(), ldc, packed_e2m1.data_ptr(), ldp,
               _stream(stream, dev))
    _check(st, "hscale_search_block")
    return scale_codes, packed_e2m1


def hdiag_accumulate(X: torch.Tensor, h64: torch.Tensor, workspace: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """h64 += diag(X^T X) for one calibration batch (fp64 accumulator)."""
    _bf16_matrix(X, "X")
    T, n = X.shape
    dev = X.device
    _tensor(h64, "h64", torch.float64, (n,), dev)
    ws_ptr, ws_bytes = _workspace(workspace, hdiag_workspace_bytes(T, n), dev)
    _check(_call(dev, _lib.hscale_hdiag_accumulate, X.data_ptr(), T, n, h64.data_ptr(), ws_ptr, ws_bytes,
                 _stream(stream, dev)), "hscale_hdiag_accumulate")
    return h64


def hdiag_finalize(h64: torch.Tensor, h: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """h = fp32(h64)."""
    if not _on_device(h64) or h64.dim() != 1:
        raise ValueError("h64 must be a 1-D fp64 CUDA tensor")
    n = h64.shape[0]
    dev = h64.device
    _tensor(h64, "h64", torch.float64, (n,), dev)
    h = _out(h, "h", torch.float32, (n,), dev)
    _check(_call(dev, _lib.hscale_hdiag_finalize, h64.data_ptr(), n, h.data_ptr(),
                 _stream(stream, dev)), "hscale_hdiag_finalize")
    return h


def quantize(W: torch.Tensor, global_scale: float, scale_codes: torch.Tensor,
             packed_e2m1: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Packed E2M1 codes of W at the given scale codes (final re-quantization)."""
    _bf16_matrix(W, "W")
    m, n = W.shape
    dev = W.device
    _tensor(scale_codes, "scale_codes", torch.uint8, (m, n // 16), dev)
    packed_e2m1 = _out(packed_e2m1, "packed_e2m1", torch.uint8, (m, n // 2), dev)
    _check(_call(dev, _lib.hscale_quantize, W.data_ptr(), m, n, float(global_scale), scale_codes.data_ptr(),
                 packed_e2m1.data_ptr(), _stream(stream, dev)), "hscale_quantize")
    return packed_e2m1


def search_stats(W: torch.Tensor, h: torch.Tensor, global_scale: float, down: int, up: int, init="maxabs",
                 stream=None):
    """The search with per-group statistics.  Returns a dict of
    scale_codes, packed_e2m1, shift (int8 [out, in/16], the chosen shift),
    err_best and err_init (fp32 [out, in/16], the score at the chosen shift
    and at shift 0)."""
    _bf16_matrix(W, "W")
    m, n = W.shape
    dev = W.device
    _tensor(h, "h", torch.float32, (n,), dev)
    G = (m, n // 16)
    mode, init_t = _init_mode(init, G, dev)
    out = dict(scale_codes=torch.empty(G, dtype=torch.uint8, device=dev),
               packed_e2m1=torch.empty((m, n // 2), dtype=torch.uint8, device=dev),
               shift=torch.empty(G, dtype=torch.int8, device=dev),
               err_best=torch.empty(G, dtype=torch.float32, device=dev),
               err_init=torch.empty(G, dtype=torch.float32, device=dev))
    st = _call(dev, _lib.hscale_search_stats, W.data_ptr(), m, n, h.data_ptr(), int(down), int(up),
               float(global_scale), mode, init_t.data_ptr() if init_t is not None else 0,
               out["scale_codes"].data_ptr(), out["packed_e2m1"].data_ptr(), out["shift"].data_ptr(),
               out["err_best"].data_ptr(), out["err_init"].data_ptr(), _stream(stream, dev))
    _check(st, "hscale_search_stats")
    return out


def shift_summary(shift: torch.Tensor, err_best: torch.Tensor, err_init: torch.Tensor, down: int, up: int,
                  stream=None) -> dict:
    """Per-shift counts and fp64 sums of initial errors, chosen errors and
    relative reductions over the groups (bins d = -down..up), as tensors of
    length down + up + 1 on the device."""
    if not _on_device(shift):
        raise ValueError("shift must be an int8 CUDA tensor")
    groups = shift.numel()
    dev = shift.device
    for t, dt, name in ((shift, torch.int8, "shift"), (err_best, torch.float32, "err_best"),
                        (err_init, torch.float32, "err_init")):
        if (not isinstance(t, torch.Tensor) or t.dtype != dt or t.device != dev or not t.is_contiguous()
                or t.numel() != groups):
            raise ValueError(f"{name} must be a contiguous {dt} tensor on {dev} with one entry per group")
    K = int(down) + int(up) + 1
    # counts are uint64 in the C ABI; int64 holds them (< 2^63) with full torch support
    out = dict(count=torch.empty(K, dtype=torch.int64, device=dev),
               sum_init=torch.empty(K, dtype=torch.float64, device=dev),
               sum_best=torch.empty(K, dtype=torch.float64, device=dev),
               sum_rel=torch.empty(K, dtype=torch.float64, device=dev))
    need = _lib.hscale_shift_summary_workspace_bytes(groups, int(down), int(up))
    ws = torch.empty(max(need, 8), dtype=torch.uint8, device=dev)
    st = _call(dev, _lib.hscale_shift_summary, shift.data_ptr(), err_best.data_ptr(), err_init.data_ptr(), groups,
               int(down), int(up), out["count"].data_ptr(), out["sum_init"].data_ptr(), out["sum_best"].data_ptr(),
               out["sum_rel"].data_ptr(), ws.data_ptr(), need, _stream(stream, dev))
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
    dev = X.device
    if W.shape[1] != n or W.device != dev:
        raise ValueError("X and W must share in_features and device")
    _tensor(scale_codes, "scale_codes", torch.uint8, (m, n // 16), dev)
    _tensor(packed_e2m1, "packed_e2m1", torch.uint8, (m, n // 2), dev)
    if row_err is None:
        row_err = torch.zeros(m, dtype=torch.float64, device=dev)
    _tensor(row_err, "row_err", torch.float64, (m,), dev)
    ws_ptr, ws_bytes = _workspace(workspace, output_error_workspace_bytes(T, n, m), dev)
    _check(_call(dev, _lib.hscale_output_error, X.data_ptr(), T, n, W.data_ptr(), m, float(global_scale),
                 scale_codes.data_ptr(), packed_e2m1.data_ptr(), row_err.data_ptr(), ws_ptr, ws_bytes,
                 _stream(stream, dev)), "hscale_output_error")
    return row_err
