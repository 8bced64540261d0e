"""ctypes binding of libhscale.so (include/hscale.h), same names as the C ABI.

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  There is no fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

LIB_PATH = Path(__file__).resolve().parent / "libhscale.so"

HSCALE_OK = 0
STATUS = {
    0: "HSCALE_OK", -1: "HSCALE_ERR_NULL", -2: "HSCALE_ERR_SHAPE", -3: "HSCALE_ERR_ALIGN",
    -4: "HSCALE_ERR_WINDOW", -5: "HSCALE_ERR_SCALE", -6: "HSCALE_ERR_WORKSPACE",
    -7: "HSCALE_ERR_HIP", -8: "HSCALE_ERR_OVERLAP", -9: "HSCALE_ERR_SCRATCH", -10: "HSCALE_ERR_DEVICE",
}

# Every symbol include/hscale.h declares.
EXPORTS = (
    "hscale_status_string",
    "hscale_hdiag_workspace_bytes",
    "hscale_hdiag",
    "hscale_hdiag_noalloc",
    "hscale_hdiag_accumulate",
    "hscale_hdiag_finalize",
    "hscale_search",
    "hscale_search_du",
    "hscale_search_4over6",
    "hscale_search_from",
    "hscale_search_block",
    "hscale_search_layers",
    "hscale_search_stats",
    "hscale_shift_summary_workspace_bytes",
    "hscale_shift_summary",
    "hscale_output_error_workspace_bytes",
    "hscale_output_error",
    "hscale_quantize",
)

HSCALE_INIT_MAXABS, HSCALE_INIT_4OVER6, HSCALE_INIT_GIVEN = 0, 1, 2


class HScaleLayer(ctypes.Structure):
    """struct hscale_layer of include/hscale.h (natural C layout)."""
    _fields_ = [("W", ctypes.c_void_p), ("out", ctypes.c_int64), ("in_", ctypes.c_int64),
                ("h", ctypes.c_void_p), ("global_scale", ctypes.c_float), ("init_codes", ctypes.c_void_p),
                ("scale_codes", ctypes.c_void_p), ("packed_e2m1", ctypes.c_void_p)]

_lib = None


class HScaleError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not LIB_PATH.exists():
        raise ImportError(
            f"{LIB_PATH} is not built; run paper_2608_28113_amd/build.py "
            "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(str(LIB_PATH))
    P, i64, i32, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    lib.hscale_status_string.argtypes = [ctypes.c_int]
    lib.hscale_status_string.restype = ctypes.c_char_p
    lib.hscale_hdiag_workspace_bytes.argtypes = [i64, i64]
    lib.hscale_hdiag_workspace_bytes.restype = sz
    lib.hscale_hdiag.argtypes = [P, i64, i64, P, P, sz, P]
    lib.hscale_hdiag.restype = ctypes.c_int
    lib.hscale_hdiag_noalloc.argtypes = [P, i64, i64, P, P]
    lib.hscale_hdiag_noalloc.restype = ctypes.c_int
    lib.hscale_search.argtypes = [P, i64, i64, P, i32, f32, P, P, P]
    lib.hscale_search.restype = ctypes.c_int
    lib.hscale_search_du.argtypes = [P, i64, i64, P, i32, i32, f32, P, P, P]
    lib.hscale_search_du.restype = ctypes.c_int
    lib.hscale_quantize.argtypes = [P, i64, i64, f32, P, P, P]
    lib.hscale_quantize.restype = ctypes.c_int
    lib.hscale_hdiag_accumulate.argtypes = [P, i64, i64, P, P, sz, P]
    lib.hscale_hdiag_accumulate.restype = ctypes.c_int
    lib.hscale_hdiag_finalize.argtypes = [P, i64, P, P]
    lib.hscale_hdiag_finalize.restype = ctypes.c_int
    lib.hscale_search_4over6.argtypes = [P, i64, i64, P, i32, i32, f32, P, P, P]
    lib.hscale_search_4over6.restype = ctypes.c_int
    lib.hscale_search_from.argtypes = [P, i64, i64, P, i32, i32, f32, P, P, P, P]
    lib.hscale_search_from.restype = ctypes.c_int
    lib.hscale_search_block.argtypes = [P, i64, i64, i64, P, i32, i32, f32, i32, P, i64, P, i64, P, i64, P]
    lib.hscale_search_block.restype = ctypes.c_int
    lib.hscale_search_layers.argtypes = [ctypes.POINTER(HScaleLayer), i32, i32, i32, i32, P]
    lib.hscale_search_layers.restype = ctypes.c_int
    lib.hscale_search_stats.argtypes = [P, i64, i64, P, i32, i32, f32, i32, P, P, P, P, P, P, P]
    lib.hscale_search_stats.restype = ctypes.c_int
    lib.hscale_shift_summary_workspace_bytes.argtypes = [i64, i32, i32]
    lib.hscale_shift_summary_workspace_bytes.restype = sz
    lib.hscale_shift_summary.argtypes = [P, P, P, i64, i32, i32, P, P, P, P, P, sz, P]
    lib.hscale_shift_summary.restype = ctypes.c_int
    lib.hscale_output_error_workspace_bytes.argtypes = [i64, i64, i64]
    lib.hscale_output_error_workspace_bytes.restype = sz
    lib.hscale_output_error.argtypes = [P, i64, i64, P, i64, f32, P, P, P, P, sz, P]
    lib.hscale_output_error.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().hscale_status_string(int(status)).decode()


def hscale_hdiag_workspace_bytes(tokens: int, in_: int) -> int:
    return int(load().hscale_hdiag_workspace_bytes(int(tokens), int(in_)))


def hscale_hdiag(X: int, tokens: int, in_: int, h: int, workspace: int, workspace_bytes: int,
                 stream: int) -> int:
    return load().hscale_hdiag(X or None, tokens, in_, h or None, workspace or None,
                               workspace_bytes, stream or None)


def hscale_hdiag_noalloc(X: int, tokens: int, in_: int, h: int, stream: int) -> int:
    return load().hscale_hdiag_noalloc(X or None, tokens, in_, h or None, stream or None)


def hscale_search(W: int, out: int, in_: int, h: int, window: int, global_scale: float,
                  scale_codes: int, packed_e2m1: int, stream: int) -> int:
    return load().hscale_search(W or None, out, in_, h or None, window, global_scale,
                                scale_codes or None, packed_e2m1 or None, stream or None)


def hscale_search_du(W: int, out: int, in_: int, h: int, down: int, up: int, global_scale: float,
                     scale_codes: int, packed_e2m1: int, stream: int) -> int:
    return load().hscale_search_du(W or None, out, in_, h or None, down, up, global_scale,
                                   scale_codes or None, packed_e2m1 or None, stream or None)


def hscale_quantize(W: int, out: int, in_: int, global_scale: float, scale_codes: int,
                    packed_e2m1: int, stream: int) -> int:
    return load().hscale_quantize(W or None, out, in_, global_scale, scale_codes or None,
                                  packed_e2m1 or None, stream or None)


def hscale_hdiag_accumulate(X: int, tokens: int, in_: int, h64: int, workspace: int,
                            workspace_bytes: int, stream: int) -> int:
    return load().hscale_hdiag_accumulate(X or None, tokens, in_, h64 or None, workspace or None,
                                          workspace_bytes, stream or None)


def hscale_hdiag_finalize(h64: int, in_: int, h: int, stream: int) -> int:
    return load().hscale_hdiag_finalize(h64 or None, in_, h or None, stream or None)


def hscale_search_4over6(W: int, out: int, in_: int, h: int, down: int, up: int, global_scale: float,
                         scale_codes: int, packed_e2m1: int, stream: int) -> int:
    return load().hscale_search_4over6(W or None, out, in_, h or None, down, up, global_scale,
                                       scale_codes or None, packed_e2m1 or None, stream or None)


def hscale_search_from(W: int, out: int, in_: int, h: int, down: int, up: int, global_scale: float,
                       init_codes: int, scale_codes: int, packed_e2m1: int, stream: int) -> int:
    return load().hscale_search_from(W or None, out, in_, h or None, down, up, global_scale,
                                     init_codes or None, scale_codes or None, packed_e2m1 or None,
                                     stream or None)


def hscale_search_block(W: int, ldw: int, out: int, cols: int, h: int, down: int, up: int,
                        global_scale: float, init_mode: int, init_codes: int, ldi: int, scale_codes: int,
                        ldc: int, packed_e2m1: int, ldp: int, stream: int) -> int:
    return load().hscale_search_block(W or None, ldw, out, cols, h or None, down, up, global_scale,
                                      init_mode, init_codes or None, ldi, scale_codes or None, ldc,
                                      packed_e2m1 or None, ldp, stream or None)


def hscale_search_layers(layers, down: int, up: int, init_mode: int, stream: int) -> int:
    """layers: sequence of (W, out, in, h, global_scale, init_codes, scale_codes, packed_e2m1)
    with device addresses as ints (0 for NULL)."""
    arr = (HScaleLayer * max(len(layers), 1))()
    for k, (W, out, in_, h, s_g, init, codes, packed) in enumerate(layers):
        arr[k] = HScaleLayer(W or None, out, in_, h or None, s_g, init or None, codes or None, packed or None)
    return load().hscale_search_layers(arr if layers else None, len(layers), down, up, init_mode, stream or None)


def hscale_search_stats(W: int, out: int, in_: int, h: int, down: int, up: int, global_scale: float,
                        init_mode: int, init_codes: int, scale_codes: int, packed_e2m1: int, shift: int,
                        err_best: int, err_init: int, stream: int) -> int:
    return load().hscale_search_stats(W or None, out, in_, h or None, down, up, global_scale, init_mode,
                                      init_codes or None, scale_codes or None, packed_e2m1 or None,
                                      shift or None, err_best or None, err_init or None, stream or None)


def hscale_shift_summary_workspace_bytes(groups: int, down: int, up: int) -> int:
    return load().hscale_shift_summary_workspace_bytes(groups, down, up)


def hscale_shift_summary(shift: int, err_best: int, err_init: int, groups: int, down: int, up: int,
                         count: int, sum_init: int, sum_best: int, sum_rel: int, workspace: int,
                         workspace_bytes: int, stream: int) -> int:
    return load().hscale_shift_summary(shift or None, err_best or None, err_init or None, groups, down, up,
                                       count or None, sum_init or None, sum_best or None, sum_rel or None,
                                       workspace or None, workspace_bytes, stream or None)


def hscale_output_error_workspace_bytes(tokens: int, in_: int, out: int) -> int:
    return load().hscale_output_error_workspace_bytes(tokens, in_, out)


def hscale_output_error(X: int, tokens: int, in_: int, W: int, out: int, global_scale: float, scale_codes: int,
                        packed_e2m1: int, row_err: int, workspace: int, workspace_bytes: int, stream: int) -> int:
    return load().hscale_output_error(X or None, tokens, in_, W or None, out, global_scale, scale_codes or None,
                                      packed_e2m1 or None, row_err or None, workspace or None, workspace_bytes,
                                      stream or None)
