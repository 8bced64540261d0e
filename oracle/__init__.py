"""CPU reference oracle for the H-Scale hot path (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  The product path (the HIP library
under ``paper_2608_28113_amd``) never imports or links it, and the two share
no code: the oracle is plain C (``hscale_oracle.c``) compiled with gcc, scoring
in fp64, written step by step from the paper's Sec. 3 (Eq. 1-2, 4, 6-13) and
its App. B algorithm HScaleGroupQuantize.

This module only marshals numpy arrays to the C functions and back.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_DIR = Path(__file__).resolve().parent
_SRC = _DIR / "hscale_oracle.c"
_LIB_PATH = _DIR / "liboracle.so"
# A planted-mistake (mutant) build of the oracle can be loaded instead, so the
# CPU tests can show that their pins catch it.
_LIB_OVERRIDE = os.environ.get("HSCALE_ORACLE_LIB")

M_CODES = 126  # positive finite E4M3FN codes 1..126
NEAR_TIE_REL = 1e-6  # near-tie band for parity reports (relative gap)

_lib = None


def build(force: bool = True) -> Path:
    """Compile the oracle with gcc (strict IEEE: no fast-math, no contraction)."""
    if force or not _LIB_PATH.exists():
        tmp = _LIB_PATH.with_suffix(".so.tmp%d" % os.getpid())
        cmd = [
            "gcc", "-O2", "-std=c11", "-fPIC", "-shared",
            "-fno-fast-math", "-ffp-contract=off", "-fno-strict-aliasing",
            "-Wall", "-Wextra", "-o", str(tmp), str(_SRC), "-lm",
        ]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if _LIB_OVERRIDE:
        lib = ctypes.CDLL(_LIB_OVERRIDE)
    else:
        if not _LIB_PATH.exists():
            build(force=False)
        lib = ctypes.CDLL(str(_LIB_PATH))
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_e4m3_value.argtypes = [ctypes.c_int]
    lib.oracle_e4m3_value.restype = ctypes.c_double
    lib.oracle_e4m3_round.argtypes = [ctypes.c_double]
    lib.oracle_e4m3_round.restype = ctypes.c_int
    lib.oracle_e2m1_index.argtypes = [ctypes.c_double]
    lib.oracle_e2m1_index.restype = ctypes.c_int
    lib.oracle_e2m1_value.argtypes = [ctypes.c_int]
    lib.oracle_e2m1_value.restype = ctypes.c_double
    lib.oracle_scale_tables.argtypes = [ctypes.c_float, P, P]
    lib.oracle_scale_tables.restype = None
    lib.oracle_hdiag.argtypes = [P, i64, i64, P]
    lib.oracle_hdiag.restype = None
    lib.oracle_search.argtypes = [P, i64, i64, P, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_float, P, P, P, P, P]
    lib.oracle_search.restype = ctypes.c_int
    lib.oracle_search_init.argtypes = [P, i64, i64, P, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                       ctypes.c_int, P, P, P, P, P, P, P, P]
    lib.oracle_search_init.restype = ctypes.c_int
    lib.oracle_search_stats.argtypes = [P, i64, i64, P, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                        ctypes.c_int, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_search_stats.restype = ctypes.c_int
    lib.oracle_anchor_codes.argtypes = [P, i64, i64, ctypes.c_float, ctypes.c_double, P]
    lib.oracle_anchor_codes.restype = ctypes.c_int
    lib.oracle_hdiag_accumulate.argtypes = [P, i64, i64, P]
    lib.oracle_hdiag_accumulate.restype = None
    lib.oracle_quantize.argtypes = [P, i64, i64, ctypes.c_float, P, P, P, P]
    lib.oracle_quantize.restype = ctypes.c_int
    lib.oracle_all_code_errors.argtypes = [P, i64, i64, P, ctypes.c_float, P]
    lib.oracle_all_code_errors.restype = ctypes.c_int
    lib.oracle_group_at_scale.argtypes = [P, P, ctypes.c_int, ctypes.c_float, P, P]
    lib.oracle_group_at_scale.restype = ctypes.c_double
    lib.oracle_group_search.argtypes = [P, P, ctypes.c_int, ctypes.c_float,
                                        ctypes.c_int, ctypes.c_int, P, P, P, P]
    lib.oracle_group_search.restype = ctypes.c_int
    lib.oracle_delta.argtypes = [P, i64, i64, ctypes.c_float, P, P, P]
    lib.oracle_delta.restype = ctypes.c_int
    lib.oracle_output_error.argtypes = [P, i64, i64, P, i64, P]
    lib.oracle_output_error.restype = ctypes.c_int
    lib.oracle_shift_summary.argtypes = [P, P, P, i64, ctypes.c_int, ctypes.c_int, P, P, P, P]
    lib.oracle_shift_summary.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _bf16_bits(a) -> np.ndarray:
    """Accepts a uint16 array of bf16 bit patterns (or a torch bf16 tensor)."""
    if hasattr(a, "dtype") and str(a.dtype) == "torch.bfloat16":
        import torch
        a = a.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 inputs are passed as uint16 bit patterns")
    return a


# --------------------------------------------------------------------------
# Formats
# --------------------------------------------------------------------------

def e4m3_value(c: int) -> float:
    """Value of the non-negative E4M3FN code byte c (0..126)."""
    return _load().oracle_e4m3_value(int(c))


def e4m3_round(t: float) -> int:
    """Q_fp8 (nearest, ties to even, saturating at 448) as a code byte."""
    return _load().oracle_e4m3_round(float(t))


def e2m1_index(x: float) -> int:
    """Nearest E2M1 magnitude index of x >= 0 (ties to even, clipped to 6)."""
    return _load().oracle_e2m1_index(float(x))


def e2m1_value(i: int) -> float:
    return _load().oracle_e2m1_value(int(i))


def scale_tables(s_g: float):
    """(S, R) fp32 arrays of length 127; S[c] = fp32(s_g * l_c), R = fp32(1/S)."""
    S = np.zeros(M_CODES + 1, np.float32)
    R = np.zeros(M_CODES + 1, np.float32)
    _load().oracle_scale_tables(np.float32(s_g), _ptr(S), _ptr(R))
    return S, R


# --------------------------------------------------------------------------
# Matrix-level
# --------------------------------------------------------------------------

def hdiag(X) -> np.ndarray:
    """Eq. 4: h_j = sum_t X[t, j]^2 in fp64. X: [tokens, n] bf16 bits."""
    X = _bf16_bits(X)
    T, n = X.shape
    h = np.zeros(n, np.float64)
    _load().oracle_hdiag(_ptr(X), T, n, _ptr(h))
    return h


INIT_RTN, INIT_4OVER6, INIT_GIVEN = 0, 1, 2


def search(W, h, s_g: float, window: int | None = None, down: int | None = None,
           up: int | None = None, init="rtn") -> dict:
    """The windowed scale search over a [m, n] bf16 matrix.

    Either ``window`` (symmetric, shifts -window..+window) or ``down``/``up``.
    ``init`` is "rtn" (max-abs, Eq. 7), "4over6" (the better of max/4 and
    max/6 under plain MSE), or a uint8 array [m, n/16] of initial codes.
    Returns codes [m, n/16] u8, packed [m, n/2] u8, e_best / e_second
    [m, n/16] f64, c0 [m, n/16] u8 (the initial codes), shift [m, n/16] i8
    (the chosen shift d*), e_init [m, n/16] f64 (the error at d = 0) and,
    for "4over6", l4 / l6 [m, n/16] f64 (the two anchors' plain squared
    errors).
    """
    if window is not None:
        down = up = int(window)
    W = _bf16_bits(W)
    m, n = W.shape
    h = np.ascontiguousarray(h, dtype=np.float32)
    assert h.shape == (n,)
    G = n // 16
    init_codes = None
    if isinstance(init, str):
        mode = {"rtn": INIT_RTN, "4over6": INIT_4OVER6}[init]
    else:
        mode = INIT_GIVEN
        init_codes = np.ascontiguousarray(init, dtype=np.uint8)
        assert init_codes.shape == (m, G)
    codes = np.zeros((m, G), np.uint8)
    packed = np.zeros((m, n // 2), np.uint8)
    e_best = np.zeros((m, G), np.float64)
    e_second = np.zeros((m, G), np.float64)
    c0 = np.zeros((m, G), np.uint8)
    l4 = np.zeros((m, G), np.float64)
    l6 = np.zeros((m, G), np.float64)
    shift = np.zeros((m, G), np.int8)
    e_init = np.zeros((m, G), np.float64)
    rc = _load().oracle_search_stats(_ptr(W), m, n, _ptr(h), int(down), int(up),
                                     np.float32(s_g), mode, _ptr(init_codes), _ptr(codes),
                                     _ptr(packed), _ptr(e_best), _ptr(e_second), _ptr(c0),
                                     _ptr(l4), _ptr(l6), _ptr(shift), _ptr(e_init))
    if rc != 0:
        raise ValueError("oracle_search_stats: bad arguments")
    out = dict(codes=codes, packed=packed, e_best=e_best, e_second=e_second, c0=c0,
               shift=shift, e_init=e_init)
    if mode == INIT_4OVER6:
        out.update(l4=l4, l6=l6)
    return out


def anchor_codes(W, s_g: float, anchor: float) -> np.ndarray:
    """Eq. 7's initial code with a general anchor (6: max-abs; 4 and 6: the
    4over6 candidates).  [m, n/16] u8."""
    W = _bf16_bits(W)
    m, n = W.shape
    out = np.zeros((m, n // 16), np.uint8)
    if _load().oracle_anchor_codes(_ptr(W), m, n, np.float32(s_g), float(anchor), _ptr(out)) != 0:
        raise ValueError("oracle_anchor_codes: bad arguments")
    return out


def hdiag_accumulate(X, h64: np.ndarray) -> np.ndarray:
    """h64 += sum_t X[t, :]^2 in place (fp64), for streamed calibration."""
    X = _bf16_bits(X)
    T, n = X.shape
    assert h64.dtype == np.float64 and h64.shape == (n,) and h64.flags["C_CONTIGUOUS"]
    _load().oracle_hdiag_accumulate(_ptr(X), T, n, _ptr(h64))
    return h64


def quantize(W, s_g: float, codes, h=None):
    """Quantize every group at the given scale codes. Returns (packed, err)."""
    W = _bf16_bits(W)
    m, n = W.shape
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    assert codes.shape == (m, n // 16)
    hh = None if h is None else np.ascontiguousarray(h, dtype=np.float32)
    packed = np.zeros((m, n // 2), np.uint8)
    err = np.zeros((m, n // 16), np.float64)
    rc = _load().oracle_quantize(_ptr(W), m, n, np.float32(s_g), _ptr(codes),
                                 _ptr(hh), _ptr(packed), _ptr(err))
    if rc != 0:
        raise ValueError("oracle_quantize: bad arguments")
    return packed, err


def all_code_errors(W, h, s_g: float) -> np.ndarray:
    """Eq. 13 error of every group at every code 1..126: [m, n/16, 126]."""
    W = _bf16_bits(W)
    m, n = W.shape
    h = np.ascontiguousarray(h, dtype=np.float32)
    err = np.zeros((m, n // 16, M_CODES), np.float64)
    rc = _load().oracle_all_code_errors(_ptr(W), m, n, _ptr(h), np.float32(s_g), _ptr(err))
    if rc != 0:
        raise ValueError("oracle_all_code_errors: bad arguments")
    return err


def group_at_scale(w, S: float, h=None):
    """Quantize one fp64 group at fp32 scale S. Returns (err, nibbles, w_hat)."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    g = w.shape[0]
    hh = None if h is None else np.ascontiguousarray(h, dtype=np.float64)
    nib = np.zeros(g, np.uint8)
    what = np.zeros(g, np.float64)
    e = _load().oracle_group_at_scale(_ptr(w), _ptr(hh), g, np.float32(S), _ptr(nib), _ptr(what))
    return e, nib, what


def group_search(w, h, s_g: float, down: int, up: int):
    """Windowed search on one fp64 group; exposes every candidate."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    g = w.shape[0]
    h = np.ascontiguousarray(h, dtype=np.float64)
    K = down + up + 1
    nib = np.zeros(g, np.uint8)
    cc = np.zeros(K, np.int32)
    ce = np.zeros(K, np.float64)
    c0 = np.zeros(1, np.int32)
    c = _load().oracle_group_search(_ptr(w), _ptr(h), g, np.float32(s_g), down, up,
                                    _ptr(nib), _ptr(cc), _ptr(ce), _ptr(c0))
    if c < 0:
        raise ValueError("oracle_group_search: bad arguments")
    return dict(code=c, nibbles=nib, cand_codes=cc, cand_err=ce, c0=int(c0[0]))


# --------------------------------------------------------------------------
# Parity classification (reporting aid)
# --------------------------------------------------------------------------

def near_tie_mask(e_best: np.ndarray, e_second: np.ndarray, rel: float = NEAR_TIE_REL):
    """Groups whose best and second-best distinct-code errors are within
    ``rel`` (relative to the second); two zero errors count as a tie.  A
    window with a single distinct code (window 0, or every candidate clipped
    to one end of the ladder) has no second-best (+inf) and no tie."""
    e_second = np.asarray(e_second, np.float64)
    return np.isfinite(e_second) & ((e_second - e_best) <= rel * e_second)


def pack_nibbles(nib: np.ndarray) -> np.ndarray:
    """[..., 2k] nibble arrays -> bytes, element 2k in the low nibble."""
    nib = np.asarray(nib, np.uint8)
    return (nib[..., 0::2] | (nib[..., 1::2] << 4)).astype(np.uint8)


def unpack_nibbles(packed: np.ndarray) -> np.ndarray:
    packed = np.asarray(packed, np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), np.uint8)
    out[..., 0::2] = packed & 0xF
    out[..., 1::2] = packed >> 4
    return out


def delta(W, s_g: float, codes, packed) -> np.ndarray:
    """Rounding error W - W^ of a stored NVFP4 tensor, fp64 [m, n]."""
    W = _bf16_bits(W)
    m, n = W.shape
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    assert codes.shape == (m, n // 16) and packed.shape == (m, n // 2)
    out = np.zeros((m, n), np.float64)
    if _load().oracle_delta(_ptr(W), m, n, np.float32(s_g), _ptr(codes), _ptr(packed), _ptr(out)) != 0:
        raise ValueError("oracle_delta: bad arguments")
    return out


def output_error(X, dW, row_err: np.ndarray | None = None) -> np.ndarray:
    """Eq. 3 per output row: row_err[r] += sum_t (X dW^T)_tr^2 (fp64 [m])."""
    X = _bf16_bits(X)
    T, n = X.shape
    dW = np.ascontiguousarray(dW, dtype=np.float64)
    m = dW.shape[0]
    assert dW.shape == (m, n)
    if row_err is None:
        row_err = np.zeros(m, np.float64)
    assert row_err.dtype == np.float64 and row_err.shape == (m,) and row_err.flags["C_CONTIGUOUS"]
    if _load().oracle_output_error(_ptr(X), T, n, _ptr(dW), m, _ptr(row_err)) != 0:
        raise ValueError("oracle_output_error: bad arguments")
    return row_err


def shift_summary(shift, e_best, e_init, down: int, up: int) -> dict:
    """Per-shift counts, sums of initial / chosen errors and of relative
    reductions (bins d = -down..up)."""
    shift = np.ascontiguousarray(shift, dtype=np.int8).ravel()
    e_best = np.ascontiguousarray(e_best, dtype=np.float64).ravel()
    e_init = np.ascontiguousarray(e_init, dtype=np.float64).ravel()
    K = down + up + 1
    count = np.zeros(K, np.int64)
    si, sb, sr = (np.zeros(K, np.float64) for _ in range(3))
    rc = _load().oracle_shift_summary(_ptr(shift), _ptr(e_best), _ptr(e_init), shift.size, int(down), int(up),
                                      _ptr(count), _ptr(si), _ptr(sb), _ptr(sr))
    if rc != 0:
        raise ValueError("oracle_shift_summary: bad arguments")
    return dict(count=count, sum_init=si, sum_best=sb, sum_rel=sr)
