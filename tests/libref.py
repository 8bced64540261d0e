"""Library-built formulations used to pin the oracle in the CPU tests.

These are not a second copy of the oracle: each quantity is formed from a
different building block than the one the oracle uses.

* E4M3 ladder and Q_fp8: torch's float8_e4m3fn decode and cast (the oracle
  decodes bit fields and rounds by nearest-value search).
* E2M1 Round/Clip: numpy's round-half-to-even on x / q, where q is the grid
  spacing of x's binade (0.5 below 2, 1 below 4, 2 above), then min(., 6)
  (the oracle searches the eight grid values).
* fp32 rounding points: numpy float32 arithmetic, which is IEEE
  round-to-nearest-even (the oracle rounds fp64 results to fp32).
* Scoring: vectorised numpy over all groups and candidates at once.
"""
from __future__ import annotations

import numpy as np

E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def ladder() -> np.ndarray:
    """float64 [127]: index c -> value of E4M3FN byte c (0..126), via torch."""
    import torch
    v = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy()
    return v[:127].astype(np.float64)


def e4m3_cast_codes(t: np.ndarray) -> np.ndarray:
    """torch's fp32 -> float8_e4m3fn cast as code bytes, saturating past 448
    (torch itself returns NaN above 464)."""
    import torch
    t = np.asarray(t, np.float32)
    c = torch.from_numpy(t.copy()).to(torch.float8_e4m3fn).view(torch.uint8).numpy().astype(np.int64)
    return np.where(t > 448.0, 126, c)


def e2m1_round_index(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    q = np.where(x < 2.0, 0.5, np.where(x < 4.0, 1.0, 2.0))
    v = np.minimum(np.round(x / q) * q, 6.0)
    return np.searchsorted(E2M1_GRID, v).astype(np.int64)


def weights_f32(W_bits: np.ndarray) -> np.ndarray:
    return (np.asarray(W_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def rtn_codes(W_bits: np.ndarray, s_g: float, anchor: float = 6.0) -> np.ndarray:
    """Max-abs initial code per group: fp32(max|w| / anchor), fp32(. / s_g),
    torch's E4M3 cast, then at least code 1.  [m, n/16] int64."""
    w = weights_f32(W_bits)
    m, n = w.shape
    amax = np.abs(w).reshape(m, n // 16, 16).max(axis=-1).astype(np.float32)
    s_init = (amax / np.float32(anchor)).astype(np.float32)
    t = (s_init / np.float32(s_g)).astype(np.float32)
    return np.maximum(e4m3_cast_codes(t), 1)


def quantize_at(W_bits: np.ndarray, s_g: float, codes: np.ndarray, h=None):
    """Quantize every group at its code.  Returns (nibbles [m, n], err [m, G])."""
    w = weights_f32(W_bits)
    m, n = w.shape
    G = n // 16
    lam = ladder().astype(np.float32)[np.asarray(codes, np.int64)]  # [m, G]
    S = (np.float32(s_g) * lam).astype(np.float32)
    R = (np.float32(1.0) / S).astype(np.float32)
    wg = w.reshape(m, G, 16)
    x = (np.abs(wg) * R[..., None]).astype(np.float32)
    idx = e2m1_round_index(x)
    neg = np.signbit(wg)
    q = E2M1_GRID[idx] * S[..., None].astype(np.float64)
    q = np.where(neg, -q, q)
    d = wg.astype(np.float64) - q
    hh = np.ones(n) if h is None else np.asarray(h, np.float64)
    err = (hh.reshape(1, G, 16) * d * d).sum(axis=-1)
    nib = (neg.astype(np.int64) << 3) | idx
    return nib.reshape(m, n).astype(np.uint8), err


def all_code_errors(W_bits: np.ndarray, h, s_g: float) -> np.ndarray:
    """err [m, G, 126] at every code 1..126."""
    w = weights_f32(W_bits)
    m, n = w.shape
    G = n // 16
    out = np.empty((m, G, 126))
    for c in range(1, 127):
        _, e = quantize_at(W_bits, s_g, np.full((m, G), c), h)
        out[:, :, c - 1] = e
    return out


def windowed_search(W_bits: np.ndarray, h, s_g: float, down: int, up: int):
    """Vectorised windowed search: codes [m, G], nibbles [m, n]."""
    w = weights_f32(W_bits)
    m, n = w.shape
    G = n // 16
    c0 = rtn_codes(W_bits, s_g)
    best_e = None
    best_c = None
    for d in range(-down, up + 1):
        c = np.clip(c0 + d, 1, 126)
        _, e = quantize_at(W_bits, s_g, c, h)
        if best_e is None:
            best_e, best_c = e, c
        else:
            better = e < best_e
            best_e = np.where(better, e, best_e)
            best_c = np.where(better, c, best_c)
    nib, _ = quantize_at(W_bits, s_g, best_c, h)
    return best_c, nib, best_e


def four_over_six_codes(W_bits: np.ndarray, s_g: float) -> np.ndarray:
    """4over6 initial code per group: the anchor (4 or 6) whose max-abs code
    gives the smaller plain squared error, anchor 4 on a tie."""
    c4 = rtn_codes(W_bits, s_g, 4.0)
    c6 = rtn_codes(W_bits, s_g, 6.0)
    _, l4 = quantize_at(W_bits, s_g, c4)
    _, l6 = quantize_at(W_bits, s_g, c6)
    return np.where(l4 <= l6, c4, c6)
