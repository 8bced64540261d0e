"""Comparison of the HIP path with the oracle (shared by the GPU tests,
smoke() and bench.py).

Bar, from the hot path's contract:
  * h within a relative 1e-5 of the fp64 oracle (exact zeros stay zero);
  * scale codes and packed E2M1 bytes bit-exact, given the same fp32 h, for
    every group that is not a near-tie (the oracle's best and second-best
    distinct-code errors within a relative 1e-6);
  * for every group, near-ties included: the GPU's code lies in the window,
    its packed bytes are exactly the oracle's quantization at that code, and
    its oracle error is within the near-tie band of the oracle's minimum.
"""
from __future__ import annotations

import numpy as np

import oracle

H_REL_TOL = 1e-5
TIE_REL = oracle.NEAR_TIE_REL


def oracle_h32(X_bits: np.ndarray) -> np.ndarray:
    """h for a search parity case, computed by the oracle from the seeded X
    and rounded to fp32; the HIP search and the oracle search both take it
    as input (no oracle input comes from the HIP path)."""
    return oracle.hdiag(X_bits).astype(np.float32)


def compare_h(h_gpu: np.ndarray, h_ref: np.ndarray) -> dict:
    h_gpu = np.asarray(h_gpu, np.float64)
    zero = h_ref == 0
    rel = np.abs(h_gpu - h_ref) / np.where(zero, 1.0, h_ref)
    return dict(max_rel=float(rel.max(initial=0.0)), zeros_exact=bool(np.all(h_gpu[zero] == 0)),
                ok=bool(rel.max(initial=0.0) <= H_REL_TOL and np.all(h_gpu[zero] == 0)))


def compare_search(W_bits: np.ndarray, h32: np.ndarray, s_g: float, down: int, up: int,
                   codes_gpu: np.ndarray, packed_gpu: np.ndarray, init="rtn", oracle_result=None) -> dict:
    """``init`` is "rtn" (max-abs), "4over6" or an array of initial codes.

    For 4over6, a group whose two anchors' plain errors are within the
    near-tie band (and whose anchor codes differ) may start from either
    anchor: its result is checked against the oracle's search from each.
    ``oracle_result`` is the oracle's search of the same inputs when the
    caller already has it."""
    m, n = W_bits.shape
    G = n // 16
    r = oracle_result if oracle_result is not None else oracle.search(W_bits, h32, s_g, down=down, up=up, init=init)
    tie = oracle.near_tie_mask(r["e_best"], r["e_second"])
    codes_gpu = np.asarray(codes_gpu, np.uint8).reshape(m, G)
    packed_gpu = np.asarray(packed_gpu, np.uint8).reshape(m, n // 2)
    code_bad = codes_gpu != r["codes"]
    pk_bad = np.any((packed_gpu != r["packed"]).reshape(m, G, 8), axis=-1)
    # The GPU's packed bytes must be the oracle's quantization at its code.
    packed_at, err_at = oracle.quantize(W_bits, s_g, codes_gpu, h32)
    packed_consistent = np.all((packed_at == packed_gpu).reshape(m, G, 8), axis=-1)
    cg = codes_gpu.astype(np.int64)

    def valid_from(res):
        c0 = res["c0"].astype(np.int64)
        in_window = (cg >= np.clip(c0 - down, 1, 126)) & (cg <= np.clip(c0 + up, 1, 126))
        return in_window & (err_at <= res["e_best"] + TIE_REL * res["e_second"])

    valid = valid_from(r)
    init_tie = np.zeros((m, G), bool)
    if isinstance(init, str) and init == "4over6":
        c4 = oracle.anchor_codes(W_bits, s_g, 4.0)
        c6 = oracle.anchor_codes(W_bits, s_g, 6.0)
        l4, l6 = r["l4"], r["l6"]
        init_tie = (np.abs(l4 - l6) <= TIE_REL * np.maximum(l4, l6)) & (c4 != c6)
        if init_tie.any():
            alt = np.where(r["c0"] == c4, c6, c4).astype(np.uint8)
            r_alt = oracle.search(W_bits, h32, s_g, down=down, up=up, init=alt)
            valid |= init_tie & valid_from(r_alt)
    strict_bad = (code_bad | pk_bad) & ~tie & ~init_tie
    return dict(
        groups=int(m * G),
        near_ties=int(tie.sum()),
        init_ties=int(init_tie.sum()),
        tie_groups_differing=int(((code_bad | pk_bad) & (tie | init_tie)).sum()),
        mismatches=int(strict_bad.sum()),
        packed_inconsistent=int((~packed_consistent).sum()),
        invalid=int((~valid).sum()),
        ok=bool(strict_bad.sum() == 0 and packed_consistent.all() and valid.all()),
        oracle=r,
        tie_mask=tie | init_tie,
        init_tie_mask=init_tie,
        err_at_gpu_codes=err_at,
    )


# fp32 score of one group against the fp64 oracle: each of the 16 positive
# terms carries a few roundings (residual, square, weight) and the sum runs
# 4 chains of 4 then a 2-level tree, about 10 units of 2^-24 in all; the
# bound below leaves a factor of 3.
ERR_REL_TOL = 2e-6


def compare_stats(W_bits: np.ndarray, h32: np.ndarray, s_g: float, down: int, up: int, gpu: dict,
                  init="rtn") -> dict:
    """hscale_search_stats' outputs against the oracle: the search outputs as
    compare_search; the chosen shift bit-exact outside near-ties (and in
    range, consistent with the code, for every group); err_best within
    ERR_REL_TOL of the oracle's error at the GPU's code; err_init within
    ERR_REL_TOL of the oracle's error at the initial code."""
    m, n = W_bits.shape
    G = n // 16
    rep = compare_search(W_bits, h32, s_g, down, up, gpu["scale_codes"], gpu["packed_e2m1"], init=init)
    r = rep["oracle"]
    skip = rep["tie_mask"]
    shift = np.asarray(gpu["shift"], np.int64).reshape(m, G)
    eb = np.asarray(gpu["err_best"], np.float64).reshape(m, G)
    ei = np.asarray(gpu["err_init"], np.float64).reshape(m, G)
    codes = np.asarray(gpu["scale_codes"], np.int64).reshape(m, G)
    in_range = (shift >= -down) & (shift <= up)
    c0 = r["c0"].astype(np.int64)
    consistent = (np.clip(c0 + shift, 1, 126) == codes) | rep["init_tie_mask"]
    shift_bad = (shift != r["shift"]) & ~skip

    def rel(a, b):
        return np.abs(a - b) / np.where(b > 0, b, 1.0)

    eb_rel = rel(eb, rep["err_at_gpu_codes"])
    ei_rel = np.where(rep["init_tie_mask"], 0.0, rel(ei, r["e_init"]))
    ok = (rep["ok"] and in_range.all() and consistent.all() and shift_bad.sum() == 0
          and eb_rel.max(initial=0) <= ERR_REL_TOL and ei_rel.max(initial=0) <= ERR_REL_TOL)
    return dict(search=rep, shift_mismatches=int(shift_bad.sum()), shift_out_of_range=int((~in_range).sum()),
                shift_inconsistent=int((~consistent).sum()), err_best_max_rel=float(eb_rel.max(initial=0)),
                err_init_max_rel=float(ei_rel.max(initial=0)), ok=bool(ok))
