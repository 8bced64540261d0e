"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here runs on the CPU.  Each one checks the oracle against
something other than itself: the paper's worked example, a library routine
(torch's E4M3 decode and cast, numpy's round-half-even), closed forms,
invariants of the method, or brute force over the whole E4M3 ladder.
"""
import json
from pathlib import Path

import numpy as np
import pytest
import torch

import oracle
from tests import libref
from synth.workloads import CONFIGS, make_weight, make_activations, harness_global_scale, tensor_bits

GOLDEN = Path(__file__).resolve().parent / "golden"
GRID = libref.E2M1_GRID


def _bits(a_f32: np.ndarray) -> np.ndarray:
    """fp32 values that are exactly bf16 -> their bf16 bit patterns."""
    u = np.asarray(a_f32, np.float32).view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def _tiny_inputs(m=64, n=256, seed=0):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu")[:m, :n].contiguous()
    X = make_activations(wl, "cpu", tokens=96, n=n)
    Wb = tensor_bits(W)
    h = oracle.hdiag(tensor_bits(X)).astype(np.float32)
    s_g = harness_global_scale(W)
    return Wb, h, s_g


# ---------------------------------------------------------------------------
# Formats (Sec. 3.1, Eq. 7-8)
# ---------------------------------------------------------------------------

def test_e4m3_ladder_matches_torch_decode():
    lib = libref.ladder()
    ours = np.array([oracle.e4m3_value(c) for c in range(127)])
    assert np.array_equal(ours, lib)
    assert ours[1] == 2.0 ** -9 and ours[126] == 448.0
    assert np.all(np.diff(ours[1:]) > 0)  # strictly increasing in the byte: M = 126


def test_e4m3_round_matches_torch_cast():
    lam = libref.ladder()
    mids = ((lam[:-1] + lam[1:]) / 2).astype(np.float32)  # every midpoint, 0..2^-9 included
    up = np.nextafter(mids, np.float32(np.inf), dtype=np.float32)
    down = np.nextafter(mids, np.float32(0), dtype=np.float32)
    rng = np.random.default_rng(0)
    rand = np.exp(rng.uniform(np.log(1e-5), np.log(460.0), 20000)).astype(np.float32)
    extra = np.array([0.0, 448.0, 449.0, 460.0, 464.0], np.float32)
    t = np.concatenate([mids, up, down, lam.astype(np.float32), rand, extra])
    t = t[t <= 464.0]
    ours = np.array([oracle.e4m3_round(float(x)) for x in t])
    assert np.array_equal(ours, libref.e4m3_cast_codes(t))


def test_e4m3_round_saturates_and_ties_even():
    assert oracle.e4m3_round(1.0625) == 56  # tie between 1.0 (0x38) and 1.125 -> even
    assert oracle.e4m3_round(1.1875) == 58  # tie between 1.125 and 1.25 -> 1.25 (even)
    for t in (448.0, 464.0, 465.0, 1e6, 3e38):
        assert oracle.e4m3_round(t) == 126
    assert oracle.e4m3_round(2.0 ** -10) == 0  # tie between 0 and 2^-9 -> 0
    assert oracle.e4m3_round(1.5 * 2.0 ** -10) == 1


def test_e2m1_index_matches_library_rounding():
    mids = (GRID[:-1] + GRID[1:]) / 2
    xs = [GRID, mids, np.linspace(0, 12, 4801)]
    m32 = mids.astype(np.float32)
    xs.append(np.nextafter(m32, np.float32(np.inf), dtype=np.float32))
    xs.append(np.nextafter(m32, np.float32(0), dtype=np.float32))
    xs.append(np.array([1e-30, 7.0, 8.0, 1e10, np.float32(3.4e38)]))
    x = np.concatenate([np.asarray(a, np.float64) for a in xs]).astype(np.float32)
    ours = np.array([oracle.e2m1_index(float(v)) for v in x])
    assert np.array_equal(ours, libref.e2m1_round_index(x))
    # The paper's grid and clip (Sec. 3.1): midpoints go to the even index.
    assert [oracle.e2m1_index(v) for v in (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0)] == [0, 2, 2, 4, 4, 6, 6]
    assert [oracle.e2m1_value(i) for i in range(8)] == list(GRID)


def test_scale_tables_are_fp32_products():
    for s_g in (1.0, 3.0517578125e-05, 7.4505806e-09, float(np.float32(0.02 / 2688))):
        S, R = oracle.scale_tables(s_g)
        lam = libref.ladder().astype(np.float32)
        S_lib = (np.float32(s_g) * lam[1:]).astype(np.float32)
        assert np.array_equal(S[1:], S_lib)
        assert np.array_equal(R[1:], (np.float32(1.0) / S_lib).astype(np.float32))


# ---------------------------------------------------------------------------
# Paper worked example: App. A.1, Table scale_search_microcase
# ---------------------------------------------------------------------------

def test_microcase_quantizer_and_errors():
    g = json.loads((GOLDEN / "microcase.json").read_text())
    w = np.array(g["w"])
    X = np.array(g["X"])
    for row in g["rows"]:
        err, nib, what = oracle.group_at_scale(w, np.float32(row["scale"]))
        tol = 2e-3 if row["name"] == "hessian-guided" else 1e-3
        vals = GRID[nib & 7] * np.where(nib & 8, -1, 1)
        assert list(vals) == row["grid_values"], row["name"]
        assert np.allclose(what, row["w_hat"], atol=1e-3), row["name"]
        assert abs(err - row["weight_err"]) <= tol, (row["name"], err)  # h = 1: weight error
        out_err = float(np.sum((X @ (w - what)) ** 2))  # Eq. 3 on the printed X
        assert abs(out_err - row["output_err"]) <= tol, (row["name"], out_err)


def test_microcase_hdiag():
    """Eq. 4 on the microcase's printed X.  The oracle reads bf16, so X is
    rounded to bf16 first: h must equal the column sums of squares of those
    values exactly, and the printed h = diag(X^T X) to bf16 accuracy."""
    g = json.loads((GOLDEN / "microcase.json").read_text())
    Xt = torch.tensor(g["X"], dtype=torch.float32).to(torch.bfloat16)
    h = oracle.hdiag(tensor_bits(Xt))
    assert np.array_equal(h, (Xt.double().numpy() ** 2).sum(axis=0))
    assert np.allclose(h, g["h_diag_XtX"], rtol=1e-2)
    assert np.allclose((np.array(g["X"]) ** 2).sum(axis=0), g["h_diag_XtX"], atol=1e-9)


# ---------------------------------------------------------------------------
# h (Eq. 4)
# ---------------------------------------------------------------------------

def test_hdiag_equals_gram_diagonal():
    wl = CONFIGS["tiny"]
    X = make_activations(wl, "cpu", tokens=200, n=272)
    Xb = tensor_bits(X)
    Xf = X.float().numpy().astype(np.float64)
    h = oracle.hdiag(Xb)
    gram = Xf.T @ Xf
    assert np.allclose(h, np.diag(gram), rtol=1e-12, atol=0)


def test_hdiag_closed_forms():
    T, n = 37, 48
    X = np.full((T, n), 1.5, np.float32)
    assert np.array_equal(oracle.hdiag(_bits(X)), np.full(n, T * 2.25))
    assert np.array_equal(oracle.hdiag(np.zeros((0, n), np.uint16)), np.zeros(n))
    X = np.zeros((T, n), np.float32)
    X[5, 7] = -3.0
    X[9, 7] = 2.0
    h = oracle.hdiag(_bits(X))
    assert h[7] == 13.0 and np.count_nonzero(h) == 1


# ---------------------------------------------------------------------------
# The search (Eq. 7, 9-13)
# ---------------------------------------------------------------------------

def test_window_zero_is_rtn():
    Wb, h, s_g = _tiny_inputs()
    r = oracle.search(Wb, h, s_g, window=0)
    c_lib = libref.rtn_codes(Wb, s_g)
    assert np.array_equal(r["codes"], c_lib)
    assert np.array_equal(r["c0"], c_lib)
    nib, _ = libref.quantize_at(Wb, s_g, c_lib)
    assert np.array_equal(r["packed"], oracle.pack_nibbles(nib))


def test_candidates_are_the_clipped_walk():
    rng = np.random.default_rng(3)
    for _ in range(200):
        w = rng.normal(0, 0.02, 16)
        s_g = float(np.float32(rng.uniform(1e-6, 1e-4)))
        h = rng.uniform(0.1, 10, 16)
        down, up = int(rng.integers(0, 12)), int(rng.integers(0, 12))
        r = oracle.group_search(w, h, s_g, down, up)
        expect = np.clip(r["c0"] + np.arange(-down, up + 1), 1, 126)
        assert np.array_equal(r["cand_codes"], expect)
        k = int(np.argmin(r["cand_err"]))  # numpy argmin keeps the first minimum
        assert r["code"] == r["cand_codes"][k]


def test_search_never_worse_than_rtn_and_nested_windows():
    Wb, h, s_g = _tiny_inputs()
    e = {w: oracle.search(Wb, h, s_g, window=w)["e_best"] for w in (0, 1, 4, 8)}
    assert np.all(e[1] <= e[0]) and np.all(e[4] <= e[1]) and np.all(e[8] <= e[4])
    assert np.mean(e[4] < e[0]) > 0.3  # the search does move most groups


def test_uniform_h_is_weight_mse_search():
    Wb, _, s_g = _tiny_inputs()
    ones = np.ones(Wb.shape[1], np.float32)
    r = oracle.search(Wb, ones, s_g, window=4)
    c_lib, nib_lib, e_lib = libref.windowed_search(Wb, None, s_g, 4, 4)
    assert np.array_equal(r["codes"], c_lib)
    assert np.array_equal(r["packed"], oracle.pack_nibbles(nib_lib))
    assert np.allclose(r["e_best"], e_lib, rtol=1e-12)


def test_hessian_weighted_search_matches_library_search():
    Wb, h, s_g = _tiny_inputs()
    for down, up in ((4, 4), (9, 6), (0, 3)):
        r = oracle.search(Wb, h, s_g, down=down, up=up)
        c_lib, nib_lib, _ = libref.windowed_search(Wb, h, s_g, down, up)
        assert np.array_equal(r["codes"], c_lib)
        assert np.array_equal(r["packed"], oracle.pack_nibbles(nib_lib))


def test_full_window_equals_bruteforce_over_ladder():
    Wb, h, s_g = _tiny_inputs(m=16, n=128)
    r = oracle.search(Wb, h, s_g, window=125)
    errs = libref.all_code_errors(Wb, h, s_g)
    best = np.argmin(errs, axis=-1) + 1  # first minimum = smallest code
    assert np.array_equal(r["codes"], best)
    assert np.allclose(oracle.all_code_errors(Wb, h, s_g), errs, rtol=1e-12)


def test_weighted_error_equals_output_error_for_orthogonal_X():
    """When X^T X is diagonal, Eq. 5 is exact: the Eq. 13 score of every
    candidate equals ||X (w - w_hat)^T||^2 of Eq. 3."""
    rng = np.random.default_rng(7)
    n = 64
    d = np.exp(rng.normal(0, 1.0, n))  # X = diag(d): orthogonal columns
    X = np.diag(d)
    h = np.sum(X * X, axis=0)
    for trial in range(20):
        w = rng.standard_t(4, n) * 0.015
        s_g = float(np.float32(np.max(np.abs(w)) / 2688))
        for i in range(n // 16):
            sl = slice(16 * i, 16 * i + 16)
            r = oracle.group_search(w[sl], h[sl], s_g, 4, 4)
            S, _ = oracle.scale_tables(s_g)
            for c, e in zip(r["cand_codes"], r["cand_err"]):
                _, nib, what = oracle.group_at_scale(w[sl], S[c])
                full = np.zeros(n)
                full[sl] = w[sl] - what
                out = float(np.sum((X @ full) ** 2))
                assert np.isclose(e, out, rtol=1e-12), (trial, i, c)
            outs = [np.sum((X[:, sl] @ (w[sl] - oracle.group_at_scale(w[sl], S[c])[2])) ** 2)
                    for c in r["cand_codes"]]
            assert r["code"] == r["cand_codes"][int(np.argmin(outs))]


def test_one_hot_h_picks_best_single_weight():
    rng = np.random.default_rng(11)
    for _ in range(100):
        w = rng.normal(0, 0.02, 16)
        j = int(rng.integers(0, 16))
        h = np.zeros(16)
        h[j] = 3.0
        s_g = float(np.float32(np.max(np.abs(w)) / 2688))
        r = oracle.group_search(w, h, s_g, 4, 4)
        S, _ = oracle.scale_tables(s_g)
        errs = [(w[j] - oracle.group_at_scale(w, S[c])[2][j]) ** 2 * 3.0 for c in r["cand_codes"]]
        assert np.allclose(r["cand_err"], errs, rtol=1e-12)


def test_exactly_representable_group_has_zero_error():
    s_g = 2.0 ** -12
    S, _ = oracle.scale_tables(s_g)
    c = 70  # S[c] is a power-of-two multiple of a 4-bit mantissa: products exact
    vals = np.array([6, -4, 3, 0.5, -1.5, 2, 0, 1, 6, -6, 4, 3, -2, 1.5, 0.5, -1])
    w = vals * float(S[c])
    Wb = _bits(w.astype(np.float32)).reshape(1, 16)
    h = np.linspace(1, 2, 16).astype(np.float32)
    r = oracle.search(Wb, h, s_g, window=8)
    assert r["e_best"][0, 0] == 0.0
    nib = oracle.unpack_nibbles(r["packed"])[0]
    got = GRID[nib & 7] * np.where(nib & 8, -1, 1) * float(S[r["codes"][0, 0]])
    assert np.array_equal(got, w)


# ---------------------------------------------------------------------------
# Invariances of the method (exact while nothing over- or underflows)
# ---------------------------------------------------------------------------

def test_invariances():
    Wb, h, s_g = _tiny_inputs()
    base = oracle.search(Wb, h, s_g, window=4)
    # (1) h -> 2^k h
    for k in (-6, 5):
        r = oracle.search(Wb, (h * 2.0 ** k).astype(np.float32), s_g, window=4)
        assert np.array_equal(r["codes"], base["codes"])
        assert np.array_equal(r["packed"], base["packed"])
    # (2) (W, s_g) -> 2^k (W, s_g): bf16 exponent shift is exact
    for k in (-3, 4):
        w = libref.weights_f32(Wb) * np.float32(2.0 ** k)
        r = oracle.search(_bits(w), h, float(np.float32(s_g * 2.0 ** k)), window=4)
        assert np.array_equal(r["codes"], base["codes"])
        assert np.array_equal(r["packed"], base["packed"])
    # (3) W -> -W flips only the sign bits
    r = oracle.search(Wb ^ np.uint16(0x8000), h, s_g, window=4)
    assert np.array_equal(r["codes"], base["codes"])
    assert np.array_equal(r["packed"], base["packed"] ^ np.uint8(0x88))
    # (4) group locality and row permutation: permute rows and group columns
    m, n = Wb.shape
    G = n // 16
    rp = np.random.default_rng(1).permutation(m)
    gp = np.random.default_rng(2).permutation(G)
    cols = (gp[:, None] * 16 + np.arange(16)).reshape(-1)
    r = oracle.search(np.ascontiguousarray(Wb[rp][:, cols]), np.ascontiguousarray(h[cols]), s_g, window=4)
    assert np.array_equal(r["codes"], base["codes"][rp][:, gp])
    pcols = (gp[:, None] * 8 + np.arange(8)).reshape(-1)
    assert np.array_equal(r["packed"], base["packed"][rp][:, pcols])


# ---------------------------------------------------------------------------
# Degenerate groups
# ---------------------------------------------------------------------------

def test_zero_group_and_saturation():
    # All-zero group (with -0 entries): c0 clips to 1, every candidate has
    # error 0, the first (smallest) code wins, nibbles keep the sign bit.
    w = np.zeros(16, np.float32)
    Wb = _bits(w).reshape(1, 16)
    Wb[0, 3] = 0x8000
    h = np.ones(16, np.float32)
    r = oracle.search(Wb, h, 1e-3, window=4)
    assert r["c0"][0, 0] == 1 and r["codes"][0, 0] == 1
    nib = oracle.unpack_nibbles(r["packed"])[0]
    assert nib[3] == 8 and np.count_nonzero(nib) == 1
    assert oracle.near_tie_mask(r["e_best"], r["e_second"])[0, 0]
    # Saturation: a global scale far too small puts t above 448.
    w = np.full(16, 1.0, np.float32)
    r = oracle.search(_bits(w).reshape(1, 16), h, 1e-6, window=2)
    assert r["c0"][0, 0] == 126 and r["codes"][0, 0] == 126
    assert np.all(oracle.unpack_nibbles(r["packed"]) == 7)
    # Underflow: t below half of 2^-9 rounds to code 0 and clips to 1.
    w = np.full(16, 2.0 ** -20, np.float32)
    r = oracle.search(_bits(w).reshape(1, 16), h, 1.0, window=0)
    assert r["codes"][0, 0] == 1


def test_single_distinct_code_is_no_tie():
    # With one distinct candidate code there is no second-best error: window
    # 0, and a saturated group whose upward shifts all clip to code 126.
    rng = np.random.default_rng(3)
    u32 = (rng.standard_normal((4, 64)) * 0.02).astype(np.float32).view(np.uint32)
    w = ((u32 + 0x7FFF + ((u32 >> 16) & 1)) & 0xFFFF0000).astype(np.uint32).view(np.float32)  # to bf16
    h = np.ones(64, np.float32)
    r = oracle.search(_bits(w), h, float(np.float32(np.abs(w).max() / 2688)), window=0)
    assert np.all(np.isinf(r["e_second"])) and not oracle.near_tie_mask(r["e_best"], r["e_second"]).any()
    w = np.full(16, 1.0, np.float32)
    r = oracle.search(_bits(w).reshape(1, 16), np.ones(16, np.float32), 1e-6, down=0, up=3)
    assert r["codes"][0, 0] == 126 and np.isinf(r["e_second"][0, 0])
    assert not oracle.near_tie_mask(r["e_best"], r["e_second"])[0, 0]
