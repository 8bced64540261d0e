"""Pins of the oracle's quality diagnostics: the rounding error Delta W of a
stored NVFP4 tensor, the layer-output error of Eq. 3 and the selected-shift
statistics (App. "Selected Scale Shifts", "Candidate-Window Width").

Each pin compares with something other than the oracle itself: a second
formula for the same quantity (the Gram form of Eq. 3), a special case that
reduces to a different oracle function (Eq. 3 with a diagonal X^T X is the
Eq. 5 surrogate), an independent numpy quantizer, the paper's worked
example, or a library histogram."""
import json
from pathlib import Path

import numpy as np
import torch

import oracle
from synth.workloads import CONFIGS, harness_global_scale, make_activations, make_weight, tensor_bits
from tests import libref

GOLDEN = Path(__file__).resolve().parent / "golden"


def _tiny(m=64, n=256, T=48, seed=0):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu")[:m, :n].contiguous()
    X = make_activations(wl, "cpu")[:T, :n].contiguous()
    return tensor_bits(W), tensor_bits(X), harness_global_scale(W)


def test_delta_matches_independent_quantizer():
    Wb, _, s_g = _tiny()
    h = np.ones(Wb.shape[1], np.float32)
    for window in (0, 4):
        r = oracle.search(Wb, h, s_g, window=window)
        d = oracle.delta(Wb, s_g, r["codes"], r["packed"])
        nib, _ = libref.quantize_at(Wb, s_g, r["codes"])
        S = (np.float32(s_g) * libref.ladder().astype(np.float32)[r["codes"].astype(np.int64)]).astype(np.float32)
        v = libref.E2M1_GRID[nib & 7] * np.where(nib & 8, -1.0, 1.0)
        what = v * np.repeat(S.astype(np.float64), 16, axis=1)
        assert np.array_equal(d, libref.weights_f32(Wb).astype(np.float64) - what)


def test_delta_zero_for_representable_weights_and_code_zero():
    s_g = 2.0 ** -10
    c = 56  # lambda = 1.0: S = 2^-10 exactly
    assert oracle.e4m3_value(c) == 1.0
    v = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6] * 2) * np.array([1] * 8 + [-1] * 8)
    w = torch.tensor((v * s_g)[None, :], dtype=torch.float32).to(torch.bfloat16)
    Wb = tensor_bits(w)
    codes = np.array([[c]], np.uint8)
    packed, _ = oracle.quantize(Wb, s_g, codes)
    assert np.array_equal(oracle.delta(Wb, s_g, codes, packed), np.zeros((1, 16)))
    # code 0 is a zero scale: W^ = 0 and Delta W = W whatever the nibbles
    d0 = oracle.delta(Wb, s_g, np.zeros((1, 1), np.uint8), packed)
    assert np.array_equal(d0, libref.weights_f32(Wb).astype(np.float64))


def test_output_error_equals_gram_form():
    """Eq. 3: ||X dW^T||_F^2 = Tr(dW X^T X dW^T), row by row."""
    Wb, Xb, s_g = _tiny()
    r = oracle.search(Wb, oracle.hdiag(Xb).astype(np.float32), s_g, window=4)
    d = oracle.delta(Wb, s_g, r["codes"], r["packed"])
    row = oracle.output_error(Xb, d)
    X = libref.weights_f32(Xb).astype(np.float64)
    G = X.T @ X
    gram = np.einsum("rj,jk,rk->r", d, G, d)
    assert np.all(row > 0)
    assert np.allclose(row, gram, rtol=1e-11, atol=0)
    # accumulating over token batches adds up
    acc = oracle.output_error(Xb[:17], d)
    oracle.output_error(Xb[17:], d, acc)
    assert np.allclose(acc, row, rtol=1e-13)


def test_output_error_with_diagonal_gram_is_the_surrogate():
    """With orthogonal columns of X, X^T X = diag(h) and Eq. 3 equals the
    Eq. 5 surrogate sum_j h_j dW_rj^2, which the quantizer scores."""
    Wb, _, s_g = _tiny(m=32, n=128)
    n = Wb.shape[1]
    a = torch.exp(torch.randn(n, generator=torch.Generator().manual_seed(3))).to(torch.bfloat16)
    X = torch.diag(a)  # T = n, one nonzero per column
    h = (a.float() ** 2).numpy()  # exact in fp32
    r = oracle.search(Wb, h, s_g, window=4)
    d = oracle.delta(Wb, s_g, r["codes"], r["packed"])
    row = oracle.output_error(tensor_bits(X), d)
    _, err = oracle.quantize(Wb, s_g, r["codes"], h)
    assert np.allclose(row, err.sum(axis=1), rtol=1e-12)
    assert np.allclose(err, r["e_best"], rtol=1e-12)


def test_output_error_paper_microcase():
    """The worked example's output errors (App. A.1), to the printed
    precision: X is rounded to bf16 for the oracle, which moves the errors
    by less than 6e-4 here."""
    g = json.loads((GOLDEN / "microcase.json").read_text())
    Xt = torch.tensor(g["X"], dtype=torch.float32).to(torch.bfloat16)
    w = np.array(g["w"])
    for row in g["rows"]:
        what = row["scale"] * np.array(row["grid_values"], dtype=np.float64)
        d = (w - what)[None, :]
        L = oracle.output_error(tensor_bits(Xt), d)[0]
        tol = 2e-3 if row["name"] == "hessian-guided" else 1e-3
        assert abs(L - row["output_err"]) <= tol, (row["name"], L)


def test_shift_summary_matches_histogram():
    Wb, Xb, s_g = _tiny()
    h = oracle.hdiag(Xb).astype(np.float32)
    for init, (down, up) in (("rtn", (9, 6)), ("4over6", (4, 4)), ("rtn", (0, 0))):
        r = oracle.search(Wb, h, s_g, down=down, up=up, init=init)
        s = oracle.shift_summary(r["shift"], r["e_best"], r["e_init"], down, up)
        d = r["shift"].ravel().astype(np.int64) + down
        assert np.array_equal(s["count"], np.bincount(d, minlength=down + up + 1))
        assert s["count"].sum() == r["shift"].size
        ei, eb = r["e_init"].ravel(), r["e_best"].ravel()
        assert np.allclose(s["sum_init"], np.bincount(d, weights=ei, minlength=down + up + 1), rtol=1e-12)
        assert np.allclose(s["sum_best"], np.bincount(d, weights=eb, minlength=down + up + 1), rtol=1e-12)
        # the d = 0 bin removes nothing; every other bin removes something
        assert s["sum_rel"][down] == 0.0 and np.array_equal(s["sum_init"][down], s["sum_best"][down])
        other = np.arange(down + up + 1) != down
        assert np.all(s["sum_best"][other] <= s["sum_init"][other])


# The per-shift relative reduction (App. "Selected Scale Shifts"): a group
# contributes (E(0) - E(d*)) / E(0) to its bin, 0 when E(0) = 0.  Worked by
# hand on six groups over bins d = -2..3:
#   d = -2: E(0) = 8, E(d*) = 2  -> 6/8 = 0.75
#   d = 1:  E(0) = 4, E(d*) = 1  -> 3/4 = 0.75;  E(0) = 2, E(d*) = 1 -> 1/2
#   d = 0:  E(0) = E(d*) = 5 -> 0;  E(0) = E(d*) = 0 -> 0
#   d = 3:  E(0) = E(d*) = 0 -> 0
HAND_SHIFT = np.array([1, 1, -2, 0, 3, 0], np.int8)
HAND_E_INIT = np.array([4.0, 2.0, 8.0, 5.0, 0.0, 0.0])
HAND_E_BEST = np.array([1.0, 1.0, 2.0, 5.0, 0.0, 0.0])
HAND_DOWN, HAND_UP = 2, 3
HAND_SUMMARY = dict(count=[1, 0, 2, 2, 0, 1], sum_init=[8.0, 0.0, 5.0, 6.0, 0.0, 0.0],
                    sum_best=[2.0, 0.0, 5.0, 2.0, 0.0, 0.0], sum_rel=[0.75, 0.0, 0.0, 1.25, 0.0, 0.0])


def test_shift_summary_hand_worked():
    s = oracle.shift_summary(HAND_SHIFT, HAND_E_BEST, HAND_E_INIT, HAND_DOWN, HAND_UP)
    for key, want in HAND_SUMMARY.items():
        assert np.array_equal(s[key], np.array(want, s[key].dtype)), (key, s[key])


def exact_groups(s_g=2.0 ** -10):
    """Groups of bf16 weights that are exactly E2M1 values times S[c] at one
    code c, with the initial code c0 != c (so that E(d*) = 0 < E(0)), and
    groups exact at their own max-abs code (E(0) = E(d*) = 0).  Every group
    holds 0.5 and its largest value (4 or 6) on the grid, so c is its only
    exact code: the ratio S[c'] / S[c] would have to map both onto the grid.

    Returns (W bits [rows, 80], initial codes [rows, 5]): the max-abs code,
    or a given code `k` codes away from c (k = -3, +2, +7)."""
    S, _ = oracle.scale_tables(s_g)
    grid = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    rng = np.random.default_rng(4)
    groups, init = [], []
    for c in range(40, 90, 3):
        for vmax, shift in ((4.0, None), (6.0, 0), (6.0, -3), (6.0, 2), (4.0, 7)):
            v = rng.choice(grid[grid <= vmax], 16)
            v[0] = vmax
            v[1] = 0.5  # not exact at c + 8 (v / 2 off the grid)
            sign = rng.choice([-1.0, 1.0], 16)
            w = (sign * v * float(S[c])).astype(np.float32)
            assert np.all((w.view(np.uint32) & 0xFFFF) == 0)  # exact in bf16
            groups.append((w.view(np.uint32) >> 16).astype(np.uint16))
            Wg = groups[-1][None, :]
            c_max = int(oracle.anchor_codes(Wg, s_g, 6.0)[0, 0])
            # max-abs start (vmax < 6 puts c0 below c), or a given start
            # `shift` codes away from c
            init.append(c_max if shift is None or shift == 0 else c - shift)
    Wb = np.stack(groups).reshape(-1, 16 * 5)
    return Wb, np.array(init, np.uint8).reshape(Wb.shape[0], 5)


def test_shift_summary_exact_groups_contribute_one():
    """A group exactly representable at its chosen code but not at its
    initial code removes all of its initial error: it adds exactly 1 to its
    bin's sum_rel.  A group exact at its initial code adds 0 (E(0) = 0).
    Brute force over all 126 codes shows each exact group's zero is unique."""
    s_g = 2.0 ** -10
    Wb, init = exact_groups(s_g)
    h = np.exp(np.random.default_rng(1).standard_normal(Wb.shape[1])).astype(np.float32)
    allerr = oracle.all_code_errors(Wb, h, s_g)  # [m, G, 126]
    zero_code = allerr.argmin(axis=-1) + 1
    exact = allerr.min(axis=-1) == 0.0
    assert exact.all()
    assert np.all((allerr == 0.0).sum(axis=-1) == 1)  # the zero is unique
    down = up = 8
    r = oracle.search(Wb, h, s_g, down=down, up=up, init=init)
    assert np.array_equal(r["codes"], zero_code.astype(np.uint8))
    assert np.all(r["e_best"] == 0.0)
    d = r["shift"].astype(np.int64)
    assert np.array_equal(d, zero_code - init.astype(np.int64))
    moved = d != 0
    assert moved.sum() >= 20 and (~moved).sum() >= 10 and np.any(d < 0) and np.any(d > 0)
    assert np.all(r["e_init"][moved] > 0) and np.all(r["e_init"][~moved] == 0)
    s = oracle.shift_summary(r["shift"], r["e_best"], r["e_init"], down, up)
    want_count = np.bincount(d.ravel() + down, minlength=down + up + 1)
    assert np.array_equal(s["count"], want_count)
    want_rel = want_count.astype(np.float64)
    want_rel[down] = 0.0  # the d = 0 groups are exact at c0: nothing to remove
    assert np.array_equal(s["sum_rel"], want_rel)
    assert np.all(s["sum_best"] == 0.0)


def test_shift_summary_mean_reduction_in_unit_interval():
    """On a real search every bin's mean relative reduction lies in [0, 1]
    (0 exactly in the d = 0 bin), and the groups with E(0) = 0 add nothing."""
    Wb, Xb, s_g = _tiny()
    h = oracle.hdiag(Xb).astype(np.float32)
    Wz = Wb.copy()
    Wz[:4, :32] = 0  # all-zero groups: E(0) = 0
    for down, up in ((4, 4), (9, 6)):
        r = oracle.search(Wz, h, s_g, down=down, up=up)
        s = oracle.shift_summary(r["shift"], r["e_best"], r["e_init"], down, up)
        cnt = s["count"].astype(np.float64)
        mean = np.divide(s["sum_rel"], cnt, out=np.zeros_like(cnt), where=cnt > 0)
        assert np.all(mean >= 0.0) and np.all(mean <= 1.0)
        assert s["sum_rel"][down] == 0.0
        assert np.all(s["sum_rel"] <= cnt)
