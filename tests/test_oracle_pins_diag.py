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
        rel = np.where(ei > 0, (ei - eb) / np.where(ei > 0, ei, 1), 0.0)
        assert np.allclose(s["sum_rel"], np.bincount(d, weights=rel, minlength=down + up + 1), rtol=1e-12)
        # the d = 0 bin removes nothing; every other bin removes something
        assert s["sum_rel"][down] == 0.0 and np.array_equal(s["sum_init"][down], s["sum_best"][down])
        other = np.arange(down + up + 1) != down
        assert np.all(s["sum_best"][other] <= s["sum_init"][other])
