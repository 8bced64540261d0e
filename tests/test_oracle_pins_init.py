"""Pins of the oracle's initial-code rules and streamed h.

* the 4over6 initialisation (App. B, Alg. combining 4over6 with H-Scale) at
  window 0 against a library-built 4over6 and a closed-form group;
* the search from caller-provided initial codes (Alg. HScaleGroupQuantize
  takes the baseline's scale as input) against the max-abs search and brute
  force;
* h accumulated over streamed batches against h of the concatenation.
"""
import numpy as np

import oracle
from tests import libref
from tests.test_oracle_pins import _bits, _tiny_inputs
from synth.workloads import CONFIGS, make_activations, tensor_bits

GRID = libref.E2M1_GRID


def test_4over6_window0_matches_library():
    Wb, h, s_g = _tiny_inputs()
    r = oracle.search(Wb, h, s_g, window=0, init="4over6")
    c_lib = libref.four_over_six_codes(Wb, s_g)
    assert np.array_equal(r["codes"], c_lib)
    assert np.array_equal(r["c0"], c_lib)
    nib, _ = libref.quantize_at(Wb, s_g, c_lib)
    assert np.array_equal(r["packed"], oracle.pack_nibbles(nib))
    # both anchors are used on this data
    c6 = libref.rtn_codes(Wb, s_g, 6.0)
    assert 0.05 < np.mean(c_lib != c6) < 0.95


def test_4over6_closed_form_group():
    """Weights on the E2M1 grid scaled so that max|w| maps to 4: anchor 4
    reproduces them exactly (L4 = 0) while anchor 6 cannot."""
    s_g = 2.0 ** -10
    S, _ = oracle.scale_tables(s_g)
    c = 80  # l_80 = 1.0 * 2^3; S[80] = 2^-7 exactly
    vals = np.array([4, 3, -3, 2, 1.5, -1, 0.5, 0, 4, -4, 3, 2, -2, 1, 0.5, -1.5])
    w = (vals * float(S[c])).astype(np.float32)
    Wb = _bits(w).reshape(1, 16)
    r = oracle.search(Wb, np.ones(16, np.float32), s_g, window=0, init="4over6")
    assert r["l4"][0, 0] == 0.0 and r["l6"][0, 0] > 0.0
    assert r["codes"][0, 0] == c and r["e_best"][0, 0] == 0.0
    nib = oracle.unpack_nibbles(r["packed"])[0]
    assert np.array_equal(GRID[nib & 7] * np.where(nib & 8, -1, 1), vals)


def test_4over6_never_worse_than_rtn_in_plain_mse():
    Wb, h, s_g = _tiny_inputs()
    r46 = oracle.search(Wb, h, s_g, window=0, init="4over6")
    rrtn = oracle.search(Wb, h, s_g, window=0)
    ones = np.ones(Wb.shape[1], np.float32)
    _, l46 = oracle.quantize(Wb, s_g, r46["codes"], ones)
    _, lrtn = oracle.quantize(Wb, s_g, rrtn["codes"], ones)
    assert np.all(l46 <= lrtn)
    assert np.allclose(np.minimum(r46["l4"], r46["l6"]), l46, rtol=1e-12)


def test_4over6_search_never_worse_than_its_init():
    Wb, h, s_g = _tiny_inputs()
    r0 = oracle.search(Wb, h, s_g, window=0, init="4over6")
    for down, up in ((4, 4), (9, 6)):
        r = oracle.search(Wb, h, s_g, down=down, up=up, init="4over6")
        assert np.array_equal(r["c0"], r0["c0"])
        assert np.all(r["e_best"] <= r0["e_best"])


def test_given_init_equals_rtn_search():
    Wb, h, s_g = _tiny_inputs()
    for down, up in ((0, 0), (4, 4), (9, 6)):
        a = oracle.search(Wb, h, s_g, down=down, up=up)
        b = oracle.search(Wb, h, s_g, down=down, up=up, init=libref.rtn_codes(Wb, s_g).astype(np.uint8))
        for k in ("codes", "packed", "e_best", "e_second", "c0"):
            assert np.array_equal(a[k], b[k]), k


def test_given_init_window0_and_clip():
    Wb, h, s_g = _tiny_inputs(m=16, n=128)
    rng = np.random.default_rng(4)
    init = rng.integers(0, 256, size=(16, 8)).astype(np.uint8)  # includes 0 and > 126
    r = oracle.search(Wb, h, s_g, window=0, init=init)
    expect = np.clip(init.astype(np.int64), 1, 126)
    assert np.array_equal(r["codes"], expect)
    nib, _ = libref.quantize_at(Wb, s_g, expect)
    assert np.array_equal(r["packed"], oracle.pack_nibbles(nib))
    # An initial code outside the ladder is clipped into it before the walk
    # (code 0 starts at 1, codes above 126 at 126), as the walk's own clip.
    for win in (3, 9):
        a = oracle.search(Wb, h, s_g, window=win, init=init)
        b = oracle.search(Wb, h, s_g, window=win, init=expect.astype(np.uint8))
        assert np.array_equal(a["codes"], b["codes"]) and np.array_equal(a["packed"], b["packed"])
        z = oracle.search(Wb, h, s_g, window=win, init=np.zeros_like(init))
        o = oracle.search(Wb, h, s_g, window=win, init=np.ones_like(init))
        assert np.array_equal(z["codes"], o["codes"]) and np.array_equal(z["packed"], o["packed"])


def test_given_init_full_window_is_bruteforce():
    Wb, h, s_g = _tiny_inputs(m=16, n=128)
    rng = np.random.default_rng(6)
    init = rng.integers(1, 127, size=(16, 8)).astype(np.uint8)
    r = oracle.search(Wb, h, s_g, window=125, init=init)
    errs = libref.all_code_errors(Wb, h, s_g)
    assert np.array_equal(r["codes"], np.argmin(errs, axis=-1) + 1)


def test_hdiag_accumulate_equals_concatenation():
    wl = CONFIGS["tiny"]
    X = tensor_bits(make_activations(wl, "cpu", tokens=300, n=160))
    h64 = np.zeros(160)
    for a, b in ((0, 7), (7, 130), (130, 131), (131, 300)):
        oracle.hdiag_accumulate(X[a:b], h64)
    assert np.allclose(h64, oracle.hdiag(X), rtol=1e-13, atol=0)
    h64b = np.full(160, 2.5)
    oracle.hdiag_accumulate(X[:0], h64b)
    assert np.all(h64b == 2.5)


def test_4over6_tie_goes_to_anchor_4():
    """Sixteen equal weights v = 6 * 2^-10 with s_g = 2^-10: anchor 6 gives
    t = 1.0 (code 56, x = 6 exactly) and anchor 4 gives t = 1.5 (code 60,
    x rounds to 4); both reproduce v exactly, so L4 = L6 = 0 and the first
    anchor of the ordered set (4, 6) must win."""
    s_g = 2.0 ** -10
    w = np.full(16, 6.0 * 2.0 ** -10, np.float32)
    Wb = _bits(w).reshape(1, 16)
    r = oracle.search(Wb, np.ones(16, np.float32), s_g, window=0, init="4over6")
    assert r["l4"][0, 0] == 0.0 and r["l6"][0, 0] == 0.0
    assert r["codes"][0, 0] == 60
    assert libref.four_over_six_codes(Wb, s_g)[0, 0] == 60


def test_anchor_codes():
    Wb, h, s_g = _tiny_inputs()
    assert np.array_equal(oracle.anchor_codes(Wb, s_g, 6.0), libref.rtn_codes(Wb, s_g, 6.0))
    assert np.array_equal(oracle.anchor_codes(Wb, s_g, 4.0), libref.rtn_codes(Wb, s_g, 4.0))
    assert np.array_equal(oracle.anchor_codes(Wb, s_g, 6.0), oracle.search(Wb, h, s_g, window=0)["c0"])


def test_shift_and_initial_error():
    """The chosen shift d* and the error at d = 0 (the selected-shift and
    error-removed statistics of Sec. 4's ablation figure)."""
    Wb, h, s_g = _tiny_inputs()
    for init in ("rtn", "4over6"):
        r = oracle.search(Wb, h, s_g, down=9, up=6, init=init)
        d = r["shift"].astype(np.int64)
        assert d.min() >= -9 and d.max() <= 6
        assert np.array_equal(np.clip(r["c0"].astype(np.int64) + d, 1, 126), r["codes"])
        _, e0 = oracle.quantize(Wb, s_g, r["c0"], h)
        assert np.allclose(r["e_init"], e0, rtol=1e-12)
        assert np.all(r["e_best"] <= r["e_init"])
        assert np.array_equal(r["e_best"] == r["e_init"], d == 0) or np.all(r["e_best"][d != 0] < r["e_init"][d != 0])
        r0 = oracle.search(Wb, h, s_g, window=0, init=init)
        assert np.all(r0["shift"] == 0) and np.array_equal(r0["e_init"], r0["e_best"])
