"""GPU parity of the quality diagnostics: the search with per-group
statistics and the per-shift summary (the appendix's selected-shift
analysis)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import parity
from synth.workloads import CONFIGS, harness_global_scale, make_activations, make_weight, tensor_bits

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()
    return hs


@pytest.fixture(scope="module")
def tiny(hs):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu")
    h = parity.oracle_h32(tensor_bits(make_activations(wl, "cpu")))
    return W, h, harness_global_scale(W)


def _np(d):
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in d.items()}


def _summary_from_arrays(shift, eb, ei, down, up):
    """Library histogram of given per-group arrays (bins d = -down..up;
    shifts outside are dropped)."""
    d = shift.ravel().astype(np.int64)
    keep = (d >= -down) & (d <= up)
    k = d[keep] + down
    K = down + up + 1
    a = ei.ravel().astype(np.float64)[keep]
    b = eb.ravel().astype(np.float64)[keep]
    rel = np.where(a > 0, (a - b) / np.where(a > 0, a, 1.0), 0.0)
    return dict(count=np.bincount(k, minlength=K), sum_init=np.bincount(k, weights=a, minlength=K),
                sum_best=np.bincount(k, weights=b, minlength=K), sum_rel=np.bincount(k, weights=rel, minlength=K))


def _check_summary_exact(s, ref):
    assert np.array_equal(s["count"].astype(np.int64), ref["count"])
    for q in ("sum_init", "sum_best", "sum_rel"):
        assert np.allclose(s[q], ref[q], rtol=1e-12, atol=1e-300), q


@pytest.mark.parametrize("init", ["maxabs", "4over6", "given"])
@pytest.mark.parametrize("down,up", [(0, 0), (4, 4), (9, 6), (125, 125)])
def test_search_stats_tiny(hs, tiny, init, down, up):
    W, h, s_g = tiny
    Wb = tensor_bits(W)
    init_arg, init_ref = init, ("rtn" if init == "maxabs" else init)
    if init == "given":
        rng = np.random.default_rng(down + 7 * up)
        base = oracle.anchor_codes(Wb, s_g, 6.0).astype(np.int64)
        init_ref = np.clip(base + rng.integers(-5, 6, base.shape), 1, 126).astype(np.uint8)
        init_arg = torch.from_numpy(init_ref).to(DEV)
    out = hs.search_stats(W.to(DEV), torch.from_numpy(h).to(DEV), s_g, down, up, init=init_arg)
    g = _np(out)
    rep = parity.compare_stats(Wb, h, s_g, down, up, g, init=init_ref)
    print(f"[stats tiny {init} -{down}..+{up}] shift_mismatches={rep['shift_mismatches']} "
          f"near_ties={rep['search']['near_ties']} err_best_max_rel={rep['err_best_max_rel']:.2e} "
          f"err_init_max_rel={rep['err_init_max_rel']:.2e}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "search"}
    # the plain entry point writes the same codes and bytes
    c, p = hs.search(W.to(DEV), torch.from_numpy(h).to(DEV), s_g, down=down, up=up, init=init_arg)
    torch.cuda.synchronize()
    assert np.array_equal(c.cpu().numpy(), g["scale_codes"]) and np.array_equal(p.cpu().numpy(), g["packed_e2m1"])
    # summary: the library histogram of the same arrays, and the oracle's
    # summary of its own search within the error tolerance
    s = _np(hs.shift_summary(out["shift"], out["err_best"], out["err_init"], down, up))
    _check_summary_exact(s, _summary_from_arrays(g["shift"], g["err_best"], g["err_init"], down, up))
    r = rep["search"]["oracle"]
    so = oracle.shift_summary(r["shift"], r["e_best"], r["e_init"], down, up)
    # Groups whose shift differs from the oracle's are near-ties or 4over6
    # anchor ties (compare_stats checked that); each moves one count.  An
    # anchor tie can also change the initial code (and so err_init) with the
    # same shift; then its code differs too.
    differ = int((g["shift"] != r["shift"]).sum())
    assert np.abs(s["count"].astype(np.int64) - so["count"]).sum() <= 2 * differ
    if differ == 0 and rep["search"]["tie_groups_differing"] == 0:
        for q in ("sum_init", "sum_best"):
            assert np.allclose(s[q], so[q], rtol=parity.ERR_REL_TOL, atol=0), q
        assert np.allclose(s["sum_rel"], so["sum_rel"], rtol=0, atol=4 * parity.ERR_REL_TOL * r["shift"].size)


def test_shift_summary_ragged_sizes_and_dropped_bins(hs):
    """Chunk boundaries of the summary (4096 groups per block) and shifts
    outside the requested bins (not counted); repeated calls are bitwise
    equal."""
    gen = torch.Generator().manual_seed(11)
    for groups in (1, 4095, 4096, 4097, 3 * 4096 + 5, 100000):
        shift = torch.randint(-9, 7, (groups,), generator=gen, dtype=torch.int8)
        ei = torch.exp(torch.randn(groups, generator=gen)).float()
        eb = ei * torch.rand(groups, generator=gen)
        eb[shift == 0] = ei[shift == 0]
        ei[::97] = 0.0
        eb[::97] = 0.0
        dev = [t.to(DEV) for t in (shift, eb, ei)]
        for down, up in ((9, 6), (3, 2), (0, 0)):
            s1 = _np(hs.shift_summary(*dev, down, up))
            s2 = _np(hs.shift_summary(*dev, down, up))
            for q in s1:
                assert np.array_equal(s1[q], s2[q])
            _check_summary_exact(s1, _summary_from_arrays(shift.numpy(), eb.numpy(), ei.numpy(), down, up))
    z = _np(hs.shift_summary(torch.empty(0, dtype=torch.int8, device=DEV),
                             torch.empty(0, device=DEV), torch.empty(0, device=DEV), 4, 4))
    assert all(np.all(v == 0) for v in z.values()) and z["count"].shape == (9,)


def test_search_stats_full_size_sampled(hs):
    """down_proj at full size, the paper's window [-9, +6]: sampled rows
    against the oracle, and the whole-matrix summary against the library
    histogram of the GPU's per-group arrays."""
    wl = CONFIGS["down_proj"]
    h = parity.oracle_h32(tensor_bits(make_activations(wl, "cpu", tokens=4096)))
    W = make_weight(wl, DEV)
    s_g = harness_global_scale(W)
    out = hs.search_stats(W, torch.from_numpy(h).to(DEV), s_g, 9, 6)
    s = _np(hs.shift_summary(out["shift"], out["err_best"], out["err_init"], 9, 6))
    g = _np(out)
    _check_summary_exact(s, _summary_from_arrays(g["shift"], g["err_best"], g["err_init"], 9, 6))
    rows = np.unique(np.r_[np.random.default_rng(3).choice(wl.out, 64, replace=False), 0, wl.out - 1])
    sub = {k: v[rows] for k, v in g.items()}
    rep = parity.compare_stats(tensor_bits(W[torch.from_numpy(rows).to(DEV)]), h, s_g, 9, 6, sub)
    removed = 1.0 - s["sum_best"].sum() / s["sum_init"].sum()
    frac = s["count"] / s["count"].sum()
    print(f"[stats down_proj -9..+6] shift_mismatches={rep['shift_mismatches']} "
          f"err_best_max_rel={rep['err_best_max_rel']:.2e} keep={frac[9]:.3f} larger={frac[10:].sum():.3f} "
          f"smaller={frac[:9].sum():.3f} removed={removed:.3f}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "search"}
    assert 0.0 < removed < 1.0


# ---------------------------------------------------------------------------
# Layer-output error (Eq. 3)
# ---------------------------------------------------------------------------

# Tolerance of the per-row output error against the fp64 oracle.  dW enters
# as hi + lo bf16 parts (relative error <= 2^-18 per element) and the
# products are accumulated in fp32, so y_t = (X dW^T)_tr carries a sum of
# independent rounding errors of about 2^-18 |x_tj dW_rj| each, which for
# sign-mixed terms is of order 2^-18 |y_t|.  L_r = sum_t y_t^2 then has a
# relative error of a few 1e-6, larger where a few tokens dominate the sum
# (up to 1.3e-5 measured on the small cases); the bar leaves a margin of 8.
LFULL_REL_TOL = 1e-4


def _lfull_case(hs, T, n, m, seed, window=4, tokens_dev=None):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu", shape=(m, n))
    X = make_activations(wl, "cpu", tokens=T, n=n)
    Wb, Xb = tensor_bits(W), tensor_bits(X)
    s_g = harness_global_scale(W)
    r = oracle.search(Wb, parity.oracle_h32(Xb), s_g, window=window)
    return W, X, Wb, Xb, s_g, r["codes"], r["packed"]


def _check_lfull(got, ref, label):
    rel = np.abs(got - ref) / np.where(ref > 0, ref, 1.0)
    print(f"[{label}] rows={len(ref)} max_rel={rel.max():.2e} total_rel="
          f"{abs(got.sum() - ref.sum()) / ref.sum():.2e}", flush=True)
    assert np.all(np.isfinite(got)) and rel.max() <= LFULL_REL_TOL, rel.max()


@pytest.mark.parametrize("T,n,m", [(128, 512, 256), (300, 48, 130), (1, 16, 1), (257, 96, 129), (513, 1040, 77)])
def test_output_error_matches_oracle(hs, T, n, m):
    W, X, Wb, Xb, s_g, codes, packed = _lfull_case(hs, T, n, m, seed=T + n + m)
    got = hs.output_error(X.to(DEV), W.to(DEV), s_g, torch.from_numpy(codes).to(DEV),
                          torch.from_numpy(packed).to(DEV))
    torch.cuda.synchronize()
    ref = oracle.output_error(Xb, oracle.delta(Wb, s_g, codes, packed))
    _check_lfull(got.cpu().numpy(), ref, f"L_full {T}x{n}x{m}")


def test_output_error_accumulates_and_code_zero(hs):
    W, X, Wb, Xb, s_g, codes, packed = _lfull_case(hs, 700, 256, 200, seed=1)
    codes = codes.copy()
    codes[5, :] = 0  # zero scale: W^ = 0 on that row
    Wd, Xd = W.to(DEV), X.to(DEV)
    ct, pt = torch.from_numpy(codes).to(DEV), torch.from_numpy(packed).to(DEV)
    whole = hs.output_error(Xd, Wd, s_g, ct, pt)
    acc = torch.zeros(200, dtype=torch.float64, device=DEV)
    for a, b in ((0, 1), (1, 256), (256, 700)):
        hs.output_error(Xd[a:b].contiguous(), Wd, s_g, ct, pt, row_err=acc)
    torch.cuda.synchronize()
    ref = oracle.output_error(Xb, oracle.delta(Wb, s_g, codes, packed))
    _check_lfull(whole.cpu().numpy(), ref, "L_full code 0")
    _check_lfull(acc.cpu().numpy(), ref, "L_full 3 batches")
    again = hs.output_error(Xd, Wd, s_g, ct, pt)
    torch.cuda.synchronize()
    assert torch.equal(again, whole)  # fixed-order sums: bitwise repeatable


def test_output_error_two_passes(hs):
    """More tokens than one tile launch covers (1024 token tiles of 384): the
    second pass adds its partials to the first."""
    T, n, m = 1024 * 384 + 300, 64, 96
    W, X, Wb, Xb, s_g, codes, packed = _lfull_case(hs, T, n, m, seed=2)
    got = hs.output_error(X.to(DEV), W.to(DEV), s_g, torch.from_numpy(codes).to(DEV),
                          torch.from_numpy(packed).to(DEV))
    torch.cuda.synchronize()
    ref = oracle.output_error(Xb, oracle.delta(Wb, s_g, codes, packed))
    _check_lfull(got.cpu().numpy(), ref, "L_full two passes")


def test_output_error_full_size_sampled(hs):
    """down_proj's full W (4096 x 14336) with 16384 calibration tokens, in the
    launch configuration the benchmark uses; the stored tensor is made by the
    oracle (max-abs codes shifted by seeded steps in -9..+6, quantized), and
    sampled rows are checked against the oracle."""
    wl = CONFIGS["down_proj"]
    X = make_activations(wl, "cpu", tokens=16384)
    Xb = tensor_bits(X)
    W = make_weight(wl, DEV)
    s_g = harness_global_scale(W)
    Wb_all = tensor_bits(W)
    c0 = oracle.anchor_codes(Wb_all, s_g, 6.0).astype(np.int64)
    codes = np.clip(c0 + np.random.default_rng(5).integers(-9, 7, c0.shape), 1, 126).astype(np.uint8)
    packed, _ = oracle.quantize(Wb_all, s_g, codes)
    got = hs.output_error(X.to(DEV), W, s_g, torch.from_numpy(codes).to(DEV), torch.from_numpy(packed).to(DEV))
    torch.cuda.synchronize()
    rows = np.unique(np.r_[np.random.default_rng(4).choice(wl.out, 10, replace=False), 0, wl.out - 1])
    ref = oracle.output_error(Xb, oracle.delta(Wb_all[rows], s_g, codes[rows], packed[rows]))
    _check_lfull(got.cpu().numpy()[rows], ref, "L_full down_proj sampled")


def test_output_error_70b_shape_sampled(hs):
    """The 70B down_proj shape (8192 x 28672: 32 row tiles, 896 k stages)
    with 2048 calibration tokens; the stored tensor is seeded random codes
    and nibbles (any stored NVFP4 tensor is a valid input); sampled rows
    against the oracle."""
    wl = CONFIGS["down_proj_70b"]
    X = make_activations(wl, "cpu", tokens=2048)
    Xb = tensor_bits(X)
    W = make_weight(wl, DEV)
    s_g = harness_global_scale(W)
    rng = np.random.default_rng(6)
    codes = rng.integers(60, 111, (wl.out, wl.inp // 16)).astype(np.uint8)
    packed = rng.integers(0, 256, (wl.out, wl.inp // 2)).astype(np.uint8)
    got = hs.output_error(X.to(DEV), W, s_g, torch.from_numpy(codes).to(DEV), torch.from_numpy(packed).to(DEV))
    torch.cuda.synchronize()
    rows = np.unique(np.r_[rng.choice(wl.out, 8, replace=False), 0, wl.out - 1])
    Wb = tensor_bits(W[torch.from_numpy(rows).to(DEV)])
    ref = oracle.output_error(Xb, oracle.delta(Wb, s_g, codes[rows], packed[rows]))
    _check_lfull(got.cpu().numpy()[rows], ref, "L_full 70b sampled")


def test_shift_summary_hand_worked_on_gpu(hs):
    """The hand-worked selected-shift case of the oracle pins, through
    hscale_shift_summary: every bin's count and fp64 sums exactly."""
    from tests.test_oracle_pins_diag import (HAND_DOWN, HAND_E_BEST, HAND_E_INIT, HAND_SHIFT, HAND_SUMMARY,
                                             HAND_UP)
    s = _np(hs.shift_summary(torch.from_numpy(HAND_SHIFT).to(DEV),
                             torch.from_numpy(HAND_E_BEST.astype(np.float32)).to(DEV),
                             torch.from_numpy(HAND_E_INIT.astype(np.float32)).to(DEV), HAND_DOWN, HAND_UP))
    for key, want in HAND_SUMMARY.items():
        assert np.array_equal(s[key], np.array(want, s[key].dtype)), (key, s[key])


def test_shift_summary_exact_groups_on_gpu(hs):
    """Groups exactly representable at their chosen code only: the GPU's
    statistics search scores them exactly 0 at that code, and each moved
    group adds exactly 1 to its bin's relative reduction (groups exact at
    their initial code add 0)."""
    from tests.test_oracle_pins_diag import exact_groups
    s_g = 2.0 ** -10
    Wb, init = exact_groups(s_g)
    h32 = np.exp(np.random.default_rng(1).standard_normal(Wb.shape[1])).astype(np.float32)
    W = torch.from_numpy(Wb.view(np.int16)).view(torch.bfloat16).to(DEV)
    down = up = 8
    st = _np(hs.search_stats(W, torch.from_numpy(h32).to(DEV), s_g, down, up,
                             init=torch.from_numpy(init).to(DEV)))
    r = oracle.search(Wb, h32, s_g, down=down, up=up, init=init)
    assert np.array_equal(st["scale_codes"], r["codes"]) and np.array_equal(st["packed_e2m1"], r["packed"])
    assert np.array_equal(st["shift"], r["shift"])
    assert np.all(st["err_best"] == 0.0)
    d = st["shift"].astype(np.int64)
    assert np.all(st["err_init"][d != 0] > 0) and np.all(st["err_init"][d == 0] == 0)
    s = _np(hs.shift_summary(torch.from_numpy(st["shift"]).to(DEV), torch.from_numpy(st["err_best"]).to(DEV),
                             torch.from_numpy(st["err_init"]).to(DEV), down, up))
    want = np.bincount(d.ravel() + down, minlength=down + up + 1)
    assert np.array_equal(s["count"], want)
    rel = want.astype(np.float64)
    rel[down] = 0.0
    assert np.array_equal(s["sum_rel"], rel)
