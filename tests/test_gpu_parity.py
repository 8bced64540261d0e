"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Small cases are compared in full; the full-size workloads are compared on
sampled rows and columns that the oracle computes one by one, in the same
launch configuration the benchmark times.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import parity
from synth.workloads import (CONFIGS, block_workloads, harness_global_scale, make_activations, make_weight,
                             tensor_bits)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()  # raises if the HIP library is not built: no fallback
    return hs


def _bits_to_bf16(bits: np.ndarray, device=DEV) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def _run_search(hs, W, h, s_g, down, up):
    codes, packed = hs.search(W, h, s_g, down=down, up=up)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), packed.cpu().numpy()


def _assert_search_parity(hs, W, h, s_g, down, up, label):
    codes, packed = _run_search(hs, W, h, s_g, down, up)
    rep = parity.compare_search(tensor_bits(W), h.cpu().numpy(), s_g, down, up, codes, packed)
    print(f"[{label}] down={down} up={up} groups={rep['groups']} near_ties={rep['near_ties']} "
          f"tie_groups_differing={rep['tie_groups_differing']} mismatches={rep['mismatches']}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}
    return rep


# ---------------------------------------------------------------------------
# hdiag
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,n", [(128, 512), (1, 16), (7, 48), (1000, 528), (3000, 1040), (257, 4096),
                                 (513, 16)])
def test_hdiag_matches_oracle(hs, T, n):
    wl = CONFIGS["tiny"]
    X = make_activations(wl, "cpu", tokens=T, n=n)
    h = hs.hdiag(X.to(DEV))
    torch.cuda.synchronize()
    rep = parity.compare_h(h.cpu().numpy(), oracle.hdiag(tensor_bits(X)))
    print(f"[hdiag T={T} n={n}] max_rel={rep['max_rel']:.3e}", flush=True)
    assert rep["ok"], rep
    assert rep["max_rel"] <= 2e-6  # the documented bound


def test_hdiag_zero_tokens_and_zero_columns(hs):
    X = torch.empty((0, 64), dtype=torch.bfloat16, device=DEV)
    h = torch.full((64,), 7.0, device=DEV)
    hs.hdiag(X, h=h)
    torch.cuda.synchronize()
    assert torch.all(h == 0)
    X = make_activations(CONFIGS["tiny"], "cpu", tokens=300, n=96)
    X[:, 5] = 0
    X[:, 90:] = 0
    h = hs.hdiag(X.to(DEV)).cpu().numpy()
    assert h[5] == 0 and np.all(h[90:] == 0)
    assert parity.compare_h(h, oracle.hdiag(tensor_bits(X)))["ok"]


def test_hdiag_deterministic(hs):
    X = make_activations(CONFIGS["tiny"], DEV, tokens=20000, n=1536)
    a = hs.hdiag(X)
    b = hs.hdiag(X)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["attn_proj", "down_proj", "down_proj_70b"])
def test_hdiag_full_size_sampled(hs, name):
    wl = CONFIGS[name]
    print(f"[hdiag full {name}] generating X {wl.tokens}x{wl.inp}", flush=True)
    X = make_activations(wl, DEV)
    h = hs.hdiag(X)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    cols = np.unique(np.concatenate([rng.choice(wl.inp, 48, replace=False), [0, wl.inp - 1]]))
    cols_t = torch.from_numpy(cols).to(DEV)
    Xs = X.index_select(1, cols_t).contiguous()
    ref = oracle.hdiag(tensor_bits(Xs))
    rep = parity.compare_h(h.cpu().numpy()[cols], ref)
    print(f"[hdiag full {name}] sampled {len(cols)} columns max_rel={rep['max_rel']:.3e}", flush=True)
    del X
    assert rep["ok"], rep


# ---------------------------------------------------------------------------
# search
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tiny_case(hs):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu")
    X = make_activations(wl, "cpu")
    h = torch.from_numpy(parity.oracle_h32(tensor_bits(X))).to(DEV)
    return W.to(DEV), h, harness_global_scale(W)


@pytest.mark.parametrize("down,up", [(0, 0), (1, 1), (4, 4), (8, 8), (125, 125), (9, 6), (0, 6), (6, 0)])
def test_search_tiny_parity(hs, tiny_case, down, up):
    W, h, s_g = tiny_case
    _assert_search_parity(hs, W, h, s_g, down, up, "tiny")


def test_search_window_zero_equals_rtn_and_quantize(hs, tiny_case):
    W, h, s_g = tiny_case
    codes, packed = _run_search(hs, W, h, s_g, 0, 0)
    packed_q = hs.quantize(W, s_g, torch.from_numpy(codes).to(DEV)).cpu().numpy()
    assert np.array_equal(packed_q, packed)
    codes4, packed4 = _run_search(hs, W, h, s_g, 4, 4)
    assert np.array_equal(hs.quantize(W, s_g, torch.from_numpy(codes4).to(DEV)).cpu().numpy(), packed4)


def test_search_symmetric_entry_point_equals_du(hs, tiny_case):
    W, h, s_g = tiny_case
    c1, p1 = hs.search(W, h, s_g, window=4)
    c2, p2 = hs.search(W, h, s_g, down=4, up=4)
    assert torch.equal(c1, c2) and torch.equal(p1, p2)


def test_search_uniform_h(hs, tiny_case):
    W, _, s_g = tiny_case
    ones = torch.ones(W.shape[1], dtype=torch.float32, device=DEV)
    _assert_search_parity(hs, W, ones, s_g, 4, 4, "tiny h=1")


@pytest.mark.parametrize("m,n", [(1, 16), (3, 48), (1000, 16 * 37), (5, 4096), (77, 1040)])
def test_search_ragged_shapes(hs, m, n):
    wl = CONFIGS["tiny"]
    W = make_weight(wl, "cpu", shape=(m, n))
    X = make_activations(wl, "cpu", tokens=64, n=n)
    h = torch.from_numpy(parity.oracle_h32(tensor_bits(X))).to(DEV)
    _assert_search_parity(hs, W.to(DEV), h, harness_global_scale(W), 4, 4, f"ragged {m}x{n}")


def test_search_edge_groups(hs):
    """Zero groups (with -0), zero-h columns, a single huge outlier, sign
    flip, and a global scale small enough to saturate every group."""
    rng = np.random.default_rng(5)
    m, n = 64, 256
    w = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    w[3, :16] = 0.0
    w[4, 16:32] = -0.0
    w[5, 40] = 50.0
    W = torch.from_numpy(w).to(torch.bfloat16)
    hv = np.exp(rng.standard_normal(n)).astype(np.float32)
    hv[100:116] = 0.0
    hv[7] = 0.0
    h = torch.from_numpy(hv).to(DEV)
    s_g = harness_global_scale(W)
    _assert_search_parity(hs, W.to(DEV), h, s_g, 4, 4, "edge")
    _assert_search_parity(hs, (-W).to(DEV), h, s_g, 4, 4, "edge -W")
    c_pos, p_pos = _run_search(hs, W.to(DEV), h, s_g, 4, 4)
    c_neg, p_neg = _run_search(hs, (-W).to(DEV), h, s_g, 4, 4)
    assert np.array_equal(c_pos, c_neg) and np.array_equal(p_pos ^ 0x88, p_neg)
    # saturation: t = max|w| / 6 / s_g far above 448
    _assert_search_parity(hs, W.to(DEV), h, 1e-9, 3, 3, "saturating")
    # a large global scale: every group underflows to code 1
    _assert_search_parity(hs, W.to(DEV), h, 1e3, 3, 3, "underflowing")


def test_search_power_of_two_scale_ties(hs):
    """With s_g a power of two, weights placed exactly on E2M1 midpoints of a
    candidate (and one bf16 ulp either side) exercise the tie rules."""
    s_g = 2.0 ** -14
    S, _ = oracle.scale_tables(s_g)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    rng = np.random.default_rng(9)
    rows = []
    for c in range(48, 80):
        for _ in range(4):
            base = rng.choice(mids, 16) * float(S[c])
            base = base.astype(np.float32)
            u = base.view(np.uint32)
            assert np.all((u & 0xFFFF) == 0)  # S[c] has a short mantissa: midpoints are bf16
            bits = (u >> 16).astype(np.int32) + rng.integers(-1, 2, 16)
            sign = rng.integers(0, 2, 16) << 15
            rows.append((bits | sign).astype(np.uint16))
    Wb = np.stack(rows).reshape(-1, 64)
    W = _bits_to_bf16(Wb)
    h = torch.from_numpy(np.exp(rng.standard_normal(64)).astype(np.float32)).to(DEV)
    for down, up in ((0, 0), (4, 4)):
        _assert_search_parity(hs, W, h, s_g, down, up, "pow2 ties")


def test_quantizer_map_exhaustive(hs):
    """Every finite bf16 magnitude (both signs) at every scale code, for
    several global scales: the GPU's packed E2M1 codes equal the oracle's."""
    mags = np.arange(0x0000, 0x7F80, dtype=np.uint16)  # +0 .. largest finite
    vals = np.concatenate([mags, mags | 0x8000])
    pad = (-len(vals)) % 16
    vals = np.concatenate([vals, np.zeros(pad, np.uint16)])
    n = len(vals)
    Wb = np.tile(vals, (126, 1))
    codes = np.repeat(np.arange(1, 127, dtype=np.uint8)[:, None], n // 16, axis=1)
    W = _bits_to_bf16(Wb)
    codes_t = torch.from_numpy(codes).to(DEV)
    for s_g in (float(np.float32(0.2 / 2688)), 2.0 ** -12, float(np.float32(3.3e-5)), 1.0,
                float(np.float32(1.7e-3))):
        packed = hs.quantize(W, s_g, codes_t).cpu().numpy()
        ref, _ = oracle.quantize(Wb, s_g, codes)
        bad = int((packed != ref).sum())
        print(f"[quantizer map] s_g={s_g:.6g} bytes={packed.size} mismatches={bad}", flush=True)
        assert bad == 0


def test_quantize_clips_out_of_range_code_bytes(hs, tiny_case):
    """Code bytes outside 1..126 (0, the NaN pattern 127, sign-bit bytes
    128..255) are clipped into the ladder as the header documents: the
    packed codes equal the oracle's window-0 search from those bytes (the
    oracle clips given initial codes) and its quantizer at the clipped codes."""
    W, h, s_g = tiny_case
    m, n = W.shape
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 256, (m, n // 16)).astype(np.uint8)
    codes[0, :6] = [0, 1, 126, 127, 128, 255]
    assert np.any(codes == 0) and np.any(codes > 126)
    packed = hs.quantize(W, s_g, torch.from_numpy(codes).to(DEV)).cpu().numpy()
    Wb = tensor_bits(W)
    ref = oracle.search(Wb, h.cpu().numpy(), s_g, down=0, up=0, init=codes)
    assert np.array_equal(packed, ref["packed"])
    at, _ = oracle.quantize(Wb, s_g, np.clip(codes, 1, 126).astype(np.uint8))
    assert np.array_equal(packed, at)
    # the search from the same bytes at window 0 writes the same bytes
    c_from, p_from = hs.search(W, h, s_g, window=0, init=torch.from_numpy(codes).to(DEV))
    assert np.array_equal(p_from.cpu().numpy(), packed)
    assert np.array_equal(c_from.cpu().numpy(), np.clip(codes, 1, 126))


def test_search_deterministic(hs):
    wl = CONFIGS["attn_proj"]
    W = make_weight(wl, DEV)
    h = torch.exp(torch.randn(wl.inp, device=DEV))
    s_g = harness_global_scale(W)
    a = hs.search(W, h, s_g, window=4)
    b = hs.search(W, h, s_g, window=4)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def _sampled_rows(m, k, seed=0):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.choice(m, min(k, m), replace=False), [0, m - 1]]))


@pytest.mark.parametrize("name", ["attn_proj", "down_proj", "down_proj_70b"])
def test_search_full_size_sampled(hs, name):
    """Full-size W in the launch configuration the benchmark times, with h
    computed by the oracle from the first 4096 calibration tokens; the oracle
    checks sampled rows given the same h."""
    wl = CONFIGS[name]
    print(f"[search full {name}] generating", flush=True)
    h = torch.from_numpy(parity.oracle_h32(tensor_bits(make_activations(wl, "cpu", tokens=4096)))).to(DEV)
    W = make_weight(wl, DEV)
    s_g = harness_global_scale(W)
    codes, packed = hs.search(W, h, s_g, window=wl.window)
    torch.cuda.synchronize()
    rows = _sampled_rows(wl.out, 96)
    rows_t = torch.from_numpy(rows).to(DEV)
    Wb = tensor_bits(W.index_select(0, rows_t))
    rep = parity.compare_search(Wb, h.cpu().numpy(), s_g, wl.window, wl.window,
                                codes.index_select(0, rows_t).cpu().numpy(),
                                packed.index_select(0, rows_t).cpu().numpy())
    print(f"[search full {name}] rows={len(rows)} groups={rep['groups']} near_ties={rep['near_ties']} "
          f"mismatches={rep['mismatches']}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}


def test_search_grid_stride_path(hs):
    """More groups than one launch has lanes (65536 blocks x 256), so lanes
    loop; rows near both ends and around the wrap are checked."""
    m, n = 8200, 32768
    wl = CONFIGS["down_proj"]
    W = make_weight(wl, DEV, shape=(m, n))
    h = torch.exp(torch.randn(n, device=DEV))
    s_g = harness_global_scale(W)
    codes, packed = hs.search(W, h, s_g, window=2)
    torch.cuda.synchronize()
    lanes = 65536 * 256
    wrap_row = lanes // (n // 16)
    rows = np.unique(np.concatenate([[0, 1, m - 2, m - 1, wrap_row - 1, wrap_row, wrap_row + 1],
                                     _sampled_rows(m, 24)]))
    rows = rows[(rows >= 0) & (rows < m)]
    rows_t = torch.from_numpy(rows).to(DEV)
    rep = parity.compare_search(tensor_bits(W.index_select(0, rows_t)), h.cpu().numpy(), s_g, 2, 2,
                                codes.index_select(0, rows_t).cpu().numpy(),
                                packed.index_select(0, rows_t).cpu().numpy())
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}


def test_search_at_the_32bit_offset_limit(hs):
    """Contiguous arrays are addressed with 32-bit byte offsets up to 2^27
    groups (a 4 GiB W) and with 64-bit ones beyond: W of exactly 2^27 groups
    (32768 x 65536) and of one row more, rows at both ends and around the
    half-way mark checked against the oracle."""
    m, n = 32769, 65536
    print(f"[search offset limit] generating W {m}x{n}", flush=True)
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    W = torch.empty((m, n), dtype=torch.bfloat16, device=DEV)
    for r0 in range(0, m, 4096):  # bounds the fp32 temporary
        r1 = min(m, r0 + 4096)
        W[r0:r1] = (torch.randn((r1 - r0, n), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    h = torch.exp(torch.randn(n, generator=g, device=DEV))
    s_g = harness_global_scale(W)
    h_np = h.cpu().numpy()
    for rows_total in (m - 1, m):
        codes, packed = hs.search(W[:rows_total], h, s_g, window=2)
        torch.cuda.synchronize()
        rows = np.array([0, 1, rows_total // 2 - 1, rows_total // 2, rows_total - 2, rows_total - 1])
        rows_t = torch.from_numpy(rows).to(DEV)
        rep = parity.compare_search(tensor_bits(W.index_select(0, rows_t)), h_np, s_g, 2, 2,
                                    codes.index_select(0, rows_t).cpu().numpy(),
                                    packed.index_select(0, rows_t).cpu().numpy())
        print(f"[search offset limit] rows={rows_total} groups={rows_total * (n // 16)} "
              f"near_ties={rep['near_ties']} mismatches={rep['mismatches']}", flush=True)
        assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}
        del codes, packed


def test_block_layers_small_windows(hs):
    """One layer of each decoder-block shape (q/k/v/o, gate/up, down) with
    its own calibration X, windows 4 and 8, sampled rows."""
    wls = block_workloads(window=4)
    for name in ("k_proj", "gate_proj"):
        wl = wls[name]
        X = make_activations(wl, "cpu", tokens=8192)
        h = torch.from_numpy(parity.oracle_h32(tensor_bits(X))).to(DEV)
        W = make_weight(wl, DEV)
        s_g = harness_global_scale(W)
        for win in (4, 8):
            codes, packed = hs.search(W, h, s_g, window=win)
            rows = _sampled_rows(wl.out, 32)
            rows_t = torch.from_numpy(rows).to(DEV)
            rep = parity.compare_search(tensor_bits(W.index_select(0, rows_t)), h.cpu().numpy(), s_g, win, win,
                                        codes.index_select(0, rows_t).cpu().numpy(),
                                        packed.index_select(0, rows_t).cpu().numpy())
            print(f"[block {name} w={win}] near_ties={rep['near_ties']} mismatches={rep['mismatches']}", flush=True)
            assert rep["ok"]


@pytest.mark.parametrize("down,up", [(9, 6), (8, 7), (8, 8), (12, 11), (12, 12), (15, 0), (0, 15)])
def test_search_class_walk_paths(hs, down, up):
    """Windows of 16..24 candidates walk the residue classes c mod 8 when
    every lane of a wave has only normal, unclipped candidates; a wave with
    one lane near either end of the ladder takes the plain walk.  Both must
    equal the oracle."""
    rng = np.random.default_rng(down * 31 + up)
    m, n = 64, 1024  # 64 groups per row: one wave per row
    w = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    w[5, 3] = 3.0        # row 5: one group with c0 at the top of the ladder
    w[9, :16] *= 1e-3    # row 9: one group with a tiny c0
    W = torch.from_numpy(w).to(torch.bfloat16)
    h = torch.from_numpy(np.exp(rng.standard_normal(n)).astype(np.float32)).to(DEV)
    s_g = harness_global_scale(W)
    c0 = oracle.anchor_codes(tensor_bits(W), s_g, 6.0)
    assert c0[5].max() == 126 and c0[9].min() < 8 + down
    _assert_search_parity(hs, W.to(DEV), h, s_g, down, up, "class walk")
