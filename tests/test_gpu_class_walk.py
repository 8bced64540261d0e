"""GPU parity of the residue-class walk at exact E2M1 midpoints.

Windows of 16..24 candidates (the paper's [-9, +6] of Sec. 3.3 Eq. 9, and
+-8) walk the residue classes c mod 8 when every lane of a wave has only
normal, unclipped candidates: the products w R of a class base are formed
once and converted at scale operand 2 (or 4) to get candidates c + 8 (or
c + 16).  That equals converting w R[c + 8] (or w R[c + 16]) only if the
conversion divides before it rounds, ties included.  These tests put the
weights on exact E2M1 midpoints of such member candidates (a power-of-two
global scale makes S[c] short), count in numpy how many midpoints reach the
scale-2 and scale-4 conversions, and compare every group with the oracle
through the plain search, the statistics search and the batched search.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import parity

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"
MIDS = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
S_G = 2.0 ** -14
WINDOWS = [(9, 6), (8, 8), (12, 11), (0, 15)]


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()  # raises if the HIP library is not built: no fallback
    return hs


def _bits_to_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(DEV)


def _midpoint_case(seed=11):
    """Groups whose weights sit on E2M1 midpoints of one code c in 48..79
    (half of them exactly, the rest one bf16 ulp to either side), with the
    group's largest midpoint varied so that c lies 1 to ~20 codes above the
    group's initial code.  64 groups per row: one wave per row."""
    S, _ = oracle.scale_tables(S_G)
    rng = np.random.default_rng(seed)
    groups = []
    for c in range(48, 80):
        for k in range(1, 7):  # largest midpoint index of the group
            for _ in range(8):
                idx = rng.integers(0, k + 1, 16)
                idx[rng.integers(0, 16)] = k
                base = (MIDS[idx] * float(S[c])).astype(np.float32)
                u = base.view(np.uint32)
                assert np.all((u & 0xFFFF) == 0)  # S[c] has a short mantissa: these are bf16 values
                ulp = rng.choice([-1, 0, 0, 1], 16)
                bits = ((u >> 16).astype(np.int32) + ulp).astype(np.uint16)
                sign = (rng.integers(0, 2, 16) << 15).astype(np.uint16)
                groups.append(bits | sign)
    Wb = np.stack(groups).reshape(-1, 64 * 16)
    h = np.exp(rng.standard_normal(Wb.shape[1])).astype(np.float32)
    return Wb, h


def _member_midpoints(Wb, down, up):
    """How many weight-candidates reach the class walk's scale-2 and scale-4
    conversions as exact E2M1 midpoints (x = fp32(|w| R[c]) of the member
    candidate c), and whether every wave takes the class walk."""
    m, n = Wb.shape
    G = n // 16
    c0 = oracle.anchor_codes(Wb, S_G, 6.0).astype(np.int64)
    K = down + up + 1
    waves = c0.reshape(-1, 64)
    class_walk = bool(16 <= K <= 24 and np.all(waves - down >= 8) and np.all(waves + up <= 126))
    _, R = oracle.scale_tables(S_G)
    w = np.abs(parity_weights(Wb)).reshape(m, G, 16)
    counts = {}
    for mult in (1, 2):
        hits = 0
        for d0 in range(-down, -down + min(K, 8)):
            d = d0 + 8 * mult
            if d > up:
                continue
            x = (w * R[(c0 + d)][:, :, None]).astype(np.float32)
            hits += int(np.isin(x, MIDS.astype(np.float32)).sum())
        counts[2 ** mult] = hits
    return class_walk, counts


def parity_weights(Wb):
    return (Wb.astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("down,up", WINDOWS)
def test_class_walk_exact_midpoints(hs, down, up):
    Wb, h32 = _midpoint_case()
    class_walk, counts = _member_midpoints(Wb, down, up)
    print(f"[class walk midpoints] down={down} up={up} class_walk={class_walk} "
          f"scale2_midpoints={counts[2]} scale4_midpoints={counts[4]}", flush=True)
    assert class_walk, "every wave must take the residue-class walk"
    assert counts[2] > 500
    if up - (-down) >= 16:  # some class has a third member
        assert counts[4] > 50
    W = _bits_to_bf16(Wb)
    h = torch.from_numpy(h32).to(DEV)

    codes, packed = hs.search(W, h, S_G, down=down, up=up)
    rep = parity.compare_search(Wb, h32, S_G, down, up, codes.cpu().numpy(), packed.cpu().numpy())
    print(f"[class walk midpoints] search groups={rep['groups']} near_ties={rep['near_ties']} "
          f"mismatches={rep['mismatches']}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k not in ("oracle", "tie_mask", "init_tie_mask",
                                                                 "err_at_gpu_codes")}

    st = hs.search_stats(W, h, S_G, down, up)
    srep = parity.compare_stats(Wb, h32, S_G, down, up, {k: v.cpu().numpy() for k, v in st.items()})
    print(f"[class walk midpoints] stats shift_mismatches={srep['shift_mismatches']} "
          f"err_best_max_rel={srep['err_best_max_rel']:.2e}", flush=True)
    assert srep["ok"], {k: v for k, v in srep.items() if k != "search"}
    assert torch.equal(st["scale_codes"], codes) and torch.equal(st["packed_e2m1"], packed)

    # The batched search: this layer twice (once sign-flipped) in one launch.
    Wn = _bits_to_bf16(Wb ^ np.uint16(0x8000))
    out = hs.search_layers([(W, h, S_G), (Wn, h, S_G)], down=down, up=up)
    torch.cuda.synchronize()
    assert torch.equal(out[0][0], codes) and torch.equal(out[0][1], packed)
    assert torch.equal(out[1][0], codes)
    assert torch.equal(out[1][1], packed ^ 0x88)


def test_class_walk_overflowing_scores_keep_a_real_candidate(hs):
    """Finite but huge h makes every candidate's fp32 score overflow to +Inf.
    The walk must then report the smallest shift (the first candidate, as
    the plain walk does) with the packed codes of that very code, also for
    a window that starts at the initial code (down = 0)."""
    rng = np.random.default_rng(21)
    m, n = 32, 1024
    w = (rng.standard_normal((m, n)) * 30.0).astype(np.float32)
    W = torch.from_numpy(w).to(torch.bfloat16)
    Wb = W.view(torch.int16).numpy().view(np.uint16)
    s_g = float(np.float32(np.float32(np.abs(w).max()) / np.float32(600.0)))
    h32 = np.full(n, 3.0e38, np.float32)
    c0 = oracle.anchor_codes(Wb, s_g, 6.0).astype(np.int64)
    for down, up in ((0, 15), (9, 6), (8, 8)):
        waves = c0.reshape(-1, 64)
        assert np.all(waves - down >= 8) and np.all(waves + up <= 126)  # class walk in every wave
        codes, packed = hs.search(W.to(DEV), torch.from_numpy(h32).to(DEV), s_g, down=down, up=up)
        codes = codes.cpu().numpy()
        want = np.clip(c0 - down, 1, 126).astype(np.uint8)
        assert np.array_equal(codes, want), (down, up)
        at, _ = oracle.quantize(Wb, s_g, codes)
        assert np.array_equal(packed.cpu().numpy(), at), (down, up)
        st = hs.search_stats(W.to(DEV), torch.from_numpy(h32).to(DEV), s_g, down, up)
        assert torch.all(st["shift"] == -down)
        assert torch.all(torch.isinf(st["err_best"]))
