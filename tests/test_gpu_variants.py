"""GPU parity of the search variants: the 4over6 initial code, baseline-
provided initial codes, the strided column-block form used blockwise as in
the paper's GPTQ combination, and h accumulated over streamed batches."""
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
    h = torch.from_numpy(parity.oracle_h32(tensor_bits(make_activations(wl, "cpu")))).to(DEV)
    return W.to(DEV), h, harness_global_scale(W)


def _check(W, h, s_g, down, up, codes, packed, init, label):
    torch.cuda.synchronize()
    rep = parity.compare_search(tensor_bits(W), h.cpu().numpy(), s_g, down, up, codes.cpu().numpy(),
                                packed.cpu().numpy(), init=init)
    print(f"[{label}] down={down} up={up} groups={rep['groups']} near_ties={rep['near_ties']} "
          f"init_ties={rep['init_ties']} mismatches={rep['mismatches']} invalid={rep['invalid']}", flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}


@pytest.mark.parametrize("down,up", [(0, 0), (4, 4), (9, 6), (8, 8)])
def test_4over6_tiny_parity(hs, tiny, down, up):
    W, h, s_g = tiny
    codes, packed = hs.search(W, h, s_g, down=down, up=up, init="4over6")
    _check(W, h, s_g, down, up, codes, packed, "4over6", "4over6 tiny")


def test_4over6_window0_is_the_4over6_quantizer(hs, tiny):
    W, h, s_g = tiny
    codes, packed = hs.search(W, h, s_g, window=0, init="4over6")
    c4 = oracle.anchor_codes(tensor_bits(W), s_g, 4.0)
    c6 = oracle.anchor_codes(tensor_bits(W), s_g, 6.0)
    c = codes.cpu().numpy()
    assert np.all((c == c4) | (c == c6))
    assert 0.05 < np.mean(c == c4) < 0.95


def test_4over6_full_size_sampled(hs):
    wl = CONFIGS["down_proj"]
    h = torch.from_numpy(parity.oracle_h32(tensor_bits(make_activations(wl, "cpu", tokens=4096)))).to(DEV)
    W = make_weight(wl, DEV)
    s_g = harness_global_scale(W)
    codes, packed = hs.search(W, h, s_g, down=9, up=6, init="4over6")
    rows = torch.from_numpy(np.unique(np.r_[np.random.default_rng(1).choice(wl.out, 48, replace=False),
                                            0, wl.out - 1])).to(DEV)
    _check(W.index_select(0, rows), h, s_g, 9, 6, codes.index_select(0, rows), packed.index_select(0, rows),
           "4over6", "4over6 down_proj")


@pytest.mark.parametrize("down,up", [(0, 0), (4, 4), (9, 6)])
def test_search_from_given_codes(hs, tiny, down, up):
    W, h, s_g = tiny
    m, n = W.shape
    rng = np.random.default_rng(down * 10 + up)
    base = oracle.anchor_codes(tensor_bits(W), s_g, 6.0).astype(np.int64)
    init = np.clip(base + rng.integers(-6, 7, base.shape), 0, 255).astype(np.uint8)
    init[0, :4] = (0, 127, 200, 255)  # outside the ladder: clipped
    init_t = torch.from_numpy(init).to(DEV)
    codes, packed = hs.search(W, h, s_g, down=down, up=up, init=init_t)
    _check(W, h, s_g, down, up, codes, packed, init, "given init")


def test_search_from_in_place_and_equivalence(hs, tiny):
    W, h, s_g = tiny
    c_ref, p_ref = hs.search(W, h, s_g, window=4)
    # initial codes = max-abs codes gives the max-abs search
    c0, _ = hs.search(W, h, s_g, window=0)
    c1, p1 = hs.search(W, h, s_g, window=4, init=c0.clone())
    assert torch.equal(c1, c_ref) and torch.equal(p1, p_ref)
    # refine in place: codes buffer is also the initial codes
    buf = c0.clone()
    hs.search(W, h, s_g, window=4, init=buf, scale_codes=buf)
    torch.cuda.synchronize()
    assert torch.equal(buf, c_ref)


def test_search_block_strided(hs):
    """A column block of a wider matrix with padded rows: only the block's
    codes and bytes are written, and they equal the oracle's on the block."""
    wl = CONFIGS["tiny"]
    m, N, pad = 96, 1024, 64
    a, b = 256, 640
    full = make_weight(wl, "cpu", shape=(m, N + pad)).to(DEV)
    Wfull = full[:, :N]  # row stride N + pad
    h = torch.exp(torch.randn(N, device=DEV))
    s_g = harness_global_scale(Wfull)
    codes = torch.full((m, N // 16 + 3), 0xAB, dtype=torch.uint8, device=DEV)
    packed = torch.full((m, N // 2 + 8), 0xCD, dtype=torch.uint8, device=DEV)
    cv = codes[:, a // 16:b // 16]
    pv = packed[:, a // 2:b // 2]
    hs.search_block(Wfull[:, a:b], h[a:b].contiguous(), s_g, 4, 4, cv, pv)
    torch.cuda.synchronize()
    c = codes.cpu().numpy()
    p = packed.cpu().numpy()
    assert np.all(c[:, :a // 16] == 0xAB) and np.all(c[:, b // 16:] == 0xAB)
    assert np.all(p[:, :a // 2] == 0xCD) and np.all(p[:, b // 2:] == 0xCD)
    Wb = tensor_bits(Wfull[:, a:b].contiguous())
    rep = parity.compare_search(Wb, h[a:b].cpu().numpy(), s_g, 4, 4, c[:, a // 16:b // 16],
                                p[:, a // 2:b // 2])
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}


@pytest.mark.parametrize("init", ["maxabs", "4over6"])
def test_blockwise_loop_equals_whole_matrix(hs, init):
    """The paper's GPTQ combination searches one column block at a time with
    the layer's fixed s_g; without error propagation the blockwise result
    must equal one search of the whole matrix."""
    wl = CONFIGS["attn_proj"]
    W = make_weight(wl, DEV, shape=(512, 4096))
    h = torch.exp(torch.randn(4096, device=DEV))
    s_g = harness_global_scale(W)
    c_ref, p_ref = hs.search(W, h, s_g, down=9, up=6, init=init)
    codes = torch.empty_like(c_ref)
    packed = torch.empty_like(p_ref)
    B = 128
    for i in range(0, 4096, B):
        hs.search_block(W[:, i:i + B], h[i:i + B].contiguous(), s_g, 9, 6, codes[:, i // 16:(i + B) // 16],
                        packed[:, i // 2:(i + B) // 2], init=init)
    torch.cuda.synchronize()
    assert torch.equal(codes, c_ref) and torch.equal(packed, p_ref)


def test_hdiag_accumulate_and_finalize(hs):
    wl = CONFIGS["attn_proj"]
    X = make_activations(wl, DEV, tokens=50000, n=1040)
    h_ref = hs.hdiag(X)
    h64 = torch.zeros(1040, dtype=torch.float64, device=DEV)
    hs.hdiag_accumulate(X, h64)
    assert torch.equal(hs.hdiag_finalize(h64), h_ref)  # one batch: identical to hdiag
    h64.zero_()
    cuts = [0, 1, 777, 20000, 20001, 50000]
    for a, b in zip(cuts[:-1], cuts[1:]):
        hs.hdiag_accumulate(X[a:b].contiguous(), h64)
    hs.hdiag_accumulate(X[:0], h64)  # empty batch: no change
    h = hs.hdiag_finalize(h64)
    torch.cuda.synchronize()
    ref = oracle.hdiag(tensor_bits(X))
    rep = parity.compare_h(h.cpu().numpy(), ref)
    assert rep["ok"] and rep["max_rel"] <= 2e-6, rep
    assert np.allclose(h64.cpu().numpy(), ref, rtol=2e-6)
