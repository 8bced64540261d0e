"""GPU parity of the batched search (hscale_search_layers): every layer of a
batch against the oracle, and bit for bit against the single-layer search of
the same layer, including batches of more than one launch (over 32 layers),
empty layers, a shared h and in-place refinement of given codes."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import parity
from synth.workloads import block_workloads, harness_global_scale, make_weight, tensor_bits

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()
    return hs


def _layer(seed, m, n, std=0.02):
    """W ~ N(0, std^2) with 1% of entries x10 (bf16), h log-normal (fp32)."""
    g = torch.Generator().manual_seed(seed)
    w = torch.randn((m, n), generator=g) * std
    mask = torch.rand((m, n), generator=g) < 0.01
    w[mask] *= 10.0
    W = w.to(torch.bfloat16)
    h = torch.exp(torch.randn(n, generator=g))
    return W.to(DEV), h.to(DEV), harness_global_scale(W)


SHAPES = [(256, 512), (77, 1040), (3, 48), (1000, 592), (1, 16), (40, 4096)]


def _given_codes(seed, W, s_g):
    rng = np.random.default_rng(seed)
    base = oracle.anchor_codes(tensor_bits(W), s_g, 6.0).astype(np.int64)
    return np.clip(base + rng.integers(-5, 6, base.shape), 0, 255).astype(np.uint8)


def _check_layer(W, h, s_g, down, up, codes, packed, init, label):
    rep = parity.compare_search(tensor_bits(W), h.cpu().numpy(), s_g, down, up, codes.cpu().numpy(),
                                packed.cpu().numpy(), init=init)
    print(f"[{label}] groups={rep['groups']} near_ties={rep['near_ties']} mismatches={rep['mismatches']}",
          flush=True)
    assert rep["ok"], {k: v for k, v in rep.items() if k != "oracle"}


@pytest.mark.parametrize("init", ["maxabs", "4over6", "given"])
@pytest.mark.parametrize("down,up", [(4, 4), (9, 6), (0, 0)])
def test_layers_match_the_oracle(hs, init, down, up):
    layers = [_layer(k, m, n) for k, (m, n) in enumerate(SHAPES)]
    if init == "given":
        given = [_given_codes(k, W, s) for k, (W, _, s) in enumerate(layers)]
        outs = hs.search_layers(layers, down=down, up=up, init=[torch.from_numpy(c).to(DEV) for c in given])
        inits = given
    else:
        outs = hs.search_layers(layers, down=down, up=up, init=init)
        inits = ["rtn" if init == "maxabs" else init] * len(layers)
    torch.cuda.synchronize()
    for k, ((W, h, s), (codes, packed)) in enumerate(zip(layers, outs)):
        _check_layer(W, h, s, down, up, codes, packed, inits[k], f"layers {init} {down},{up} layer {k}")


def test_layers_equal_single_layer_searches_on_a_decoder_block(hs):
    """The seven layers of the 8B-class decoder block (q/o 4096x4096, k/v
    1024x4096, gate/up 14336x4096, down 4096x14336) with q/k/v/o and
    gate/up sharing an h: the batched result equals each layer's own search
    bit for bit; sampled rows of each layer against the oracle."""
    wls = block_workloads(window=4)
    hkey = {"q_proj": "attn", "k_proj": "attn", "v_proj": "attn", "o_proj": "attn", "gate_proj": "mlp",
            "up_proj": "mlp", "down_proj": "down"}
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    hs_by_key = {}
    layers = []
    for name, wl in wls.items():
        if hkey[name] not in hs_by_key:
            hs_by_key[hkey[name]] = torch.exp(torch.randn(wl.inp, generator=g, device=DEV))
        W = make_weight(wl, DEV)
        layers.append((W, hs_by_key[hkey[name]], harness_global_scale(W)))
    for win in (4, 8):
        outs = hs.search_layers(layers, window=win)
        for (name, (W, h, s)), (codes, packed) in zip(zip(wls, layers), outs):
            c1, p1 = hs.search(W, h, s, window=win)
            torch.cuda.synchronize()
            assert torch.equal(codes, c1) and torch.equal(packed, p1), (name, win)
            rows = np.unique(np.linspace(0, W.shape[0] - 1, 6).astype(np.int64))
            rows_t = torch.from_numpy(rows).to(DEV)
            rep = parity.compare_search(tensor_bits(W.index_select(0, rows_t)), h.cpu().numpy(), s, win, win,
                                        codes.index_select(0, rows_t).cpu().numpy(),
                                        packed.index_select(0, rows_t).cpu().numpy())
            print(f"[layers block {name} w={win}] near_ties={rep['near_ties']} mismatches={rep['mismatches']}",
                  flush=True)
            assert rep["ok"]
        del outs


def test_layers_beyond_one_launch_with_empty_layers(hs):
    """71 layers (three launches of at most 32) of varied small shapes, with
    empty layers among them, all against the oracle."""
    rng = np.random.default_rng(3)
    shapes = []
    for k in range(71):
        if k % 10 == 4:
            shapes.append((0, 64) if k % 20 == 4 else (5, 0))
        else:
            shapes.append((int(rng.integers(1, 40)), 16 * int(rng.integers(1, 40))))
    layers = []
    for k, (m, n) in enumerate(shapes):
        if m == 0 or n == 0:
            W = torch.empty((m, n), dtype=torch.bfloat16, device=DEV)
            layers.append((W, torch.ones(n, device=DEV), 1e-3))
        else:
            layers.append(_layer(100 + k, m, n))
    outs = hs.search_layers(layers, down=3, up=5)
    torch.cuda.synchronize()
    for k, ((W, h, s), (codes, packed)) in enumerate(zip(layers, outs)):
        if W.numel() == 0:
            assert codes.numel() == 0 and packed.numel() == 0
            continue
        _check_layer(W, h, s, 3, 5, codes, packed, "rtn", f"layers many {k}")


def test_layers_refine_in_place(hs):
    """Given codes refined in place (each layer's init tensor is its own
    output), as a blockwise pipeline would: equals the search from a copy."""
    layers = [_layer(200 + k, m, n) for k, (m, n) in enumerate(SHAPES[:4])]
    given = [torch.from_numpy(_given_codes(7 + k, W, s)).to(DEV) for k, (W, _, s) in enumerate(layers)]
    ref = hs.search_layers(layers, window=4, init=[c.clone() for c in given])
    outs = hs.search_layers(layers, window=4, init=given,
                            outputs=[(c, torch.empty((W.shape[0], W.shape[1] // 2), dtype=torch.uint8,
                                                     device=DEV)) for c, (W, _, _) in zip(given, layers)])
    torch.cuda.synchronize()
    for (c0, p0), (c1, p1), g in zip(ref, outs, given):
        assert c1.data_ptr() == g.data_ptr()
        assert torch.equal(c0, c1) and torch.equal(p0, p1)
