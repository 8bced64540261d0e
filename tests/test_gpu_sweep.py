"""A seeded random sweep of the search against the oracle (Sec. 3.3, Eq. 7,
9-13; App. B for the 4over6 and given-code forms).

Each case draws its own shape (1-69 rows, 1-89 groups per row: ragged
against the 64-lane wave and the 256-lane block), window (0-24 shifts each
way, so both the plain walk and the residue-class walk run), initial-code
rule (max-abs, 4over6, or given code bytes over the whole byte range, which
the search clips), global scale (the harness rule, a power of two that puts
weights on exact E2M1 midpoints, one large enough that codes clamp to 1, one
small enough that they saturate at 126), weights with outliers and all-zero
groups, and h with zeros over a wide dynamic range.  Every fourth case runs
the statistics variant and checks the shift and the two scores as well.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from tests import parity

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"
CASES = 40


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()  # raises if the HIP library is not built: no fallback
    return hs


def _case(i: int):
    rng = np.random.default_rng(7000 + i)
    m = int(rng.integers(1, 70))
    G = int(rng.integers(1, 90))
    n = 16 * G
    down, up = int(rng.integers(0, 25)), int(rng.integers(0, 25))
    if i % 10 == 0:
        down = up = 0  # the initial code alone
    w = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    w[rng.random((m, n)) < 0.01] *= 10.0
    w.reshape(m, G, 16)[rng.random((m, G)) < 0.05] = 0.0
    W = torch.from_numpy(w).to(torch.bfloat16)
    bits = W.view(torch.int16).numpy().view(np.uint16)
    amax = float(W.abs().max().float()) or 1.0
    base = float(np.float32(np.float32(amax) / np.float32(2688.0)))
    rule = i % 4
    if rule == 0:
        s_g = base
    elif rule == 1:
        s_g = float(2.0 ** np.round(np.log2(base)))
    elif rule == 2:
        s_g = float(np.float32(base * 64.0))  # small groups clamp to code 1
    else:
        s_g = float(np.float32(base / 32.0))  # large groups saturate at code 126
    h = rng.lognormal(0.0, 1.5, n).astype(np.float32)
    h[rng.random(n) < 0.05] = 0.0
    kind = ("maxabs", "4over6", "given")[i % 3]
    given = rng.integers(0, 256, (m, G), dtype=np.uint8) if kind == "given" else None
    return W, bits, h, s_g, down, up, kind, given


@pytest.mark.parametrize("i", range(CASES))
def test_search_sweep_matches_oracle(hs, i):
    W, bits, h, s_g, down, up, kind, given = _case(i)
    m, n = W.shape
    print(f"[sweep {i}] m={m} n={n} down={down} up={up} init={kind} s_g={s_g:.3e}", flush=True)
    init_gpu = torch.from_numpy(given).to(DEV) if kind == "given" else kind
    init_oracle = given if kind == "given" else ("rtn" if kind == "maxabs" else "4over6")
    Wd, hd = W.to(DEV), torch.from_numpy(h).to(DEV)
    if i % 4 == 3:
        out = hs.search_stats(Wd, hd, s_g, down, up, init=init_gpu)
        torch.cuda.synchronize()
        gpu = {k: v.cpu().numpy() for k, v in out.items()}
        rep = parity.compare_stats(bits, h, s_g, down, up, gpu, init=init_oracle)
        srep = rep["search"]
        print(f"[sweep {i}] stats: near_ties={srep['near_ties']} mismatches={srep['mismatches']} "
              f"shift_mismatches={rep['shift_mismatches']} err_best_rel={rep['err_best_max_rel']:.2e}", flush=True)
        assert rep["ok"], {k: v for k, v in rep.items() if k != "search"}
    else:
        codes, packed = hs.search(Wd, hd, s_g, down=down, up=up, init=init_gpu)
        torch.cuda.synchronize()
        rep = parity.compare_search(bits, h, s_g, down, up, codes.cpu().numpy(), packed.cpu().numpy(),
                                    init=init_oracle)
        print(f"[sweep {i}] groups={rep['groups']} near_ties={rep['near_ties']} "
              f"mismatches={rep['mismatches']} invalid={rep['invalid']}", flush=True)
        assert rep["ok"], {k: v for k, v in rep.items() if k not in ("oracle", "tie_mask", "init_tie_mask",
                                                                      "err_at_gpu_codes")}
