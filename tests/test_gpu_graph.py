"""The entry points enqueue only kernels on the caller's stream (no
allocation, synchronisation or memset inside), so a caller can capture them
in a HIP graph.  The graph is replayed several times with eager work and
synchronisations between replays, and every replay must equal the eager
results bit for bit."""
from __future__ import annotations

import pytest
import torch

from synth.workloads import CONFIGS, harness_global_scale, make_activations, make_weight

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()
    return hs


def test_hdiag_search_and_output_error_replay_in_a_graph(hs):
    wl = CONFIGS["attn_proj"]
    X = make_activations(wl, DEV, tokens=8192, n=2048)
    W = make_weight(wl, DEV, shape=(1024, 2048))
    s_g = harness_global_scale(W)
    T, n = X.shape
    m = W.shape[0]
    # every buffer is allocated before capture
    h = torch.empty(n, dtype=torch.float32, device=DEV)
    ws_h = torch.empty(hs.hdiag_workspace_bytes(T, n), dtype=torch.uint8, device=DEV)
    codes = torch.empty((m, n // 16), dtype=torch.uint8, device=DEV)
    packed = torch.empty((m, n // 2), dtype=torch.uint8, device=DEV)
    row = torch.empty(m, dtype=torch.float64, device=DEV)
    ws_l = torch.empty(hs.output_error_workspace_bytes(T, n, m), dtype=torch.uint8, device=DEV)

    def step(stream=None):
        hs.hdiag(X, h=h, workspace=ws_h, stream=stream)
        hs.search(W, h, s_g, down=9, up=6, scale_codes=codes, packed_e2m1=packed, stream=stream)
        row.fill_(0.0)  # a fill kernel, not a memset node
        hs.output_error(X, W, s_g, codes, packed, row_err=row, workspace=ws_l, stream=stream)

    step()
    torch.cuda.synchronize()
    ref = (h.clone(), codes.clone(), packed.clone(), row.clone())

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for i in range(4):
        h.zero_()
        codes.zero_()
        packed.zero_()
        row.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((h, codes, packed, row), ref):
            assert torch.equal(got, want), f"replay {i}"
        # eager work between replays
        X.mul_(1.0)
        torch.cuda.synchronize()
