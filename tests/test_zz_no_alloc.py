"""hscale_hdiag_noalloc, the entry point that allocates nothing (its slice
partials live in the library's static device scratch), against
hscale_hdiag with a caller workspace, both through the C ABI: bit-identical
h on two calls in a row (the second smaller, so stale scratch contents from
the first would show), h within the oracle's 1e-5 bar, and the size limit
rejected before anything is enqueued."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from tests import parity
from synth.workloads import CONFIGS, make_activations, tensor_bits

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"
SCRATCH_BYTES = 8 << 20


@pytest.fixture(scope="module")
def L():
    from paper_2608_28113_amd import _lib
    _lib.load()  # raises if the HIP library is not built: no fallback
    return _lib


def _hdiag_with_workspace(L, X, stream):
    T, n = X.shape
    h = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
    need = L.hscale_hdiag_workspace_bytes(T, n)
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device=DEV)
    assert L.hscale_hdiag(X.data_ptr(), T, n, h.data_ptr(), ws.data_ptr(), need, stream) == 0
    return h


def _hdiag_noalloc(L, X, stream):
    T, n = X.shape
    h = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
    assert L.hscale_hdiag_noalloc(X.data_ptr(), T, n, h.data_ptr(), stream) == 0
    return h


def test_noalloc_equals_workspace_entry_point_two_calls(L):
    stream = torch.cuda.current_stream().cuda_stream
    wl = CONFIGS["down_proj"]
    # First call: the largest partials the plan makes (64 slices x 14336
    # columns = 7.3 MB of the 8 MiB scratch); second call: a smaller,
    # ragged problem that reuses the front of the same scratch.
    cases = [(65536, 14336), (3000, 1040)]
    assert L.hscale_hdiag_workspace_bytes(*cases[0]) > L.hscale_hdiag_workspace_bytes(*cases[1])
    assert L.hscale_hdiag_workspace_bytes(*cases[0]) <= SCRATCH_BYTES
    for k, (T, n) in enumerate(cases):
        print(f"[no-alloc] call {k}: T={T} n={n}", flush=True)
        X = make_activations(wl, DEV, tokens=T, n=n)
        h_na = _hdiag_noalloc(L, X, stream)
        h_ws = _hdiag_with_workspace(L, X, stream)
        torch.cuda.synchronize()
        assert torch.equal(h_na, h_ws), f"call {k}: no-alloc h differs from the workspace entry point"
        # the oracle's bar: every column for the small call, sampled columns
        # for the large one
        cols = np.arange(n) if n <= 2048 else np.unique(np.concatenate(
            [np.random.default_rng(k).choice(n, 64, replace=False), [0, n - 1]]))
        Xs = X.index_select(1, torch.from_numpy(cols).to(DEV)).contiguous()
        rep = parity.compare_h(h_na.cpu().numpy()[cols], oracle.hdiag(tensor_bits(Xs)))
        print(f"[no-alloc] call {k}: max_rel={rep['max_rel']:.2e}", flush=True)
        assert rep["ok"], rep
        del X


def test_noalloc_zero_tokens_and_size_limit(L):
    stream = torch.cuda.current_stream().cuda_stream
    X = torch.empty((0, 64), dtype=torch.bfloat16, device=DEV)
    h = torch.full((64,), 7.0, device=DEV)
    assert L.hscale_hdiag_noalloc(X.data_ptr(), 0, 64, h.data_ptr(), stream) == 0
    torch.cuda.synchronize()
    assert torch.all(h == 0)
    # A problem whose partials exceed the static scratch is refused before
    # any launch (pointers are never dereferenced on that path).
    n = (1 << 20) + 16
    assert L.hscale_hdiag_workspace_bytes(1024, n) > SCRATCH_BYTES
    assert L.hscale_hdiag_noalloc(1 << 20, 1024, n, 1 << 40, stream) == -9


def test_noalloc_replays_in_a_graph(L):
    """The callers this entry point is for include code under HIP graph
    capture: hdiag_noalloc and the search captured together (no buffer is
    allocated during capture, the scratch included), replayed four times;
    between replays an eager hdiag_noalloc of another, smaller X overwrites
    the shared scratch.  Every replay equals the eager results bit for bit."""
    import paper_2608_28113_amd as hs
    from synth.workloads import harness_global_scale, make_weight
    wl = CONFIGS["attn_proj"]
    X = make_activations(wl, DEV, tokens=8192, n=2048)
    X2 = make_activations(wl, DEV, tokens=700, n=1040)
    W = make_weight(wl, DEV, shape=(512, 2048))
    s_g = harness_global_scale(W)
    T, n = X.shape
    m = W.shape[0]
    h = torch.empty(n, dtype=torch.float32, device=DEV)
    h2 = torch.empty(X2.shape[1], dtype=torch.float32, device=DEV)
    codes = torch.empty((m, n // 16), dtype=torch.uint8, device=DEV)
    packed = torch.empty((m, n // 2), dtype=torch.uint8, device=DEV)

    def step(stream):
        assert L.hscale_hdiag_noalloc(X.data_ptr(), T, n, h.data_ptr(), stream.cuda_stream) == 0
        hs.search(W, h, s_g, down=9, up=6, scale_codes=codes, packed_e2m1=packed, stream=stream)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = (h.clone(), codes.clone(), packed.clone())

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        step(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(torch.cuda.current_stream())
    for i in range(4):
        h.zero_()
        codes.zero_()
        packed.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((h, codes, packed), ref):
            assert torch.equal(got, want), f"replay {i}"
        # eager work between replays that reuses the scratch
        stream = torch.cuda.current_stream().cuda_stream
        assert L.hscale_hdiag_noalloc(X2.data_ptr(), X2.shape[0], X2.shape[1], h2.data_ptr(), stream) == 0
        torch.cuda.synchronize()
    assert parity.compare_h(h2.cpu().numpy(), oracle.hdiag(tensor_bits(X2)))["ok"]
