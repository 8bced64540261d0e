"""The library from several host threads on different streams (the contract
in include/hscale.h: no global state but the no-alloc scratch): two threads,
each with its own stream (default priority), run hdiag and the searches on
their own inputs several times over; every result equals the serial run's
bit for bit."""
from __future__ import annotations

import threading

import pytest
import torch

from synth.workloads import CONFIGS, harness_global_scale, make_activations, make_weight

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

DEV = "cuda"
ROUNDS = 6


@pytest.fixture(scope="module")
def hs():
    import paper_2608_28113_amd as hs
    from paper_2608_28113_amd import _lib
    _lib.load()  # raises if the HIP library is not built: no fallback
    return hs


def _case(seed_shift: int):
    wl = CONFIGS["tiny"]
    X = make_activations(wl, DEV, tokens=8192 + 512 * seed_shift, n=2048 + 512 * seed_shift)
    W = make_weight(wl, DEV, shape=(768 + 128 * seed_shift, X.shape[1]))
    if seed_shift:
        W = (W * 1.5).to(torch.bfloat16)
    return X, W, harness_global_scale(W)


def _run(hs, X, W, s_g, stream):
    h = hs.hdiag(X, stream=stream)
    codes, packed = hs.search(W, h, s_g, down=9, up=6, stream=stream)
    st = hs.search_stats(W, h, s_g, 4, 4, stream=stream)
    return h, codes, packed, st["scale_codes"], st["packed_e2m1"], st["err_best"]


def test_two_host_threads_on_two_streams(hs):
    cases = [_case(0), _case(1)]
    print(f"[concurrency] X {[tuple(c[0].shape) for c in cases]} W {[tuple(c[1].shape) for c in cases]}", flush=True)
    ref = [[t.clone() for t in _run(hs, X, W, s_g, torch.cuda.current_stream())] for X, W, s_g in cases]
    torch.cuda.synchronize()

    results = [[None] * ROUNDS for _ in cases]
    errors = []

    def worker(k):
        try:
            X, W, s_g = cases[k]
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for r in range(ROUNDS):
                    results[k][r] = _run(hs, X, W, s_g, stream)
            stream.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    torch.cuda.synchronize()
    assert not errors, errors
    assert all(not t.is_alive() for t in threads)
    for k in range(len(cases)):
        for r in range(ROUNDS):
            for a, b in zip(results[k][r], ref[k]):
                assert torch.equal(a, b), (k, r)
