"""The C ABI loads, exports what include/hscale.h declares, and rejects bad
arguments on the host before any launch (these run without a GPU: no path
exercised here reaches the HIP runtime)."""
import re
import subprocess
from pathlib import Path

import numpy as np
import pytest

ROOT = Path(__file__).resolve().parent.parent
HEADER = ROOT / "include" / "hscale.h"


@pytest.fixture(scope="module")
def L():
    from paper_2608_28113_amd import _lib
    if not _lib.LIB_PATH.exists():
        from paper_2608_28113_amd import build
        build.build()
    _lib.load()
    return _lib


def _declared():
    text = HEADER.read_text()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|size_t|int)\s*\**\s*(hscale_\w+)\s*\(", text, re.M)))


def test_header_declarations_match_binding(L):
    assert _declared() == sorted(L.EXPORTS)


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", str(L.LIB_PATH)], capture_output=True, text=True,
                         check=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in _declared():
        assert name in syms, name


def test_status_strings(L):
    for code, name in L.STATUS.items():
        assert L.status_string(code).startswith(name)
    assert "unknown" in L.status_string(12345)


def test_workspace_bytes(L):
    assert L.hscale_hdiag_workspace_bytes(0, 4096) == 0
    assert L.hscale_hdiag_workspace_bytes(100, 15) == 0
    assert L.hscale_hdiag_workspace_bytes(-1, 16) == 0
    for T, n in ((128, 512), (262144, 4096), (262144, 14336), (131072, 28672), (1, 16)):
        b = L.hscale_hdiag_workspace_bytes(T, n)
        assert b > 0 and b % (8 * n) == 0
        slices = b // (8 * n)
        assert 1 <= slices <= T
        assert b <= 0.02 * 2 * T * n or T * n < 1 << 20  # partials are a small fraction of X


# Fake but aligned device addresses: validation never dereferences them.
A = 1 << 20


def test_hdiag_validation(L):
    ws = L.hscale_hdiag_workspace_bytes(64, 32)
    assert L.hscale_hdiag(A, 64, 33, 2 * A, 3 * A, ws, 0) == -2
    assert L.hscale_hdiag(A, -1, 32, 2 * A, 3 * A, ws, 0) == -2
    assert L.hscale_hdiag(A, 64, -16, 2 * A, 3 * A, ws, 0) == -2
    assert L.hscale_hdiag(0, 64, 32, 2 * A, 3 * A, ws, 0) == -1
    assert L.hscale_hdiag(A, 64, 32, 0, 3 * A, ws, 0) == -1
    assert L.hscale_hdiag(A, 64, 32, 2 * A, 0, ws, 0) == -1
    assert L.hscale_hdiag(A + 8, 64, 32, 2 * A, 3 * A, ws, 0) == -3
    assert L.hscale_hdiag(A, 64, 32, 2 * A + 2, 3 * A, ws, 0) == -3
    assert L.hscale_hdiag(A, 64, 32, 2 * A, 3 * A + 8, ws, 0) == -3
    assert L.hscale_hdiag(A, 64, 32, 2 * A, 3 * A, ws - 1, 0) == -6
    # h inside X, workspace inside X
    assert L.hscale_hdiag(A, 64, 32, A + 64, 3 * A, ws, 0) == -8
    assert L.hscale_hdiag(A, 64, 32, 2 * A, A + 1024, ws, 0) == -8
    # in == 0 is a no-op
    assert L.hscale_hdiag(0, 64, 0, 0, 0, 0, 0) == 0


def test_hdiag_noalloc_validation(L):
    """The static-scratch entry point checks its arguments, and the scratch
    limit, before its first HIP call (so these run without a GPU)."""
    assert L.hscale_hdiag_noalloc(A, 64, 33, 2 * A, 0) == -2
    assert L.hscale_hdiag_noalloc(A, -1, 32, 2 * A, 0) == -2
    assert L.hscale_hdiag_noalloc(0, 64, 32, 2 * A, 0) == -1
    assert L.hscale_hdiag_noalloc(A, 64, 32, 0, 0) == -1
    assert L.hscale_hdiag_noalloc(A + 8, 64, 32, 2 * A, 0) == -3
    assert L.hscale_hdiag_noalloc(A, 64, 32, 2 * A + 2, 0) == -3
    assert L.hscale_hdiag_noalloc(A, 64, 32, A + 64, 0) == -8
    assert L.hscale_hdiag_noalloc(0, 64, 0, 0, 0) == 0
    # every plan with in <= 2^20 columns fits the 8 MiB scratch; wider
    # problems are refused with HSCALE_ERR_SCRATCH
    limit = 8 << 20
    for n in (16, 512, 528, 14336, 28672, 917504, 917520, 1 << 20):
        for T in (1, 256, 4096, 262144, 1 << 24):
            assert L.hscale_hdiag_workspace_bytes(T, n) <= limit, (T, n)
    n = (1 << 20) + 16
    assert L.hscale_hdiag_workspace_bytes(1, n) > limit
    assert L.hscale_hdiag_noalloc(A, 1, n, 1 << 40, 0) == -9
    assert L.status_string(-9).startswith("HSCALE_ERR_SCRATCH")
    assert L.status_string(-10).startswith("HSCALE_ERR_DEVICE")


def test_search_validation(L):
    m, n = 4, 64
    W, h, codes, packed = A, 2 * A, 3 * A, 4 * A
    ok = dict(W=W, h=h, codes=codes, packed=packed)

    def call(W=W, out=m, in_=n, h=h, window=4, s=1e-3, codes=codes, packed=packed):
        return L.hscale_search(W, out, in_, h, window, s, codes, packed, 0)

    assert call(in_=65) == -2
    assert call(out=-1) == -2
    assert call(in_=-16) == -2
    assert call(out=1 << 40, in_=1 << 10) == -2
    assert call(window=-1) == -4
    assert call(window=126) == -4
    for s in (0.0, -1.0, float("inf"), float("nan"), 1e-40, 2.0 ** -118, 1e36):
        assert call(s=s) == -5, s
    assert call(W=0) == -1
    assert call(h=0) == -1
    assert call(codes=0) == -1
    assert call(packed=0) == -1
    assert call(W=W + 2) == -3
    assert call(h=h + 4) == -3
    assert call(packed=packed + 4) == -3
    assert call(codes=W + 16) == -8
    assert call(packed=h) == -8
    assert call(codes=packed + 8) == -8
    # empty problems are no-ops (no pointer needed)
    assert L.hscale_search(0, 0, n, 0, 4, 1e-3, 0, 0, 0) == 0
    assert L.hscale_search(0, m, 0, 0, 4, 1e-3, 0, 0, 0) == 0
    assert L.hscale_search_du(W, m, n, h, 9, 126, 1e-3, codes, packed, 0) == -4
    assert L.hscale_search_du(W, m, n, h, -1, 6, 1e-3, codes, packed, 0) == -4


def test_quantize_validation(L):
    m, n = 4, 64
    W, codes, packed = A, 2 * A, 3 * A
    assert L.hscale_quantize(W, m, 17, 1e-3, codes, packed, 0) == -2
    assert L.hscale_quantize(W, m, n, 0.0, codes, packed, 0) == -5
    assert L.hscale_quantize(0, m, n, 1e-3, codes, packed, 0) == -1
    assert L.hscale_quantize(W, m, n, 1e-3, 0, packed, 0) == -1
    assert L.hscale_quantize(W + 4, m, n, 1e-3, codes, packed, 0) == -3
    assert L.hscale_quantize(W, m, n, 1e-3, codes, W + 32, 0) == -8
    assert L.hscale_quantize(0, 0, n, 1e-3, 0, 0, 0) == 0


def test_torch_front_end_rejects_bad_tensors():
    import torch
    from paper_2608_28113_amd import ops
    with pytest.raises(ValueError):
        ops.hdiag(torch.zeros(4, 16, dtype=torch.float32))
    with pytest.raises(ValueError):
        ops.search(torch.zeros(4, 16, dtype=torch.bfloat16), torch.zeros(16), 1e-3, window=4)


def test_variant_validation(L):
    m, n = 4, 64
    W, h, codes, packed, init, h64 = A, 2 * A, 3 * A, 4 * A, 5 * A, 6 * A
    # Every call here must fail validation (or be empty) so that nothing is
    # launched: the addresses are fake.  4over6 and given-init share the
    # search validation.
    assert L.hscale_search_4over6(W, m, n, h, 9, 126, 1e-3, codes, packed, 0) == -4
    assert L.hscale_search_4over6(W, m, 17, h, 9, 6, 1e-3, codes, packed, 0) == -2
    assert L.hscale_search_from(W, m, n, h, 4, 4, 1e-3, 0, codes, packed, 0) == -1
    assert L.hscale_search_from(W, m, n, h, 4, 4, 1e-3, codes + 1, codes, packed, 0) == -8  # partial overlap
    assert L.hscale_search_from(W, m, n, h, 4, 4, 0.0, init, codes, packed, 0) == -5
    # strided block
    blk = lambda **k: L.hscale_search_block(k.get("W", W), k.get("ldw", 128), k.get("out", m), k.get("cols", n),
                                            h, 4, 4, 1e-3, k.get("mode", 0), k.get("init", 0), k.get("ldi", 0),
                                            codes, k.get("ldc", 8), packed, k.get("ldp", 64), 0)
    assert blk(cols=48 + 8) == -2
    assert blk(ldw=32) == -2            # ldw < cols
    assert blk(ldw=68) == -3            # rows not 16-byte aligned
    assert blk(ldc=3) == -2
    assert blk(ldp=31) == -2
    assert blk(ldp=36) == -3            # packed rows not 8-byte aligned
    assert blk(mode=3) == -2
    assert blk(mode=2, ldi=4) == -1     # given init without codes
    assert blk(mode=2, init=init, ldi=2) == -2
    assert blk(out=0) == 0
    # accumulate / finalize
    ws = L.hscale_hdiag_workspace_bytes(64, 32)
    assert L.hscale_hdiag_accumulate(A, 64, 32, 0, 3 * A, ws, 0) == -1
    assert L.hscale_hdiag_accumulate(A, 64, 32, h64 + 4, 3 * A, ws, 0) == -3
    assert L.hscale_hdiag_accumulate(A, 64, 33, h64, 3 * A, ws, 0) == -2
    assert L.hscale_hdiag_accumulate(A, 64, 32, A + 8, 3 * A, ws, 0) == -8
    assert L.hscale_hdiag_accumulate(0, 0, 32, h64, 0, 0, 0) == 0  # empty batch: no-op, no launch
    assert L.hscale_hdiag_finalize(0, 32, h, 0) == -1
    assert L.hscale_hdiag_finalize(h64, 33, h, 0) == -2
    assert L.hscale_hdiag_finalize(h64, 32, h64 + 64, 0) == -8
    assert L.hscale_hdiag_finalize(0, 0, 0, 0) == 0


def test_stats_and_summary_validation(L):
    m, n = 4, 64
    W, h, codes, packed, sh, eb, ei = A, 2 * A, 3 * A, 4 * A, 5 * A, 6 * A, 7 * A

    def st(**k):
        return L.hscale_search_stats(W, m, n, h, 4, 4, 1e-3, k.get("mode", 0), k.get("init", 0), codes, packed,
                                     k.get("sh", sh), k.get("eb", eb), k.get("ei", ei), 0)
    # every call fails validation: nothing is launched on the fake addresses
    assert st(sh=0) == -1
    assert st(eb=0) == -1
    assert st(ei=0) == -1
    assert st(eb=eb + 2) == -3
    assert st(mode=2) == -1
    assert st(ei=eb + 8) == -8          # err arrays overlap
    assert st(sh=W + 16) == -8          # statistics overlap W
    assert st(eb=codes) == -8           # statistics overlap the codes
    assert L.hscale_search_stats(W, m, n, h, 126, 4, 1e-3, 0, 0, codes, packed, sh, eb, ei, 0) == -4

    assert L.hscale_shift_summary_workspace_bytes(0, 4, 4) == 0
    assert L.hscale_shift_summary_workspace_bytes(-5, 4, 4) == 0
    assert L.hscale_shift_summary_workspace_bytes(10, -1, 4) == 0
    b1 = L.hscale_shift_summary_workspace_bytes(1, 4, 4)
    b2 = L.hscale_shift_summary_workspace_bytes(4097, 4, 4)
    assert b1 > 0 and b2 == 2 * b1 and L.hscale_shift_summary_workspace_bytes(1, 9, 6) > b1

    cnt, si, sb, sr, ws = 8 * A, 9 * A, 10 * A, 11 * A, 12 * A
    need = L.hscale_shift_summary_workspace_bytes(1000, 4, 4)

    def su(groups=1000, down=4, up=4, **k):
        return L.hscale_shift_summary(k.get("sh", sh), k.get("eb", eb), k.get("ei", ei), groups, down, up,
                                      k.get("cnt", cnt), k.get("si", si), k.get("sb", sb), k.get("sr", sr),
                                      k.get("ws", ws), k.get("wsb", need), 0)
    assert su(groups=-1) == -2
    assert su(groups=1 << 33) == -2
    assert su(down=-1) == -4
    assert su(up=126) == -4
    assert su(cnt=0) == -1
    assert su(sr=0) == -1
    assert su(sh=0) == -1
    assert su(ws=0) == -1
    assert su(wsb=need - 1) == -6
    assert su(cnt=cnt + 4) == -3
    assert su(eb=eb + 2) == -3
    assert su(ws=ws + 4) == -3
    assert su(si=cnt + 8) == -8         # outputs overlap
    assert su(sb=eb) == -8              # output overlaps an input
    assert su(ws=sh) == -8              # workspace overlaps an input


def test_output_error_validation(L):
    T, n, m = 64, 64, 8
    X, W, codes, packed, row, ws = A, 2 * A, 3 * A, 4 * A, 5 * A, 6 * A
    need = L.hscale_output_error_workspace_bytes(T, n, m)
    assert need > 0 and need % 8 == 0
    assert L.hscale_output_error_workspace_bytes(0, n, m) == 0
    assert L.hscale_output_error_workspace_bytes(T, 17, m) == 0
    # the workspace is bounded: more than one pass of token tiles reuses it
    assert L.hscale_output_error_workspace_bytes(10 ** 7, n, m) == L.hscale_output_error_workspace_bytes(2 ** 20, n, m)

    def oe(**k):
        return L.hscale_output_error(k.get("X", X), k.get("T", T), k.get("n", n), k.get("W", W), k.get("m", m),
                                     k.get("s", 1e-3), k.get("codes", codes), k.get("packed", packed),
                                     k.get("row", row), k.get("ws", ws), k.get("wsb", need), 0)
    # every call fails validation: nothing is launched on the fake addresses
    assert oe(n=17) == -2
    assert oe(T=-1) == -2
    assert oe(m=-3) == -2
    # a tile of X is addressed with 32-bit offsets: in <= 2^21
    assert L.hscale_output_error_workspace_bytes(T, 2 ** 21 + 16, 1) == 0
    assert L.hscale_output_error_workspace_bytes(1, 2 ** 21, 1) > 0
    assert oe(n=2 ** 21 + 16, m=1, T=1) == -2
    assert oe(s=0.0) == -5
    assert oe(X=0) == -1
    assert oe(row=0) == -1
    assert oe(ws=0) == -1
    assert oe(X=X + 8) == -3
    assert oe(W=W + 2) == -3
    assert oe(packed=packed + 4) == -3
    assert oe(row=row + 4) == -3
    assert oe(ws=ws + 128) == -3
    assert oe(wsb=need - 1) == -6
    assert oe(row=X + 64) == -8         # output inside X
    assert oe(ws=W) == -8               # workspace over W
    assert oe(row=ws + 256) == -8       # output inside the workspace
    # empty problems add nothing (no pointer needed)
    assert L.hscale_output_error(0, 0, n, 0, m, 1e-3, 0, 0, 0, 0, 0, 0) == 0
    assert L.hscale_output_error(0, T, n, 0, 0, 1e-3, 0, 0, 0, 0, 0, 0) == 0


def test_torch_front_end_rejects_bad_tensors_diagnostics():
    import torch
    from paper_2608_28113_amd import ops
    W = torch.zeros(4, 16, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ops.search_stats(W, torch.zeros(16), 1e-3, 4, 4)  # not on the GPU
    with pytest.raises(ValueError):
        ops.shift_summary(torch.zeros(4, dtype=torch.int8), torch.zeros(4), torch.zeros(4), 4, 4)
    with pytest.raises(ValueError):
        ops.output_error(torch.zeros(8, 16, dtype=torch.bfloat16), W, 1e-3, torch.zeros(4, 1, dtype=torch.uint8),
                         torch.zeros(4, 8, dtype=torch.uint8))


def test_search_layers_validation(L):
    """The batched search checks every layer as hscale_search_du does, and
    refuses outputs that overlap another layer's buffers, before any launch."""
    m, n = 4, 64
    B = 1 << 24  # layer k's buffers start at (k + 1) * B

    def layer(k, **kw):
        base = (k + 1) * B
        d = dict(W=base, out=m, in_=n, h=base + A, s=1e-3, init=0, codes=base + 2 * A, packed=base + 3 * A)
        d.update(kw)
        return (d["W"], d["out"], d["in_"], d["h"], d["s"], d["init"], d["codes"], d["packed"])

    def call(layers, down=4, up=4, mode=0):
        return L.hscale_search_layers(layers, down, up, mode, 0)

    good = [layer(0), layer(1), layer(2)]
    assert call([]) == 0                                   # nothing to do
    assert call([layer(0, out=0), layer(1, in_=0)]) == 0   # every layer empty: no launch
    assert L.load().hscale_search_layers(None, -1, 4, 4, 0, None) == -2
    assert L.load().hscale_search_layers(None, 2, 4, 4, 0, None) == -1
    assert call(good, down=-1) == -4
    assert call(good, up=126) == -4
    assert call(good, mode=3) == -2
    assert call(good[:1] + [layer(1, in_=65)]) == -2
    assert call(good[:2] + [layer(2, s=0.0)]) == -5
    assert call([layer(0, W=0)] + good[1:]) == -1
    assert call(good, mode=2) == -1                        # given codes but no init pointer
    assert call([layer(0, W=B + 8)]) == -3
    assert call([layer(0, packed=B + 3 * A + 4)]) == -3
    # within a layer: codes over its own W
    assert call([layer(0, codes=B + 16)]) == -8
    # across layers: layer 1's codes over layer 0's W, h or packed codes
    assert call([layer(0), layer(1, codes=B)]) == -8
    assert call([layer(0), layer(1, packed=B + A)]) == -8
    assert call([layer(0), layer(1, codes=B + 3 * A + 8)]) == -8
    # layer 0's codes as layer 1's initial codes (read while layer 0 writes them)
    assert call([layer(0, init=B + 5 * A), layer(1, init=B + 2 * A)], mode=2) == -8
