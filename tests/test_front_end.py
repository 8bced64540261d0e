"""The torch front end checks every buffer it hands to the C ABI (dtype,
shape, contiguity, device) before any call into the library (CPU only).

The C ABI sees raw pointers, so a host tensor or a short output that got
through would be read or written by a kernel out of bounds.  Here 'meta'
tensors stand in for device tensors and every compute entry point of the
library is replaced by a stub that fails the test if it is reached: each
bad buffer must raise ValueError first, and each good call must reach its
stub."""
import pytest
import torch

from paper_2608_28113_amd import _lib, ops

DEV = "meta"
m, n, T = 4, 64, 8


class Reached(Exception):
    pass


@pytest.fixture
def fake_gpu(monkeypatch):
    monkeypatch.setattr(ops, "_on_device", lambda t: isinstance(t, torch.Tensor) and t.device.type == DEV)
    # no device to make current: call the (stubbed) library directly
    monkeypatch.setattr(ops, "_call", lambda device, fn, *args: fn(*args))

    def reached(*args):
        raise Reached

    for name in _lib.EXPORTS:
        if name.endswith("_workspace_bytes"):
            monkeypatch.setattr(_lib, name, lambda *args: 64)
        elif hasattr(_lib, name):
            monkeypatch.setattr(_lib, name, reached)


def _t(dtype, *shape):
    return torch.empty(shape, dtype=dtype, device=DEV)


def bf(*s):
    return _t(torch.bfloat16, *s)


def u8(*s):
    return _t(torch.uint8, *s)


def f32(*s):
    return _t(torch.float32, *s)


def f64(*s):
    return _t(torch.float64, *s)


def i8(*s):
    return _t(torch.int8, *s)


# Mutations of a good buffer; each must be refused.
def on_host(t):
    return torch.empty(t.shape, dtype=t.dtype)


def wrong_dtype(t):
    return _t(torch.float16 if t.dtype != torch.float16 else torch.float32, *t.shape)


def one_more_row(t):
    return _t(t.dtype, t.shape[0] + 1, *t.shape[1:])


def strided(t):
    return _t(t.dtype, *t.shape[:-1], 2 * t.shape[-1])[..., ::2]


def flat(t):
    return _t(t.dtype, t.numel())


ALL = (on_host, wrong_dtype, one_more_row, strided)
MATRIX_IN = (on_host, wrong_dtype, strided, flat)   # any row count is a valid input matrix
SCRATCH = (on_host, strided)                        # any dtype, the library checks the size

# function, good arguments, the mutations each buffer argument must refuse
CASES = {
    "hdiag": (ops.hdiag, lambda: dict(X=bf(T, n), h=f32(n), workspace=u8(64)),
              dict(X=MATRIX_IN, h=ALL, workspace=SCRATCH)),
    "hdiag_accumulate": (ops.hdiag_accumulate, lambda: dict(X=bf(T, n), h64=f64(n), workspace=u8(64)),
                         dict(X=MATRIX_IN, h64=ALL, workspace=SCRATCH)),
    "hdiag_finalize": (ops.hdiag_finalize, lambda: dict(h64=f64(n), h=f32(n)),
                       dict(h64=(on_host, wrong_dtype, strided), h=ALL)),
    "search": (ops.search, lambda: dict(W=bf(m, n), h=f32(n), global_scale=1e-3, window=4, init=u8(m, n // 16),
                                        scale_codes=u8(m, n // 16), packed_e2m1=u8(m, n // 2)),
               dict(W=MATRIX_IN + (one_more_row,), h=ALL, init=ALL, scale_codes=ALL, packed_e2m1=ALL)),
    "search_block": (ops.search_block,
                     lambda: dict(W=bf(m, 2 * n)[:, :n], h=f32(n), global_scale=1e-3, down=4, up=4,
                                  scale_codes=u8(m, n // 8)[:, :n // 16], packed_e2m1=u8(m, n)[:, :n // 2],
                                  init=u8(m, n // 16)),
                     dict(W=(on_host, wrong_dtype, strided, flat, one_more_row), h=ALL, scale_codes=ALL,
                          packed_e2m1=ALL, init=ALL)),
    "quantize": (ops.quantize, lambda: dict(W=bf(m, n), global_scale=1e-3, scale_codes=u8(m, n // 16),
                                            packed_e2m1=u8(m, n // 2)),
                 dict(W=MATRIX_IN + (one_more_row,), scale_codes=ALL, packed_e2m1=ALL)),
    "search_stats": (ops.search_stats, lambda: dict(W=bf(m, n), h=f32(n), global_scale=1e-3, down=4, up=4,
                                                    init=u8(m, n // 16)),
                     dict(W=MATRIX_IN, h=ALL, init=ALL)),
    "shift_summary": (ops.shift_summary, lambda: dict(shift=i8(m, n // 16), err_best=f32(m, n // 16),
                                                      err_init=f32(m, n // 16), down=4, up=4),
                      dict(shift=(on_host, wrong_dtype, strided), err_best=ALL, err_init=ALL)),
    "output_error": (ops.output_error,
                     lambda: dict(X=bf(T, n), W=bf(m, n), global_scale=1e-3, scale_codes=u8(m, n // 16),
                                  packed_e2m1=u8(m, n // 2), row_err=f64(m), workspace=u8(64)),
                     dict(X=MATRIX_IN, W=MATRIX_IN + (one_more_row,), scale_codes=ALL, packed_e2m1=ALL,
                          row_err=ALL, workspace=SCRATCH)),
}

BAD = [(fn, arg, mut.__name__) for fn, (_, _, args) in CASES.items() for arg, muts in args.items() for mut in muts]


@pytest.mark.parametrize("fn", sorted(CASES))
def test_good_buffers_reach_the_library(fake_gpu, fn):
    f, good, _ = CASES[fn]
    with pytest.raises(Reached):
        f(**good(), stream=0)


@pytest.mark.parametrize("fn,arg,mutation", BAD)
def test_bad_buffer_refused_before_the_library(fake_gpu, fn, arg, mutation):
    f, good, _ = CASES[fn]
    kwargs = good()
    kwargs[arg] = globals()[mutation](kwargs[arg])
    with pytest.raises(ValueError):
        f(**kwargs, stream=0)


@pytest.mark.parametrize("init", ["maxabs", "rtn", "4over6"])
def test_named_initial_codes_reach_the_library(fake_gpu, init):
    with pytest.raises(Reached):
        ops.search(bf(m, n), f32(n), 1e-3, down=9, up=6, init=init, stream=0)
    with pytest.raises(Reached):
        ops.search_stats(bf(m, n), f32(n), 1e-3, 9, 6, init=init, stream=0)


def test_unknown_initial_codes_and_windows_refused(fake_gpu):
    with pytest.raises(ValueError):
        ops.search(bf(m, n), f32(n), 1e-3, window=4, init="gptq", stream=0)
    with pytest.raises(ValueError):
        ops.search(bf(m, n), f32(n), 1e-3, window=4, down=1, up=1, stream=0)
    with pytest.raises(ValueError):
        ops.search(bf(m, n), f32(n), 1e-3, down=4, stream=0)


def test_output_error_needs_matching_operands(fake_gpu):
    with pytest.raises(ValueError):   # in_features differ
        ops.output_error(bf(T, 2 * n), bf(m, n), 1e-3, u8(m, n // 16), u8(m, n // 2), stream=0)
    with pytest.raises(ValueError):   # X and W on different devices
        ops.output_error(bf(T, n), on_host(bf(m, n)), 1e-3, u8(m, n // 16), u8(m, n // 2), stream=0)


def test_host_tensors_refused_without_stubs():
    """With the real library and no fakes, host tensors never reach it."""
    W = torch.zeros(m, n, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        ops.search(W, torch.zeros(n), 1e-3, window=4, stream=0)
    with pytest.raises(ValueError):
        ops.hdiag(W, stream=0)
    with pytest.raises(ValueError):
        ops.search_block(W, torch.zeros(n), 1e-3, 4, 4, torch.zeros(m, n // 16, dtype=torch.uint8),
                         torch.zeros(m, n // 2, dtype=torch.uint8), stream=0)


def _layers():
    return [(bf(m, n), f32(n), 1e-3), (bf(2 * m, n), f32(n), 2e-3), (bf(m, 2 * n), f32(2 * n), 1e-3)]


def test_search_layers_good_call_reaches_the_library(fake_gpu):
    with pytest.raises(Reached):
        ops.search_layers(_layers(), window=4, stream=0)
    with pytest.raises(Reached):
        ops.search_layers(_layers(), down=9, up=6, init="4over6", stream=0)
    L = _layers()
    with pytest.raises(Reached):
        ops.search_layers(L, window=4, init=[u8(W.shape[0], W.shape[1] // 16) for W, _, _ in L],
                          outputs=[(u8(W.shape[0], W.shape[1] // 16), u8(W.shape[0], W.shape[1] // 2))
                                   for W, _, _ in L], stream=0)
    assert ops.search_layers([], window=4, stream=0) == []


@pytest.mark.parametrize("k", [0, 2])
@pytest.mark.parametrize("part", ["W", "h", "codes", "packed", "init"])
@pytest.mark.parametrize("mutation", ["on_host", "wrong_dtype", "strided"])
def test_search_layers_bad_buffer_refused(fake_gpu, k, part, mutation):
    L = _layers()
    mut = globals()[mutation]
    outs = [(u8(W.shape[0], W.shape[1] // 16), u8(W.shape[0], W.shape[1] // 2)) for W, _, _ in L]
    init = [u8(W.shape[0], W.shape[1] // 16) for W, _, _ in L]
    W, h, s = L[k]
    if part == "W":
        L[k] = (mut(W), h, s)
    elif part == "h":
        L[k] = (W, mut(h), s)
    elif part == "codes":
        outs[k] = (mut(outs[k][0]), outs[k][1])
    elif part == "packed":
        outs[k] = (outs[k][0], mut(outs[k][1]))
    else:
        init[k] = mut(init[k])
    with pytest.raises(ValueError):
        ops.search_layers(L, window=4, init=init, outputs=outs, stream=0)


def test_search_layers_shape_mismatches_refused(fake_gpu):
    L = _layers()
    with pytest.raises(ValueError):
        ops.search_layers(L, window=4, outputs=[(u8(m, n // 16), u8(m, n // 2))], stream=0)  # too few
    with pytest.raises(ValueError):
        ops.search_layers(L, window=4, init=[u8(m, n // 16)], stream=0)
    with pytest.raises(ValueError):
        ops.search_layers([(bf(m, n), f32(n))], window=4, stream=0)                       # no s_g
    with pytest.raises(ValueError):
        ops.search_layers([(bf(m, n), f32(n + 16), 1e-3)], window=4, stream=0)            # h length
    with pytest.raises(ValueError):
        ops.search_layers(L, window=4, down=1, up=1, stream=0)
