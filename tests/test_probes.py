"""The benchmark's measurement probes (libhscale_probes.so, no part of the
hscale C ABI).  CPU: the library exports its three entry points and rejects
bad arguments on the host before any launch.  GPU: the streaming read covers
every byte of its chunks (its per-lane word sums equal the host's), and the
VALU probes run and record advancing clocks."""
import subprocess

import numpy as np
import pytest

PROBES = ("hsprobe_stream_read", "hsprobe_valu", "hsprobe_wall_clock_khz")


@pytest.fixture(scope="module")
def P():
    import bench
    from paper_2608_28113_amd import build
    if not build.PROBE_LIB.exists():
        build.build()
    return bench.load_probes()


def test_probe_library_exports(P):
    import bench
    out = subprocess.run(["nm", "-D", "--defined-only", bench.PROBE_LIB], capture_output=True, text=True,
                         check=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in PROBES:
        assert name in syms, name


def test_probe_arguments_are_checked_on_the_host(P):
    fake = 1 << 20  # aligned, never dereferenced: every case returns before a launch
    assert P.hsprobe_stream_read(None, 1 << 20, 4, fake, None) == -1
    assert P.hsprobe_stream_read(fake, 1 << 20, 4, None, None) == -1
    assert P.hsprobe_stream_read(fake + 4, 1 << 20, 4, fake, None) == -1  # not 16-byte aligned
    assert P.hsprobe_stream_read(fake, 0, 4, fake, None) == -1
    assert P.hsprobe_stream_read(fake, 1 << 20, 0, fake, None) == -1
    assert P.hsprobe_stream_read(fake, 65535 * 4, 4, fake, None) == -1  # under one 64 KiB round per block
    for kind in (-1, 5):
        assert P.hsprobe_valu(kind, 8, 16, fake, fake, None) == -1
    assert P.hsprobe_valu(0, 0, 16, fake, fake, None) == -1
    assert P.hsprobe_valu(0, 8, 0, fake, fake, None) == -1
    assert P.hsprobe_valu(0, 8, 16, None, fake, None) == -1


@pytest.mark.gpu
def test_stream_read_reads_every_byte(P):
    import torch
    blocks, rounds = 48, 3
    chunk = rounds * 256 * 16 * 16  # bytes per block: whole 64 KiB rounds
    nbytes = blocks * chunk + 4096 + 16  # a ragged tail the probe leaves unread
    g = torch.Generator().manual_seed(11)
    host = torch.randint(-(2 ** 31), 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int32, generator=g)
    buf = host.cuda()
    sums = torch.full((blocks * 256,), -1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    print(f"[probe] stream_read blocks={blocks} bytes={nbytes}", flush=True)
    n = P.hsprobe_stream_read(buf.data_ptr(), nbytes, blocks, sums.data_ptr(), stream.cuda_stream)
    torch.cuda.synchronize()
    assert n == blocks * chunk
    words = host.numpy().view(np.uint32)[: n // 4].reshape(blocks, -1, 256, 4).astype(np.uint64)
    ref = (words.sum(axis=(1, 3)) % (1 << 32)).astype(np.uint32)
    assert np.array_equal(sums.cpu().numpy().view(np.uint32).reshape(blocks, 256), ref)


@pytest.mark.gpu
@pytest.mark.parametrize("kind", [0, 1, 2, 3, 4])
def test_valu_probe_runs_and_records_clocks(P, kind):
    import torch
    blocks = 16
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(blocks * 4 * 4, dtype=torch.int64, device="cuda")
    print(f"[probe] valu kind={kind} blocks={blocks}", flush=True)
    assert P.hsprobe_valu(kind, blocks, 64, sink.data_ptr(), clocks.data_ptr(),
                          torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    c = clocks.view(-1, 4).cpu().numpy()
    assert (c[:, 1] > c[:, 0]).all() and (c[:, 3] >= c[:, 2]).all()
    assert P.hsprobe_wall_clock_khz() > 0
