"""Register and scratch use of the gfx950 kernels, from the compiler's own
metadata for the sources as built (device-only assembly, on the CPU).

The launch shapes assume occupancies that these figures decide: the search
and hdiag kernels run 7 waves per SIMD (at most 72 VGPRs: 512 / 7 rounded
down to the allocation granule of 8), and the output-error tile kernel 3
(at most 168).  No kernel may use scratch memory: a spill turns into
per-wave memory traffic the rooflines do not count.
"""
from __future__ import annotations

import re
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
CSRC = ROOT / "paper_2608_28113_amd" / "csrc"


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    from paper_2608_28113_amd import build
    out = {}
    tmp = tmp_path_factory.mktemp("asm")
    for src in ("hdiag.hip", "search.hip", "diag.hip"):
        asm = tmp / (src + ".s")
        flags = [f for f in build.FLAGS if f not in ("-shared", "-fPIC")]
        cmd = [build.HIPCC, *flags, "--cuda-device-only", "-S", "-I", str(ROOT / "include"), "-I", str(CSRC),
               "-o", str(asm), str(CSRC / src)]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        text = asm.read_text()
        for m in re.finditer(r"^\s+\.set (\S+)\.num_vgpr, (\d+)", text, re.M):
            name = m.group(1)
            scratch = int(re.search(re.escape(name) + r"\.private_seg_size, (\d+)", text).group(1))
            out[name] = (src, int(m.group(2)), scratch)
    return out


def _find(kernels, fragment):
    found = {k: v for k, v in kernels.items() if fragment in k}
    assert found, fragment
    return found


def test_no_kernel_uses_scratch(kernels):
    spilled = {k: v for k, v in kernels.items() if v[2] != 0}
    assert not spilled, spilled


@pytest.mark.parametrize("fragment,limit", [("search_kernel", 72), ("search_layers_kernel", 72),
                                            ("hdiag_partial", 72), ("lfull_tile_kernel", 168)])
def test_vgprs_fit_the_assumed_occupancy(kernels, fragment, limit):
    for name, (src, vgpr, _) in _find(kernels, fragment).items():
        assert vgpr <= limit, (name, src, vgpr)
