"""bench.py on the CPU: its command-line contract (more than one GPU is
refused with a message before anything touches a GPU, inconsistent window
flags are rejected), and the committed profiles it quotes, which must be
current for the kernel sources."""
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent


def _run(*args):
    return subprocess.run([sys.executable, str(ROOT / "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=str(ROOT))


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_window_flags_are_checked():
    r = _run("--down", "9")
    assert r.returncode == 2 and "--down and --up" in r.stderr
    r = _run("--window", "4", "--down", "9", "--up", "6")
    assert r.returncode == 2


@pytest.mark.parametrize("workload", ["down_proj", "attn_proj", "down_proj_70b", "block"])
def test_committed_profile_traffic_matches_the_algorithmic_bytes(workload):
    """The rocprofv3 summary under profiles/ that the bench line quotes as
    `traffic` is per step and equals the algorithmic bytes of hdiag (X read
    once) and of the search (W read, codes written) within 1%."""
    import bench
    from synth.workloads import CONFIGS, block_workloads

    t = bench.measured_traffic(workload)
    # A missing or stale summary fails: the bench line would silently lose
    # its measured traffic.  Re-collect the profile after a kernel change.
    assert t is not None, f"profiles/{workload}.json is absent or older than the kernel sources"
    if workload == "block":
        wls = block_workloads()
        # X_attn and X_mlp (262144 x 4096) and X_down (262144 x 14336)
        hd = 2 * (2 * 262144 * 4096 + 4 * 4096) + (2 * 262144 * 14336 + 4 * 14336)
        weights = sum(wl.out * wl.inp for wl in wls.values())
    else:
        wl = CONFIGS[workload]
        hd = 2 * wl.tokens * wl.inp + 4 * wl.inp
        weights = wl.out * wl.inp
    assert abs(t["hdiag"] / hd - 1) < 0.01, (t["hdiag"], hd)
    assert abs(t["search"] / (bench.SEARCH_BYTES_PER_WEIGHT * weights) - 1) < 0.01


def test_committed_diagnostics_profile_is_current():
    """The output-error summary the diagnostics leg quotes as `traffic` was
    collected on the current output-error kernel sources."""
    import bench
    t = bench.diag_traffic("down_proj")
    assert t is not None, "profiles/output_error_down_proj.json is absent or older than the kernel sources"


def test_committed_ceilings_profile_is_current():
    """profiles/ceilings_down_proj.md (the probe kernels' trace beside the
    bench's timings) names the source hash of csrc/probes.hip it was taken
    on; it must be the current one."""
    import hashlib
    import re
    text = (ROOT / "profiles" / "ceilings_down_proj.md").read_text()
    m = re.search(r"csrc/probes\.hip at collection: `([0-9a-f]{16})`", text)
    assert m, "the summary names no source hash"
    src = (ROOT / "paper_2608_28113_amd" / "csrc" / "probes.hip").read_bytes()
    assert m.group(1) == hashlib.sha256(src).hexdigest()[:16], "re-collect the ceilings profile"
