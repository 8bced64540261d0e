"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds tests/native/sanitize_driver.cpp against the oracle's C source and the
library's HIP source, with the sanitizers on the host side only (GPU code is
compiled normally and never launched: every library call in the driver fails
validation or is empty), and runs it.
"""
import os
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not Path(HIPCC).exists(), reason="hipcc not installed")
def test_host_code_is_sanitizer_clean(tmp_path):
    oracle_o = tmp_path / "oracle.o"
    subprocess.run(["gcc", "-c", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    "-ffp-contract=off", "-o", str(oracle_o), str(ROOT / "oracle" / "hscale_oracle.c")], check=True)
    common = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-ffp-contract=off",
              "-fhip-fp32-correctly-rounded-divide-sqrt", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-I", str(ROOT / "include"),
              "-I", str(ROOT / "paper_2608_28113_amd" / "csrc")]
    csrc = ROOT / "paper_2608_28113_amd" / "csrc"
    units = [(csrc / f"{u}.hip", tmp_path / f"{u}.o") for u in ("hdiag", "search", "diag")]
    units.append((ROOT / "tests" / "native" / "sanitize_driver.cpp", tmp_path / "driver.o"))
    exe = tmp_path / "driver"
    for src, obj in units:
        r = subprocess.run(common + ["-x", "hip", "-c", "-o", str(obj), str(src)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address",
                        "-Xarch_host", "-fsanitize=undefined", "-o", str(exe), *[str(o) for _, o in units],
                        str(oracle_o), "-lm"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "sanitize driver: ok" in r.stdout, (r.stdout + r.stderr)[-3000:]
