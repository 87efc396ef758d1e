"""The host code of libacrl under AddressSanitizer: the library's sources are
compiled with the sanitizer on the host side only (-Xarch_host, device code
untouched) and linked into a C driver (tests/host_validation.c) that runs
every entry point's argument validation and the host helpers.  No device is
used: every call in the driver fails validation before any HIP call."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_24062_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
SOURCES = ["api.hip", "quantize.hip", "score.hip", "reduce.hip"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_validation_paths_under_asan(tmp_path):
    flags = ["--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-O1", "-fPIC", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    procs = []
    for src in SOURCES:
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, src),
                                       "-o", str(tmp_path / src.replace(".hip", ".o"))],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    for pr in procs:
        out = pr.communicate(timeout=600)[0]
        assert pr.returncode == 0, out.decode(errors="replace")[-2000:]
    drv = str(tmp_path / "driver.o")
    r = subprocess.run([HIPCC, "-Xarch_host", "-fsanitize=address", "-I", os.path.join(ROOT, "include"), "-x", "c",
                        "-c", os.path.join(ROOT, "tests", "host_validation.c"), "-o", drv],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    exe = str(tmp_path / "host_validation")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-o", exe, drv,
                        *[str(tmp_path / s.replace(".hip", ".o")) for s in SOURCES]],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "0 unexpected results" in r.stdout, (r.stdout[-3000:] + r.stderr[-3000:])
    assert "ERROR: AddressSanitizer" not in r.stderr and "LeakSanitizer" not in r.stderr, r.stderr[-3000:]
