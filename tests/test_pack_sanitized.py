"""The host planning code (pp_plan_bounds, pp_pack, pp_pack_padded) under AddressSanitizer and
UndefinedBehaviorSanitizer.

``tests/host/pack_sanitize.cpp`` drives the library's own ``pack.cpp`` and ``status.cpp``,
built here with g++ and both sanitizers, over seeded random batches: every plan array is a
separate allocation of exactly the size ``pp_plan_bounds`` reports, so any write past the
documented sizes (section 3.1's rows and segments, section 3.2's slot maps, the work lists)
stops the run; each call is repeated with one capacity one element short, which must be
rejected without writing out of bounds.  CPU only, no GPU code involved.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2404_09529_amd", "csrc")


def test_pack_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("a library is preloaded here; the sanitizer runtime has to come first")
    exe = str(tmp_path / "pack_sanitize")
    build = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             os.path.join(ROOT, "tests", "host", "pack_sanitize.cpp"), os.path.join(CSRC, "pack.cpp"),
             os.path.join(CSRC, "status.cpp"), "-o", exe]
    subprocess.run(build, check=True, timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, "600"], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failed checks" in r.stdout, r.stdout
