"""The C header from plain C: ``tests/host/abi_c_example.c`` is compiled as C99 with
``-pedantic -Wall -Wextra -Werror`` against ``include/prepack.h``, linked to the built
``libprepack.so`` and run (host planning only, no GPU): FFD of six prompts into rows of 8
(section 3.1) with their restart positions (section 3.2), and an over-long prompt rejected
with its message."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2404_09529_amd")


def test_header_compiles_as_c99_and_plans_from_c(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    if not os.path.exists(os.path.join(PKG, "libprepack.so")):
        pytest.skip("libprepack.so is not built")
    exe = str(tmp_path / "abi_c_example")
    subprocess.run([gcc, "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "host", "abi_c_example.c"), "-L", PKG, "-lprepack",
                    f"-Wl,-rpath,{PKG}", "-o", exe], check=True, timeout=120)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "6 prompts, 25 tokens, 4 rows of 8" in r.stdout
    assert "row 1: prompt 4 (len 6) prompt 3 (len 2) | positions 0 1 2 3 4 5 0 1" in r.stdout
    assert "does not fit a row of 4" in r.stdout
