"""The library's host code (CSR and dense packing, pack.cpp) and the C oracle
built with AddressSanitizer and UndefinedBehaviorSanitizer (gcc/g++, CPU only)
and run over randomized packing cases, the packers' error paths and small
oracle layers (tests/sanitize_driver.cpp). Any sanitizer report aborts the
driver; any packing mismatch against the oracle fails it."""
import os
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc/g++")
def test_packers_and_oracle_under_sanitizers(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
    inc = ["-I", str(ROOT / "include"), "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]
    objs = []
    for cmd, src in ((["gcc", "-std=c11", "-fopenmp"], ROOT / "oracle" / "spconv_oracle.c"),
                     (["g++", "-std=c++17"], ROOT / "paper_2005_04091_amd" / "csrc" / "pack.cpp"),
                     (["g++", "-std=c++17"], ROOT / "tests" / "sanitize_driver.cpp")):
        obj = tmp_path / (src.stem + ".o")
        subprocess.run(cmd + san + inc + ["-c", str(src), "-o", str(obj)], check=True)
        objs.append(str(obj))
    exe = tmp_path / "sanitize_driver"
    subprocess.run(["g++", "-fopenmp"] + san + objs + ["-o", str(exe), "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failures" in r.stdout
