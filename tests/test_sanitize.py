"""The host code of the library (the attention planner, the KV hand-off
planner, deficit admission) and the C oracle, built with AddressSanitizer
and UndefinedBehaviorSanitizer and driven over random and malformed inputs
(tests/sanitize/san_driver.cpp). CPU only: g++ / gcc, no HIP."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_04206_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if not shutil.which("g++") or not shutil.which("gcc"):
        pytest.skip("needs g++ and gcc")
    out = tmp_path_factory.mktemp("san")
    objs = []
    for src in ("plan.cpp", "sched.cpp", "kv_plan.cpp"):
        o = str(out / (src + ".o"))
        subprocess.run(["g++", "-std=c++17", *SAN, "-c", os.path.join(CSRC, src), "-o", o], check=True)
        objs.append(o)
    o = str(out / "oracle.o")
    subprocess.run(["gcc", "-std=c11", *SAN, "-c", os.path.join(ROOT, "oracle", "attn_oracle.c"), "-o", o],
                   check=True)
    objs.append(o)
    exe = str(out / "san_driver")
    subprocess.run(["g++", "-std=c++17", *SAN, os.path.join(ROOT, "tests", "sanitize", "san_driver.cpp"),
                    *objs, "-lm", "-o", exe], check=True)
    return exe


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_host_code_under_asan_ubsan(driver, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    r = subprocess.run([driver, str(seed)], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert " 0 failed checks" in r.stdout, r.stdout
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
