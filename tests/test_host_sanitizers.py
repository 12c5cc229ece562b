"""The library's host half (compressors, stream validation, metadata-slot builder, worker
pool) and the CPU oracle under AddressSanitizer, LeakSanitizer and
UndefinedBehaviorSanitizer: a CPU-only build of those sources with g++/gcc and the
driver tests/sanitize/host_driver.cpp (no GPU code is built or run)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_30728_amd", "csrc")
FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


@pytest.mark.slow
@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_sanitizers(tmp_path):
    inc = [f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    objs = []
    for src in ("ibp_host.cpp", "ibp_pool.cpp", "ibp_meta_slots.cpp"):
        o = str(tmp_path / (src + ".o"))
        subprocess.run(["g++", "-std=c++17", *FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", o], check=True)
        objs.append(o)
    o = str(tmp_path / "oracle.o")
    subprocess.run(["gcc", "-std=c99", *FLAGS, "-c", os.path.join(ROOT, "oracle", "ibp_oracle.c"), "-o", o],
                   check=True)
    objs.append(o)
    exe = str(tmp_path / "host_driver")
    subprocess.run(["g++", "-std=c++17", *FLAGS, *inc, os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"),
                    *objs, "-o", exe, "-lpthread"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    env.pop("IBP_TEST_FAIL_ALLOC", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-6000:]
    assert "host sanitize ok" in r.stdout
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-4000:]
