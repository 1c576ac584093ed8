"""The C-ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer:
the Eq. 2 schedule and every argument-validation path, built host-only (no
device code, no GPU) and linked with device-side stand-ins that abort if a
launch is ever reached. Golden keep counts come from the cited fixture."""
import json
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"
SOURCES = [
    os.path.join(ROOT, "paper_2509_01190_amd", "csrc", "zsa_api.cpp"),
    os.path.join(ROOT, "tests", "host", "launch_stubs.cpp"),
    os.path.join(ROOT, "tests", "host", "validate_driver.cpp"),
]
# the sanitizers go to the host compilation only (each flag behind -Xarch_host)
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


def golden_lines():
    with open(os.path.join(ROOT, "tests", "golden", "keep_schedule.json")) as f:
        cases = json.load(f)["cases"]
    lines = []
    for c in cases:
        n = c["n"]
        for cnt in c["counts"]:
            lines.append(f"{n} {c['alpha']!r} {c.get('tau', 5)} {cnt}")
            n = cnt
    return "\n".join(lines) + "\n"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                    reason="ROCm compilers not installed")
def test_validation_and_schedule_under_sanitizers():
    tmp = tempfile.mkdtemp(prefix="zsa_san_")
    try:
        objs = []
        for src in SOURCES:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            subprocess.run([HIPCC, "-x", "hip", "--cuda-host-only", "--offload-arch=gfx950", "-O1",
                            "-g", "-fno-omit-frame-pointer", *SAN, "-c", src, "-o", obj],
                           check=True, capture_output=True, text=True, timeout=300)
            objs.append(obj)
        exe = os.path.join(tmp, "validate_driver")
        subprocess.run([CLANG, "-fsanitize=address,undefined", *objs, "-o", exe],
                       check=True, capture_output=True, text=True, timeout=300)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], input=golden_lines(), capture_output=True, text=True,
                           timeout=300, env=env)
        assert r.returncode == 0, r.stdout + r.stderr
        assert r.stdout.startswith("ok "), r.stdout
        assert int(r.stdout.split()[1]) > 10000
        assert "runtime error" not in r.stderr, r.stderr
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
