"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only): tests/sanitize/san_driver.cpp links
oracle/*.c and the host sources of libeq (encoders, container validation,
scale optimiser) built with -fsanitize=address,undefined and runs them on
small seeded matrices and on damaged containers (random bit flips in the
header, the section tables and the payload; truncated blobs).  Any report
from either sanitizer makes the program exit non-zero."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


def _build(out_dir):
    inc = ["-I", os.path.join(ROOT, "include"), "-I",
           os.path.join(ROOT, "paper_2601_22787_amd", "csrc"), "-I", os.path.join(ROOT, "oracle"),
           "-I", "/opt/rocm/include"]
    objs = []
    for src in ("oracle/eq_oracle.c", "oracle/eq_phrase.c"):
        obj = os.path.join(out_dir, os.path.basename(src) + ".o")
        subprocess.run(["gcc", "-std=c99", "-ffp-contract=off", *SAN, *inc, "-c",
                        os.path.join(ROOT, src), "-o", obj], check=True)
        objs.append(obj)
    for src in ("paper_2601_22787_amd/csrc/eq_encode.cpp", "paper_2601_22787_amd/csrc/eq_rd.cpp",
                "paper_2601_22787_amd/csrc/eq_layer.cpp", "tests/sanitize/san_driver.cpp"):
        obj = os.path.join(out_dir, os.path.basename(src) + ".o")
        subprocess.run(["g++", "-std=c++17", "-pthread", "-D__HIP_PLATFORM_AMD__", *SAN, *inc,
                        "-c", os.path.join(ROOT, src), "-o", obj], check=True)
        objs.append(obj)
    exe = os.path.join(out_dir, "san_driver")
    subprocess.run(["g++", "-pthread", *SAN, *objs, "-o", exe, "-lm"], check=True)
    return exe


@pytest.mark.timeout(600)
def test_host_code_under_asan_ubsan(tmp_path):
    exe = _build(str(tmp_path))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=540)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "sanitized host run ok" in r.stdout
