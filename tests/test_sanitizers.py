"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The C oracle (every entry point, on edge cases: empty and malformed
scoreboards, queues under caps, the size guard, special IPS values, depth 0
to 12 forests with NaN / inf thresholds) and the library's host-side forest
preparation (leaf boxes, tree records, cuts; checked against plain tree walks
on odd depths and NaN / inf thresholds) are built with gcc / g++ and
-fsanitize=address,undefined; a sanitizer report or a failed check fails the
test, and the checksum of everything computed must equal that of a plain -O2
build of the same program.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2408_05235_amd", "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]

PROGRAMS = {
    "oracle": (["gcc", "-std=c11", "-ffp-contract=off"],
               [os.path.join(HERE, "oracle_check.c"), os.path.join(ROOT, "oracle", "tl_oracle.c")], ["-lm"]),
    "host_forest": (["g++", "-std=c++17", "-I", CSRC],
                    [os.path.join(HERE, "host_forest_check.cpp"), os.path.join(CSRC, "host_forest.cpp")], []),
}


def _build_and_run(tmp_path, name, flags):
    cc, srcs, libs = PROGRAMS[name]
    exe = str(tmp_path / f"{name}_{'san' if flags is SAN else 'plain'}")
    subprocess.run(cc + flags + srcs + ["-o", exe] + libs, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    return r


@pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None, reason="no host compiler")
@pytest.mark.parametrize("name", sorted(PROGRAMS))
def test_host_code_under_sanitizers(tmp_path, name):
    san = _build_and_run(tmp_path, name, SAN)
    report = san.stderr
    assert san.returncode == 0, f"{name} under sanitizers: rc {san.returncode}\n{report[-3000:]}"
    assert "runtime error" not in report and "AddressSanitizer" not in report, report[-3000:]
    plain = _build_and_run(tmp_path, name, ["-O2"])
    assert plain.returncode == 0, plain.stderr[-2000:]
    ck = lambda out: re.search(r"checksum=([0-9a-f]+)", out).group(1)
    assert ck(san.stdout) == ck(plain.stdout), (san.stdout, plain.stdout)
