"""The LDS staging copies set M0 in inline assembly (CPU only, gfx950 code
from hipcc).

The compiler accepts M0 in an inline-assembly clobber list but warns that a
reserved register may not be preserved around the statement.  These checks
compile the two kernel files that stage tree records into LDS to gfx950
assembly and show that nothing else in them uses M0: every instruction
naming it is a `s_mov_b32 m0, s<n>` directly followed by the
`global_load_lds_dwordx4` that reads it, and none of the instructions that
read M0 implicitly (message sends, relative register moves, GWS and
interpolation) appear.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2408_05235_amd import build

IMPLICIT_M0 = re.compile(r"^\s*(s_sendmsg\w*|s_movrel\w*|v_movrel\w*|s_set_gpr_idx\w*|ds_gws\w*|v_interp\w*)\b")
INSTR = re.compile(r"^\s+[a-z_][a-z0-9_]*(\s|$)")


def _device_asm(tmp_path, src):
    flags = [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    out = str(tmp_path / (os.path.basename(src) + ".s"))
    cmd = [build.hipcc(), *flags, "--cuda-device-only", "-S", "-I", build.INCLUDE, "-I", build.CSRC,
           "-x", "hip", src, "-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return open(out).read().splitlines()


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="no hipcc")
@pytest.mark.parametrize("name", ["forest.hip", "column.hip"])
def test_m0_only_feeds_the_staging_copies(tmp_path, name):
    lines = _device_asm(tmp_path, os.path.join(build.CSRC, name))
    instrs = [ln.split(";")[0].rstrip() for ln in lines if INSTR.match(ln) and not ln.lstrip().startswith(".")]
    writes = 0
    for i, ins in enumerate(instrs):
        assert not IMPLICIT_M0.match(ins), f"{name}: {ins.strip()} reads M0"
        if re.search(r"\bm0\b", ins):
            assert re.fullmatch(r"\s*s_mov_b32 m0, s\d+", ins), f"{name}: unexpected use of M0: {ins.strip()}"
            assert instrs[i + 1].split()[0] == "global_load_lds_dwordx4", \
                f"{name}: M0 set but not read by the next instruction: {instrs[i + 1].strip()}"
            writes += 1
    assert writes > 0, f"{name}: no staging copy found"
