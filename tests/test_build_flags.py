"""The library's device code is built without packed fp32 arithmetic: the
build passes the flag that turns the target feature off, and the gfx950
assembly of every source holds no v_pk_add_f32, v_pk_mul_f32 or
v_pk_fma_f32 (some forms of them have given wrong results on MI355X
without any error).  Runs on the CPU: hipcc cross-compiles."""
import os
import re
import shutil
import subprocess

import pytest

import paper_1601_04033_amd._build as lib_build

PACKED = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def test_build_turns_packed_fp32_off():
    f = lib_build.FLAGS
    i = f.index("-packed-fp32-ops")
    assert f[i - 3:i] == ["-Xclang", "-target-feature", "-Xclang"]
    assert "--offload-arch=gfx950" in f


@pytest.mark.skipif(shutil.which(lib_build.HIPCC) is None and not os.path.exists(lib_build.HIPCC),
                    reason="hipcc is not installed")
@pytest.mark.parametrize("src", lib_build.SOURCES)
def test_device_assembly_has_no_packed_fp32(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [lib_build.HIPCC, *lib_build.FLAGS, "-Wno-unused-command-line-argument", "--cuda-device-only", "-S",
           os.path.join(lib_build.CSRC, src),
           "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    asm = out.read_text()
    assert ".amdgcn_target" in asm and "gfx950" in asm
    hits = sorted({m.group(0) for m in PACKED.finditer(asm)})
    assert not hits, f"{src}: {hits}"
