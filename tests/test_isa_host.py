"""Host check on the AMD assembly of the GEMM kernels as built here for
gfx950 (the code object inside the build's object file, disassembled): the
direct LDS loads set M0 through inline assembly that declares M0 clobbered,
which is sound only while nothing else in those kernels keeps a value in M0.
Every M0 write must be the one immediately before its direct load, and no
other instruction may name M0."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OBJ = os.path.join(ROOT, "paper_1809_02839_amd", "_build", "gemm_bf16.hip.o")
LLVM = "/opt/rocm/llvm/bin"


@pytest.mark.skipif(not os.path.exists(OBJ), reason="the library has not been built here")
@pytest.mark.skipif(not os.path.exists(os.path.join(LLVM, "llvm-objdump")), reason="ROCm LLVM tools not available")
def test_m0_only_feeds_the_direct_lds_loads(tmp_path):
    fat, co = tmp_path / "fatbin", tmp_path / "gfx950.co"
    subprocess.run([os.path.join(LLVM, "llvm-objcopy"), f"--dump-section=.hip_fatbin={fat}", OBJ,
                    str(tmp_path / "host.o")], check=True, capture_output=True)
    subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle", "--type=o",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--input={fat}", f"--output={co}"],
                   check=True, capture_output=True)
    dis = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950", str(co)], check=True,
                         capture_output=True, text=True).stdout
    lines = [l.split("//")[0].strip() for l in dis.splitlines()]
    lines = [l for l in lines if l and not l.endswith(":")]
    pairs, other = 0, []
    for i, l in enumerate(lines):
        if not re.search(r"\bm0\b", l):
            continue
        nxt = lines[i + 1] if i + 1 < len(lines) else ""
        if l.startswith("s_mov_b32 m0,") and nxt.startswith("buffer_load_dwordx4") and nxt.endswith(" lds"):
            pairs += 1
        else:
            other.append(l)
    assert pairs > 0, "no direct LDS loads found"
    assert not other, other[:10]
