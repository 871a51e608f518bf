"""The built library's device code: every kernel keeps its indices in
hardware registers.  With the IEEE mode bit off, the runtime's blockIdx /
threadIdx accessors are not inlined and would become real calls
(``s_swappc_b64``) in every kernel; this checks the disassembly of the code
object built here for any call."""
import os
import subprocess

import pytest

from paper_2606_12688_amd import attn

LLVM = "/opt/rocm/llvm/bin"
TOOLS = ("llvm-objcopy", "clang-offload-bundler", "llvm-objdump")


@pytest.mark.skipif(not all(os.path.exists(os.path.join(LLVM, t)) for t in TOOLS), reason="ROCm LLVM tools missing")
def test_kernels_make_no_calls(tmp_path):
    if not os.path.exists(attn.LIB_PATH):
        pytest.skip("library not built")
    fat, co = tmp_path / "fatbin", tmp_path / "gfx950.co"
    subprocess.run([os.path.join(LLVM, "llvm-objcopy"), f"--dump-section=.hip_fatbin={fat}", attn.LIB_PATH,
                    str(tmp_path / "stripped.so")], check=True, capture_output=True)
    subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle", "--type=o", f"--input={fat}",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--output={co}"], check=True, capture_output=True)
    dis = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--no-show-raw-insn", str(co)], check=True,
                         capture_output=True, text=True).stdout
    kernels = [ln for ln in dis.splitlines() if ln.endswith(">:") and "_kernel" in ln]
    assert len(kernels) >= 10, "expected the tile, few-row, f32, merge and append kernels"
    assert "s_swappc" not in dis, "a kernel calls a function (index accessor not inlined?)"
