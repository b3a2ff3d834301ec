"""Host check of the KV cache block layout (kv_key_offset, kv_val_offset in kernels.h): each
map is a bijection onto the 64-position block, and the 16-byte fragment that the attention
loads for (tile, step, lane) holds exactly the keys and head dims that its MFMA operand
layout multiplies.  The layout functions are compiled for the host from the library's own
header."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2510_05421_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="hipcc not available")
def test_kv_block_layout_matches_the_attention_fragments(tmp_path):
    exe = tmp_path / "kv_layout_check"
    hipcc = HIPCC if os.path.exists(HIPCC) else shutil.which("hipcc")
    subprocess.run([hipcc, "-O1", "-std=c++17", "-I", CSRC, os.path.join(HERE, "kv_layout_check.cpp"), "-o",
                    str(exe)], check=True, capture_output=True, timeout=300)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout
