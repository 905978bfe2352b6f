"""The append kernels' division-free int4 code rule (quant_code, shared with
the device code through pask_device.h), compiled for the host and checked
exhaustively on the CPU against RNE(x / s) in fp64 (tests/native/quant_code_check.hip)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="no hipcc")
def test_quant_code_rule_exhaustive(tmp_path):
    exe = tmp_path / "quant_code_check"
    b = subprocess.run([HIPCC, "-O2", "-std=c++17", "--offload-arch=gfx950", f"-I{ROOT}/include",
                        f"-I{ROOT}/paper_2608_28276_amd/csrc", f"{ROOT}/tests/native/quant_code_check.hip",
                        "-o", str(exe)], capture_output=True, text=True, timeout=300)
    assert b.returncode == 0, b.stderr[-4000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout[-3000:]
