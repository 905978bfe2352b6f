"""The attention call's work split (pask_plan.h, shared with the device code),
compiled for the host and checked on random calls
(tests/native/plan_check.hip): every page attended once, every piece index
in bounds and written once, at most `splits` pieces per segment."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="no hipcc")
def test_work_split_invariants(tmp_path):
    exe = tmp_path / "plan_check"
    b = subprocess.run([HIPCC, "-O2", "-std=c++17", "--offload-arch=gfx950", f"-I{ROOT}/paper_2608_28276_amd/csrc",
                        f"{ROOT}/tests/native/plan_check.hip", "-o", str(exe)], capture_output=True, text=True,
                       timeout=300)
    assert b.returncode == 0, b.stderr[-4000:]
    r = subprocess.run([str(exe), "600"], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout[-3000:]
