"""Build libpask.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2608_28276_amd.build

Every build compiles from source.  Flags:
  --offload-arch=gfx950                         CDNA4 only
  -fhip-fp32-correctly-rounded-divide-sqrt      IEEE division in the quantiser
  -Xclang -target-feature -Xclang -packed-fp32-ops
                                                no packed fp32 VALU instructions
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpask.so")
KERNEL_SOURCES = ("pask_append.hip", "pask_attn.hip")   # persisting entries; reading them
# The benchmark's on-device bandwidth probes: a library of their own, outside the C ABI.
PROBE_LIB = os.path.join(PKG, "libpask_probe.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall", "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-fhip-fp32-correctly-rounded-divide-sqrt",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"build step failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    """Compile and link libpask.so; returns its path."""
    with tempfile.TemporaryDirectory(prefix="pask_build_") as tmp:
        objs = []
        for src in KERNEL_SOURCES:
            objs.append(os.path.join(tmp, src.replace(".hip", ".o")))
            _run([HIPCC, *COMMON, *DEVICE, "-c", os.path.join(CSRC, src), "-o", objs[-1]])
        objs.append(os.path.join(tmp, "pask_api.o"))
        _run([HIPCC, *COMMON, "-c", os.path.join(CSRC, "pask_api.cpp"), "-o", objs[-1]])
        tmp_lib = os.path.join(tmp, "libpask.so")
        _run([HIPCC, *DEVICE, "-shared", "-fPIC", *objs, "-o", tmp_lib])
        shutil.move(tmp_lib, LIB)
        tmp_probe = os.path.join(tmp, "libpask_probe.so")
        _run([HIPCC, *COMMON, *DEVICE, "-shared", os.path.join(CSRC, "probe.hip"), "-o", tmp_probe])
        shutil.move(tmp_probe, PROBE_LIB)
    if verbose:
        print(f"built {LIB} and {PROBE_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
