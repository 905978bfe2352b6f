"""The host side of the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: pask_api.cpp is compiled with g++
together with a seeded mutation fuzzer (tests/native/policy_fuzz.cpp) that
feeds pask_policy_load mutated policy blobs (the untrusted input of the
library) and the geometry checks random geometries."""

import os
import shutil
import subprocess

import pytest

from workload import make_policy, pack_blob
from workload.policy import uniform_policy, with_budget_controller
from workload.tags import CRITICAL_STATES, PARSER_STATES, function_call_tags_with_states

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _seed_blobs(tmp_path):
    pol_a = make_policy(6, 2, 2, 0.33, seed=1)
    pol_b = make_policy(12, 4, 36, 0.33, seed=2, n_sink=16)
    pol_b.recent_window = 16
    pol_c = with_budget_controller(make_policy(6, 4, 36, 0.33, seed=3),
                                   [function_call_tags_with_states(400, 5)], len(PARSER_STATES), CRITICAL_STATES)
    pol_d = uniform_policy(64, 16, 128, 1)
    paths = []
    for i, p in enumerate((pol_a, pol_b, pol_c, pol_d)):
        path = tmp_path / f"seed{i}.bin"
        path.write_bytes(pack_blob(p))
        paths.append(str(path))
    return paths


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_policy_load_and_geometry_checks_under_sanitizers(tmp_path):
    exe = tmp_path / "policy_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT}/include",
           f"-I{ROOT}/paper_2608_28276_amd/csrc", f"{ROOT}/tests/native/policy_fuzz.cpp",
           f"{ROOT}/paper_2608_28276_amd/csrc/pask_api.cpp", "-o", str(exe)]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert b.returncode == 0, b.stderr[-4000:]
    # verify_asan_link_order=0: the environment may preload a library of its own ahead of ASan's runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe), "12345", "200000", *_seed_blobs(tmp_path)], capture_output=True, text=True,
                       timeout=600, env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert r.stdout.startswith("ok:")
