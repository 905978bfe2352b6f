"""Debug mode (PASK_DEBUG=1): every launching entry point waits for its
stream and reports failures and new device status flags on stderr.  Run in a
child process, since the library reads the variable once."""

import os
import re
import subprocess
import sys

import pytest
import torch

from tests.gpu_util import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def test_debug_mode_checks_and_reports_flags():
    from paper_2608_28276_amd import pask
    say("case: PASK_DEBUG=1 child process")
    env = dict(os.environ, PASK_DEBUG="1")
    p = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "debug_child.py")], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=110)
    assert p.returncode == 0, f"child failed ({p.returncode}):\n{p.stdout[-3000:]}\n{p.stderr[-3000:]}"
    assert "child ok" in p.stdout
    reports = re.findall(r"pask: (\w+): device status flags 0x([0-9a-f]+)", p.stderr)
    assert reports, p.stderr[-2000:]
    where, word = reports[-1]
    assert where == "pask_kv_append"
    word = int(word, 16)
    assert word & pask.PASK_FLAG_BAD_TAG and word & pask.PASK_FLAG_LO_POOL_EXHAUSTED
    assert f"flags {word:#x}" in p.stdout                 # the same word pask_cache_stats reads
    errors = [l for l in p.stderr.splitlines() if l.startswith("pask: ") and "device status flags" not in l]
    assert not errors, errors                             # no launch or execution error reported
    assert len(reports) == 1, reports                     # the decode loop and the graph raised no flag
