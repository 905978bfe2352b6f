"""Run by test_gpu_debug.py in a process of its own with PASK_DEBUG=1 (the
library reads the variable once): a decode loop checked against the CPU
oracle, one layer's decode captured in a HIP graph and replayed, and an
append that sets device status flags.  Prints "child ok" at the end."""

import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import oracle  # noqa: E402
from tests.gpu_util import Scenario  # noqa: E402
from workload import make_policy  # noqa: E402
from workload.policy import pack_blob, uniform_policy  # noqa: E402
from workload.tags import iid_tags  # noqa: E402


def main():
    from paper_2608_28276_amd.session import PaskSession

    pol = make_policy(6, 2, 2, 0.33, seed=1000)
    tags = iid_tags(10, 7)[None].repeat(2, axis=0)
    sc = Scenario(pol, B=2, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[64, 37], gen_tags=tags, seed=1000)
    sc.fill_prompt()
    for t in range(8):
        sc.decode_step(t)                       # each step checked against the oracle
    sc.check_state()
    print("decode loop matches the oracle", flush=True)

    dev = sc.sess.device
    q = sc.q(0, 8).to(dev)
    out = torch.empty((2, 8, 64), dtype=torch.bfloat16, device=dev)
    want = torch.empty_like(out)
    sc.sess.decode(0, q, want)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):               # a capturing stream is not waited on
        sc.sess.decode(0, q, out)
    for _ in range(2):
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want), "graph replay differs from the eager call"
    print("graph replays match", flush=True)

    flagged = PaskSession(pack_blob(uniform_policy(6, 1, 1, oracle.LOW)), max_batch=2, n_layers=1, n_q_heads=8,
                          n_kv_heads=2, head_dim=64, max_tokens_per_seq=64, hi_pages=1, lo_pages=2)
    k = torch.randn((2, 64, 2, 64), generator=torch.Generator().manual_seed(5)).to(torch.bfloat16).to(dev)
    t = torch.zeros((2, 64), dtype=torch.uint8, device=dev)
    t[0, 3] = 200                               # a tag outside the table, and more LOW tokens than pages
    flagged.append(0, t, k, k)
    st, _, _ = flagged.stats(batch=2)
    print(f"flags {st.device_flags:#x}", flush=True)
    assert np.isfinite(sc.sess.stats()[0].c_kv_all)
    print("child ok", flush=True)


if __name__ == "__main__":
    main()
