"""The decode step captured in a HIP graph: two layers' fused append +
attention calls (pask_decode_attn with a token to persist) recorded once and
replayed step after step, the step's inputs copied into the graph's buffers
before each replay, with eager work and synchronisations between replays.
Every replay's outputs and log-sum-exps must equal, bit for bit, those of the
same calls made eagerly on a second cache fed the same inputs (which are
themselves compared with the CPU oracle), and the caches' final states must
agree."""

import numpy as np
import pytest
import torch

from tests.gpu_util import Scenario, say
from workload import function_call_tags, make_policy

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


@pytest.mark.parametrize("B,Hq,Hkv,D,noalloc", [(1, 32, 8, 128, False), (12, 32, 8, 128, False), (3, 8, 2, 64, False),
                                                 (12, 32, 8, 128, True), (1, 32, 8, 128, True)])
def test_graph_replays_match_eager_steps(B, Hq, Hkv, D, noalloc):
    """noalloc: the captured calls are pask_decode_attn_noalloc (no workspace
    argument: the callers it is for include code under graph capture), the
    eager twin's calls too."""
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob
    say(f"case: HIP graph of the decode step, B={B} Hq={Hq} Hkv={Hkv} D={D} noalloc={noalloc}")
    L, T, R = 2, 30, 5
    rng = np.random.default_rng(B + D)
    P = rng.integers(40, 900, size=B)
    pol = make_policy(6, 2, L, 0.33, seed=600 + B)
    tags = np.stack([function_call_tags(T, 610 + b) for b in range(B)])
    eager = Scenario(pol, B=B, L=L, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=P, gen_tags=tags, seed=61)
    eager.fill_prompt()
    eager.append_steps(0, T - R)
    g = eager.sess.geom
    sess = PaskSession(pack_blob(pol), max_batch=B, n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D,
                       max_tokens_per_seq=g.max_tokens_per_seq, hi_pages=g.hi_pages, lo_pages=g.lo_pages)
    dev = sess.device
    for layer in range(L):                                   # the same history, eagerly
        k, v = eager.prompt_kv(layer)
        sess.append(layer, None, k.to(dev), v.to(dev), n_new=torch.as_tensor(P, dtype=torch.int32, device=dev),
                    keep_all=True)
        k, v = eager.gen_kv(layer, 0, T - R)
        sess.append(layer, torch.as_tensor(np.ascontiguousarray(tags[:, :T - R]), device=dev), k.to(dev), v.to(dev))
    # the graph's input and output buffers
    tags_cur = torch.empty(B, dtype=torch.uint8, device=dev)
    q_cur = torch.empty((L, B, Hq, D), dtype=torch.bfloat16, device=dev)
    k_cur = torch.empty((L, B, Hkv, D), dtype=torch.bfloat16, device=dev)
    v_cur = torch.empty((L, B, Hkv, D), dtype=torch.bfloat16, device=dev)
    out = torch.empty((L, B, Hq, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((L, B, Hq), dtype=torch.float32, device=dev)

    def load(t):
        tags_cur.copy_(torch.as_tensor(np.ascontiguousarray(tags[:, t]), device=dev))
        for layer in range(L):
            k, v = eager.gen_kv(layer, t, t + 1)
            q_cur[layer].copy_(eager.q(layer, t).to(dev))
            k_cur[layer].copy_(k[:, 0].to(dev))
            v_cur[layer].copy_(v[:, 0].to(dev))

    def calls():
        for layer in range(L):
            fn = sess.decode_noalloc if noalloc else sess.decode
            fn(layer, q_cur[layer], out[layer], lse[layer], tags_cur, k_cur[layer], v_cur[layer])

    load(T - R)
    if noalloc:                                              # the scratch's address is taken before capture
        o = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=dev)
        eager.sess.decode_noalloc(0, eager.q(0, T - R).to(dev), o)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):                            # recorded, not run
        calls()
    torch.cuda.synchronize()
    for r in range(R):
        t = T - R + r
        load(t)
        graph.replay()
        torch.cuda.synchronize()
        got_o, got_l = out.clone(), lse.clone()
        for layer in range(L):                               # the same calls, eagerly (oracle-checked)
            eager.decode_step(t, layers=[layer], check=True, noalloc=noalloc)
        want_o = [eager.last[layer][0] for layer in range(L)]
        want_l = [eager.last[layer][1] for layer in range(L)]
        torch.cuda.synchronize()
        for layer in range(L):
            assert torch.equal(got_o[layer], want_o[layer]), f"replay {r} layer {layer}: outputs differ"
            assert torch.equal(got_l[layer], want_l[layer]), f"replay {r} layer {layer}: lse differs"
    eager.check_state()
    assert torch.equal(sess.counters(), eager.sess.counters()), "counters differ after the replays"
    for b in range(B):
        for layer in range(L):
            for st in (0, 1):
                a, e = sess.gather_store(b, layer, st), eager.sess.gather_store(b, layer, st)
                assert all(np.array_equal(x, y) for x, y in zip(a, e)), ("stores", b, layer, st)
    say(f"{R} replays equal the eager steps bit for bit")
