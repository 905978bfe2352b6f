"""pask_decode_attn_noalloc (the attention entry point that takes no
workspace and allocates nothing) against pask_decode_attn, through the C ABI:
two calls in a row, the second with a smaller input, each compared with the
workspace entry point's output and with the CPU oracle."""

import numpy as np
import pytest
import torch

from tests.gpu_util import Scenario, assert_attn_close, bf16_f64, bits16, say
from workload import make_policy, function_call_tags

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def _outs(sc, batch):
    out = torch.empty((batch, sc.Hq, sc.D), dtype=torch.bfloat16, device=sc.dev)
    lse = torch.empty((batch, sc.Hq), dtype=torch.float32, device=sc.dev)
    return out, lse


def _close_to(other: torch.Tensor, mine: torch.Tensor, what: str):
    """|mine - other| <= 2e-3 + 1e-2 |other|, element by element."""
    assert_attn_close(bf16_f64(mine), bf16_f64(other), what)


def test_noalloc_matches_workspace_entry_point_two_calls():
    from paper_2608_28276_amd import pask
    # Call 1: 64 sequences x 8 KV heads, one 8,000-token prompt among ~200-token
    # ones.  The workspace entry point sizes its partials for the whole hint
    # (65 pieces per (sequence, KV head), 69 MB); the scratch holds 31, so the
    # long sequence is cut into fewer, longer pieces: same results to tolerance.
    say("case: no-alloc attention, batch 64 with one long sequence (scratch holds fewer pieces)")
    B, Hq, Hkv, D = 64, 32, 8, 128
    rng = np.random.default_rng(41)
    P = rng.integers(150, 260, size=B)
    P[17] = 8000
    pol = make_policy(6, 1, 1, 0.33, seed=41)
    tags = np.stack([function_call_tags(12, 400 + b) for b in range(B)])
    sc = Scenario(pol, B=B, L=1, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=P, gen_tags=tags, seed=41)
    per_split = Hq // Hkv * (D + 2) * 4
    assert sc.sess.ws_bytes > pask.PASK_NOALLOC_SCRATCH_BYTES > 4 * B * Hkv * per_split
    sc.fill_prompt()
    sc.append_steps(0, 12)
    q = sc.q(0, 12)
    qd = q.to(sc.dev)
    o_na, l_na = _outs(sc, B)
    o_ws, l_ws = _outs(sc, B)
    sc.sess.decode_noalloc(0, qd, o_na, l_na)
    sc.sess.decode(0, qd, o_ws, l_ws)
    torch.cuda.synchronize()
    _close_to(o_ws, o_na, "call 1: no-alloc vs workspace entry point")
    assert np.abs(l_na.cpu().double().numpy() - l_ws.cpu().double().numpy()).max() <= 1e-4
    on = bf16_f64(o_na)
    for b in (17, 0, 40, 63):
        o_ref, _ = sc.oc.attend(0, b, bits16(q[b]), sc.scale)
        assert_attn_close(on[b], o_ref, f"call 1: no-alloc vs oracle, seq {b}")
    say("call 1: no-alloc matches the workspace entry point and the oracle")

    # Call 2, smaller: 5 sequences x 2 KV heads (few segments: the sliced
    # merge path), the step's token persisted by the same call, on two caches
    # in the same state: one through the no-alloc entry point, the other
    # through pask_decode_attn.  The scratch still holds call 1's partials.
    # Both entry points then use the same pieces, so their outputs and the
    # caches they leave agree bit for bit.
    say("case: no-alloc attention, second call with a smaller input (fused append)")
    pol2 = make_policy(6, 2, 2, 0.33, seed=42)
    tags2 = np.stack([function_call_tags(8, 500 + b) for b in range(5)])
    twins = [Scenario(pol2, B=5, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[3, 40, 170, 0, 333], gen_tags=tags2, seed=42)
             for _ in range(2)]
    for x in twins:
        x.fill_prompt()
        x.append_steps(0, 7)
    sc2, sc2w = twins
    for layer in range(2):
        k, v = sc2.gen_kv(layer, 7, 8)
        q2 = sc2.q(layer, 7)
        q2d = q2.to(sc2.dev)
        o_na, l_na = _outs(sc2, 5)
        o_ws, l_ws = _outs(sc2, 5)
        tg = torch.as_tensor(np.ascontiguousarray(sc2.gen_tags[:, 7]), device=sc2.dev)
        kd, vd = k[:, 0].contiguous().to(sc2.dev), v[:, 0].contiguous().to(sc2.dev)
        sc2.sess.decode_noalloc(layer, q2d, o_na, l_na, tg, kd, vd)
        sc2w.sess.decode(layer, q2d, o_ws, l_ws, tg, kd, vd)
        for x in twins:
            for b in range(5):
                x.oc.append(layer, b, x.gen_tags[b, 7:8], bits16(k[b]), bits16(v[b]))
        torch.cuda.synchronize()
        assert torch.equal(o_na, o_ws), f"call 2 layer {layer}: outputs differ from the workspace entry point"
        assert torch.equal(l_na, l_ws), f"call 2 layer {layer}: lse differs from the workspace entry point"
        on = bf16_f64(o_na)
        for b in range(5):
            o_ref, _ = sc2.oc.attend(layer, b, bits16(q2[b]), sc2.scale)
            assert_attn_close(on[b], o_ref, f"call 2: no-alloc vs oracle, layer {layer} seq {b}")
    for x in twins:
        x.check_state()
    say("call 2: no-alloc equals the workspace entry point bit for bit and matches the oracle")
