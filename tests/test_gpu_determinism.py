"""Determinism of the HIP path: the same inputs through two fresh caches give
bit-identical decisions, counters, index lists, stored bits / codes / scales
(gathered through the block tables: physical page ids depend on the order in
which blocks take pages and may differ) and bit-identical attention outputs
and log-sum-exps, on both attention paths (few and many segments) and with
the recent window and the online controller.  And no result depends on
memory the library has not written: caches and workspaces whose every byte
was set to 0x00, 0xFF (NaN in bf16, fp16 and fp32) or 0x7F before
pask_cache_init give the same bits (a second fresh cache in the same process
may reuse the first one's memory, so the plain repeat cannot show this)."""

import numpy as np
import pytest
import torch

from tests.gpu_util import Scenario, say
from workload import function_call_tags, make_policy
from workload.policy import with_budget_controller
from workload.tags import CRITICAL_STATES, PARSER_STATES, function_call_tags_with_states

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def _run(pol, B, Hq, Hkv, D, P, tags, seed, states=None, prefill=None, prompt_tags=None):
    """Fill, bulk-append, then fused steps; returns everything observable."""
    sc = Scenario(pol, B=B, L=2, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=P, gen_tags=tags, seed=seed, gen_states=states,
                  prefill=prefill, prompt_tags=prompt_tags)
    if states is not None:
        sc.budget_init(tags.shape[1])
    sc.fill_prompt()
    sc.append_steps(0, tags.shape[1] - 3)
    outs = []
    for t in range(tags.shape[1] - 3, tags.shape[1]):
        for layer in range(2):
            k, v = sc.gen_kv(layer, t, t + 1)
            q = sc.q(layer, t).to(sc.dev)
            out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=sc.dev)
            lse = torch.empty((B, Hq), dtype=torch.float32, device=sc.dev)
            tg = torch.as_tensor(np.ascontiguousarray(tags[:, t]), device=sc.dev)
            sd = None if states is None else torch.as_tensor(np.ascontiguousarray(states[:, t]), device=sc.dev)
            sc.sess.decode(layer, q, out, lse, tg, k[:, 0].contiguous().to(sc.dev), v[:, 0].contiguous().to(sc.dev),
                           states_new=sd)
            outs.append((out.view(torch.int16).cpu().numpy(), lse.view(torch.int32).cpu().numpy()))
    torch.cuda.synchronize()
    cnt = sc.sess.counters().cpu().numpy()
    full = sc.sess.index_lists().cpu().numpy()     # entries past a store's count are not written
    lists = [full[b, l, st, :cnt[b, l, st]] for b in range(B) for l in range(2) for st in (0, 1)]
    stores = [[sc.sess.gather_store(b, layer, st) for st in (0, 1)] for b in range(B) for layer in range(2)]
    windows = [sc.sess.gather_window(b, layer) for b in range(B) for layer in range(2)] if sc.sess.window else []
    return cnt, lists, stores, windows, outs


def _same(a, b, what):
    if isinstance(a, (list, tuple)):
        assert len(a) == len(b), what
        for i, (x, y) in enumerate(zip(a, b)):
            _same(x, y, f"{what}[{i}]")
    else:
        assert np.array_equal(np.asarray(a), np.asarray(b)), what


@pytest.mark.parametrize("B,Hq,Hkv,D,window,controller", [
    (5, 32, 8, 128, 0, False),        # 40 segments: equal ranges, sliced merge
    (12, 64, 8, 128, 0, False),       # 96 segments: per-XCD ranges, four-wave workgroups
    (12, 16, 4, 64, 24, True),        # recent window and the online controller
])
def test_two_runs_bit_identical(B, Hq, Hkv, D, window, controller):
    say(f"case: determinism B={B} Hq={Hq} Hkv={Hkv} D={D} W={window} controller={controller}")
    rng = np.random.default_rng(B * 7 + D)
    P = rng.integers(1, 700, size=B)
    T = 40
    pol = make_policy(6, 2, 2, 0.33, seed=900 + B)
    pol.recent_window = window
    states = None
    if controller:
        ts = [function_call_tags_with_states(T, 950 + b) for b in range(B)]
        tags = np.stack([t for t, _ in ts])
        states = np.stack([s for _, s in ts])
        cal = [function_call_tags_with_states(T, 990 + i) for i in range(4)]
        pol = with_budget_controller(pol, cal, len(PARSER_STATES), CRITICAL_STATES)
    else:
        tags = np.stack([function_call_tags(T, 950 + b) for b in range(B)])
    first = _run(pol, B, Hq, Hkv, D, P, tags, seed=77, states=states)
    second = _run(pol, B, Hq, Hkv, D, P, tags, seed=77, states=states)
    for name, a, b in zip(("counters", "index lists", "stores", "windows", "attention outputs"), first, second):
        _same(a, b, name)
    say("two runs bit-identical")


@pytest.mark.parametrize("B,Hq,Hkv,D,window,tagged", [
    (5, 32, 8, 128, 0, False),        # few segments
    (12, 64, 8, 128, 0, True),        # many segments, tagged prompts (LOW-heavy, partial pages)
    (7, 16, 4, 64, 21, False),        # recent window
])
def test_unwritten_memory_never_reaches_a_result(B, Hq, Hkv, D, window, tagged):
    say(f"case: prefilled caches B={B} Hq={Hq} Hkv={Hkv} D={D} W={window} tagged={tagged}")
    from workload.tags import schema_prompt_tags
    rng = np.random.default_rng(B * 11 + D)
    P = rng.integers(1, 500, size=B)
    T = 37
    tags = np.stack([function_call_tags(T, 970 + b) for b in range(B)])
    ptags = None
    if tagged:
        pol = make_policy(12, 2, 2, 0.33, seed=930 + B, n_sink=4)
        ptags = np.zeros((B, int(P.max())), np.uint8)
        for b, p in enumerate(P):
            ptags[b, :p] = schema_prompt_tags(int(p), 940 + b)
    else:
        pol = make_policy(6, 2, 2, 0.33, seed=930 + B)
    pol.recent_window = window
    runs = [_run(pol, B, Hq, Hkv, D, P, tags, seed=78, prefill=fill, prompt_tags=ptags) for fill in (0x00, 0xFF, 0x7F)]
    for other in runs[1:]:
        for name, a, b in zip(("counters", "index lists", "stores", "windows", "attention outputs"), runs[0], other):
            _same(a, b, name)
    say("prefill patterns 0x00 / 0xFF / 0x7F give the same bits")
