"""Parity of the protected recent window (Section 3.1) on the HIP path with
the CPU oracle: the last W positions of every (sequence, layer) are held at
bf16 and attended whatever their action; a token is persisted by its action
(taken when it was appended) when it leaves the window.  Window contents,
decisions, lists, counters, codes and scales bit-exact; attention within
|gpu - ref| <= 2e-3 + 1e-2 |ref|."""

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import Scenario, budgets, say
from workload import make_policy, function_call_tags
from workload.policy import uniform_policy, with_budget_controller
from workload.tags import CRITICAL_STATES, PARSER_STATES, function_call_tags_with_states
from workload.tensors import sub_seed

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def _windowed(pol, W):
    pol.recent_window = W
    return pol


@pytest.mark.parametrize("Hq,Hkv,D,W", [(8, 2, 64, 16), (8, 2, 64, 37), (32, 8, 128, 16), (64, 8, 128, 53),
                                        (12, 3, 128, 24)])
def test_window_bulk_step_and_fused(Hq, Hkv, D, W):
    """3 sequences, 4 layers in 2 groups, 3 sinks, prompts of 0 / 37 / 300
    tokens kept HIGH (they pass through the window too), then 900 generated
    tagger-tagged tokens: bulk appends of 5, 195 and 600 tokens (several
    256-entry chunks, entries leaving from the window and from the call
    itself), one-token appends, then fused append + attention steps."""
    say(f"case: window W={W} Hq={Hq} Hkv={Hkv} D={D}")
    T = 900
    pol = _windowed(make_policy(6, 2, 4, 0.33, seed=W + D, n_sink=3), W)
    tags = np.stack([function_call_tags(T, sub_seed(W, "tags", b)) for b in range(3)])
    sc = Scenario(pol, B=3, L=4, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=[0, 37, 300], gen_tags=tags, seed=W * 7 + D)
    sc.fill_prompt()
    sc.check_state()
    sc.append_steps(0, 5)
    sc.append_steps(5, 200)
    sc.check_state()
    sc.append_steps(200, 800)
    sc.check_state()
    for t in range(800, 840):
        sc.append_steps(t, t + 1)
    sc.check_state()
    worst = 0.0
    for t in range(840, 900):
        worst = max(worst, sc.decode_step(t, check=(t % 20 == 0 or t == 899)))
    say(f"window W={W}: worst |err| {worst:.2e}")


def test_window_all_drop_sees_prompt_and_last_w():
    """All-DROP table, W = 24: attention at every step sees the 40-token
    prompt and the last 24 positions only (the prompt's tokens included
    while they are inside the window)."""
    say("case: window, all-DROP")
    pol = _windowed(uniform_policy(6, 2, 2, oracle.DROP), 24)
    T = 70
    tags = np.stack([function_call_tags(T, 3 + b) for b in range(2)])
    sc = Scenario(pol, B=2, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[0, 40], gen_tags=tags, seed=5)
    sc.fill_prompt()
    for t in range(T):
        sc.decode_step(t)
    sc.check_state()
    hi, lo = sc.oc.lists(1, 0)
    assert hi.tolist() == list(range(40)) and lo.size == 0
    assert sc.oc.counts(0, 0)["drop"] == T - 24


def test_window_larger_than_the_sequence():
    """W = max_tokens_per_seq: nothing ever leaves the window, every token is
    attended at bf16 and the stores stay empty."""
    say("case: window covering the sequence")
    T = 48
    tags = function_call_tags(T, 9)[None]
    pol = _windowed(make_policy(6, 2, 2, 0.33, seed=4), 16 + T)
    sc = Scenario(pol, B=1, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[16], gen_tags=tags, seed=6)
    sc.fill_prompt()
    sc.append_steps(0, 20)
    for t in range(20, T):
        sc.decode_step(t)
    sc.check_state()
    c = sc.oc.counts(0, 1)
    assert (c["hi"], c["lo"], c["drop"], c["window"]) == (0, 0, 0, 16 + T)


def test_window_with_the_online_controller():
    """Parser states and W = 20: the controller decides and charges R when a
    token is appended; the window delays its persistence.  R, decisions,
    lists, window and stores bit-exact; an unknown state is flagged."""
    from paper_2608_28276_amd.pask import PASK_FLAG_BAD_STATE
    say("case: window + controller")
    T, W = 400, 20
    cal = [function_call_tags_with_states(T, sub_seed(31, "tags", 100 + i)) for i in range(4)]
    pol = make_policy(6, 2, 4, 0.33, seed=31, n_sink=2)
    pol = _windowed(with_budget_controller(pol, cal, len(PARSER_STATES), CRITICAL_STATES), W)
    ts = [function_call_tags_with_states(T, sub_seed(31, "tags", b)) for b in range(2)]
    tags = np.stack([t for t, _ in ts])
    states = np.stack([s for _, s in ts]).astype(np.uint8)
    states[1, 50] = 99
    sc = Scenario(pol, B=2, L=4, Hq=16, Hkv=8, D=64, prompt_lens=[0, 64], gen_tags=tags, seed=31,
                  gen_states=states)
    sc.budget_init(T)
    sc.fill_prompt()
    sc.append_steps(0, 40)
    sc.check_state()
    sc.append_steps(40, 300)
    sc.expect_flags = PASK_FLAG_BAD_STATE
    sc.check_state()
    for t in range(300, 340):
        sc.append_steps(t, t + 1)
    for t in range(340, 400):
        sc.decode_step(t, check=(t % 10 == 0 or t == 399))
    R = budgets(sc.sess.counters().cpu().numpy())[:2]
    assert (R == R[:, :1]).all()
    say(f"final R {R[:, 0].tolist()}")
