"""Parity of the online budget controller (Alg. 2; Eq. 9-10) on the HIP path
with the CPU oracle: tokens carry parser states, every layer's remaining
budget R, every decision, list, counter, code and scale bit-exact, attention
within |gpu - ref| <= 2e-3 + 1e-2 |ref|."""

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import Scenario, bits16, budgets, policy_dict, say
from workload import make_policy
from workload.policy import pack_blob, with_budget_controller
from workload.tags import CRITICAL_STATES, PARSER_STATES, tag_mix, function_call_tags_with_states
from workload.tensors import bf16_normal, sub_seed

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def controller_policy(n_groups, n_layers, beta, seed, n_sink, cal_len):
    """A 6-tag table plus the controller's reserve, calibrated on four tagged
    traces of cal_len tokens."""
    cal = [function_call_tags_with_states(cal_len, sub_seed(seed, "tags", 100 + i)) for i in range(4)]
    probs = tag_mix(np.concatenate([c[0] for c in cal]), 6)
    pol = make_policy(6, n_groups, n_layers, beta, seed, tag_probs=probs, n_sink=n_sink)
    return with_budget_controller(pol, cal, len(PARSER_STATES), CRITICAL_STATES)


def replay_changes(pol, tags, states, t_max, Hkv, D):
    """Oracle-only replay of one sequence: (demoted, promoted) group actions
    relative to the static lookup of Eq. 10."""
    m = oracle.group_costs(pol.group_of_layer, pol.n_groups, Hkv, D)
    gamma = oracle.reserve_bytes(pol.reserve_q, m)
    R = oracle.initial_budget(pol.beta_q, t_max, m)
    dem = pro = 0
    for i, (z, s) in enumerate(zip(tags, states)):
        forced = i < pol.n_sink
        known = int(s) < pol.n_states
        a, cost = oracle.online_actions(int(z), int(s), R, pol.action, pol.floor, pol.rho_up, m,
                                        gamma[s] if known else 0, bool(pol.crit[s]) if known else False, forced)
        static = np.full(pol.n_groups, oracle.HIGH) if forced else np.maximum(pol.action[z], pol.floor[z])
        dem += int((a < static).sum())
        pro += int((a > static).sum())
        R -= cost
    return dem, pro, R


@pytest.mark.parametrize("Hq,Hkv,D", [(8, 2, 64), (32, 8, 128), (20, 5, 64)])
def test_controller_bulk_step_and_fused(Hq, Hkv, D):
    """3 sequences, 4 layers in 2 groups, 3 sinks; prompts of 0 / 37 / 300
    tokens kept HIGH (they bypass the controller), then 600 generated tokens
    with tagger tags and parser states: 0..519 bulk-appended in two calls
    (the controller walks several 256-token chunks), 520..539 one-token
    appends, 540..599 fused append + attention.  R_0 from beta = 0.33 and
    T_max = 600 runs out part-way, so tokens are both demoted and promoted and
    R ends below zero.  Sequence 2 carries an unknown parser state at two
    positions (flagged, decided with Gamma = 0 and no promotion)."""
    say(f"case: controller Hq={Hq} Hkv={Hkv} D={D}")
    T, seed = 600, 11
    pol = controller_policy(2, 4, 0.33, seed, n_sink=3, cal_len=600)
    ts = [function_call_tags_with_states(T, sub_seed(seed, "tags", b)) for b in range(3)]
    tags = np.stack([t for t, _ in ts])
    states = np.stack([s for _, s in ts]).astype(np.uint8)
    states[2, 100] = 200
    states[2, 560] = 7
    dem, pro, R_end = replay_changes(pol, tags[0], states[0], T, Hkv, D)
    say(f"oracle replay of sequence 0: {dem} demoted, {pro} promoted group actions, final R {R_end}")
    assert dem > 100 and pro > 100 and R_end < 0
    from paper_2608_28276_amd.pask import PASK_FLAG_BAD_STATE
    sc = Scenario(pol, B=3, L=4, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=[0, 37, 300], gen_tags=tags, seed=seed + D,
                  gen_states=states)
    sc.budget_init(T)
    sc.fill_prompt()
    sc.check_state()
    sc.append_steps(0, 300)
    sc.expect_flags = PASK_FLAG_BAD_STATE        # position 100 of sequence 2
    sc.append_steps(300, 520)
    sc.check_state()
    for t in range(520, 540):
        sc.append_steps(t, t + 1)
    sc.check_state()
    worst = 0.0
    for t in range(540, 600):
        worst = max(worst, sc.decode_step(t, check=(t % 15 == 0 or t == 599)))
    assert sc.oc.bad_state
    R = budgets(sc.sess.counters().cpu().numpy())[:3]
    say(f"final R per sequence (layer 0): {R[:, 0].tolist()}; worst |err| {worst:.2e}")
    assert (R == R[:, :1]).all(), "every layer holds the same R"


def test_controller_without_budget_init_and_keep_all_bypass():
    """Parser states before pask_budget_init, and again after a cache reset:
    decisions fall back to Eq. 10 and PASK_FLAG_NO_BUDGET is set.  A keep-all
    append that passes states leaves R unchanged."""
    from paper_2608_28276_amd import pask
    from paper_2608_28276_amd.session import PaskSession
    say("case: controller set-up and bypass")
    pol = controller_policy(2, 2, 0.33, 5, n_sink=0, cal_len=300)
    B, n, Hkv, D = 2, 300, 2, 64
    sess = PaskSession(pack_blob(pol), max_batch=B, n_layers=2, n_q_heads=8, n_kv_heads=Hkv, head_dim=D,
                       max_tokens_per_seq=2 * n, hi_pages=2 * B * 2 * n // 16, lo_pages=2 * B * 2 * n // 16)
    dev = sess.device
    ts = [function_call_tags_with_states(n, sub_seed(5, "tags", b)) for b in range(B)]
    tags = np.stack([t for t, _ in ts])
    states = np.stack([s for _, s in ts]).astype(np.uint8)
    k = bf16_normal((B, n, Hkv, D), 1)
    v = bf16_normal((B, n, Hkv, D), 2)
    put = lambda x: torch.as_tensor(x, device=dev)
    for trial in ("fresh", "after_reset"):
        if trial == "after_reset":
            sess.budget_init(n, batch=B)
            sess.reset()
        sess.append(0, put(tags), k.to(dev), v.to(dev), states=put(states))       # bulk path
        for t in range(4):                                                        # one-token path
            sess.append(1, put(tags[:, t:t + 1].copy()), k[:, t:t + 1].contiguous().to(dev),
                        v[:, t:t + 1].contiguous().to(dev), states=put(states[:, t:t + 1].copy()))
        st, status, _ = sess.stats(batch=B)
        assert st.device_flags == pask.PASK_FLAG_NO_BUDGET, (trial, hex(st.device_flags))
        il = sess.index_lists().cpu().numpy()
        cnt = sess.counters().cpu().numpy()
        for layer, m_tok in ((0, n), (1, 4)):
            for b in range(B):
                acts, _, _ = oracle.decide(tags[b, :m_tok], np.arange(m_tok), int(pol.group_of_layer[layer]),
                                           pol.action, pol.floor, pol.n_sink, False)
                hi, lo = oracle.compact(acts, np.arange(m_tok))
                assert (cnt[b, layer, 0], cnt[b, layer, 1]) == (hi.size, lo.size), (trial, layer, b)
                assert (il[b, layer, 0, :hi.size] == hi).all() and (il[b, layer, 1, :lo.size] == lo).all()
                assert budgets(cnt[b, layer]) == 0
    sess.reset()
    sess.budget_init(n, batch=B)
    r0 = oracle.initial_budget(pol.beta_q, n, oracle.group_costs(pol.group_of_layer, 2, Hkv, D))
    sess.append(0, None, k.to(dev), v.to(dev), keep_all=True, states=put(states))
    st, status, _ = sess.stats(batch=B)
    assert st.device_flags == 0 and st.n_forced_high == B * n
    got = budgets(sess.counters().cpu().numpy())[:B]
    assert (got == r0).all(), (got, r0)
    say(f"R_0 = {r0} in every layer; keep-all append left it unchanged")


def test_controller_one_token_path_matches_oracle_every_step():
    """One sequence through the fused call only, every layer compared after
    every step: the decode step's controller (one thread, table read from
    device memory) against the oracle, with 16 sinks and the budget tight
    enough that R crosses zero."""
    say("case: controller, fused steps only")
    T = 160
    pol = controller_policy(2, 2, 0.25, 23, n_sink=16, cal_len=T)
    tags, states = function_call_tags_with_states(T, sub_seed(23, "tags", 0))
    sc = Scenario(pol, B=1, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[0], gen_tags=tags[None],
                  gen_states=states[None], seed=23)
    sc.budget_init(T // 2)
    for t in range(T):
        sc.decode_step(t)
    R = int(budgets(sc.sess.counters().cpu().numpy())[0, 0])
    assert R == sc.oc.counts(0, 0)["R"] and R < 0
