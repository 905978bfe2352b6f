"""Parity at the workloads' full sizes (shapes, batch, prompt lengths and
layer counts of the five workloads), each checked as far as the oracle can
follow in seconds: every decision, list and counter of every sequence, and
the stored bits, codes and attention outputs of sampled (sequence, layer)
pairs."""

import numpy as np
import pytest
import torch

from tests.gpu_util import Scenario, say
from workload import CONFIGS, make_policy, prompt_lengths, tag_mix, function_call_tags
from workload.tags import schema_prompt_tags
from workload.tensors import sub_seed

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def _call_tags(cfg, n):
    return np.stack([function_call_tags(n, sub_seed(cfg.seed, "tags", b)) for b in range(cfg.batch)])


def _calls_policy(cfg, beta=0.33):
    probs = tag_mix(function_call_tags(200000, sub_seed(cfg.seed, "tags", 1 << 20)), 6)
    return make_policy(6, cfg.n_groups, cfg.n_layers, beta, cfg.seed, tag_probs=probs)


def test_qwen3_4b_one_sequence_every_step():
    """1 sequence, 36 layers in 4 groups, 32 query / 8 KV heads, head_dim 128,
    a 2048-token prompt kept HIGH and 512 generated tokens with tagger tags,
    each through the fused append + attention call on every layer: every
    decision, list, code and scale bit-exact; attention at steps 0, 1, 127,
    255 and 511 on all 36 layers."""
    cfg = CONFIGS[1]
    say(f"case: {cfg.name}")
    pol = _calls_policy(cfg)
    tags = _call_tags(cfg, cfg.gen_tokens)
    sc = Scenario(pol, B=1, L=cfg.n_layers, Hq=cfg.n_q_heads, Hkv=cfg.n_kv_heads, D=cfg.head_dim,
                  prompt_lens=prompt_lengths(cfg), gen_tags=tags, seed=cfg.seed)
    sc.fill_prompt()
    checked = (0, 1, 127, 255, 511)
    worst = 0.0
    for t in range(cfg.gen_tokens):
        worst = max(worst, sc.decode_step(t, check=t in checked))
        if t in checked:
            say(f"step {t}: 36 layers within tolerance")
    sc.check_state()
    say(f"{cfg.name}: worst |err| {worst:.2e}")


def test_qwen3_4b_batch64_bench_launch():
    """The timed workload in the launch configuration the bench times: 64
    sequences, prompts U{1024..8192} kept HIGH, 512 generated tokens
    bulk-appended, then decode steps over all 36 layers, each one
    pask_decode_attn call that persists the step's token (the attention and
    merge kernels do it themselves at this batch) with the bench's workspace
    hint.  Every counter and list of all 64 sequences x 36 layers bit-exact;
    attention of all 64 sequences in the first layer of each group at two
    steps; stores of all 64 sequences in layer 27 and of 7 sequences x the
    first layer of each group."""
    from bench import build_workload
    from tests.fullsize_util import DeviceRun
    cfg, P, tags, pol, _ = build_workload(2)
    say(f"case: {cfg.name}")
    layers = (0, 9, 18, 27)
    sample = sorted({(b, l) for b in range(cfg.batch) for l in layers})
    stores = sorted({(b, l) for b in (0, 9, 21, 33, 42, 50, 63) for l in layers} |
                    {(b, 27) for b in range(cfg.batch)})
    run = DeviceRun(pol, n_layers=cfg.n_layers, layers=range(cfg.n_layers), Hq=cfg.n_q_heads,
                    Hkv=cfg.n_kv_heads, D=cfg.head_dim, P=P, prompt_tags=None, gen_tags=tags, sample=sample,
                    seed=cfg.seed, n_bulk=512, n_steps=3)
    run.fill()
    run.step(check=True, fused=True)
    run.step(check=False, fused=True)
    run.step(check=True, fused=True)
    run.check_lists()
    run.check_stores(stores)


@pytest.mark.parametrize("beta", [0.25, 0.33, 0.5, 1.0])
def test_qwen3_4b_batch128_tagged_prompts_budget_sweep(beta):
    """128 sequences, prompts U{4096..16384} labelled by the schema-prompt
    tagger and persisted through the same 12-tag table (prompt-side
    companion, 16 sinks), bulk-appended after prefill, then 64 generated
    tokens and two fused decode steps, at budgets 0.25 / 0.33 / 0.5 / 1.0.
    Driven layers: the first of each of the 4 groups.  Every counter and list
    bit-exact; stores and attention of 3 sequences x 4 layers, and at budget
    0.33 of 5 more sequences in layer 27."""
    from tests.fullsize_util import DeviceRun
    cfg = CONFIGS[3]
    say(f"case: {cfg.name} at budget {beta}")
    P = prompt_lengths(cfg)
    ptags = np.zeros((cfg.batch, int(P.max())), np.uint8)
    for b, p in enumerate(P):
        ptags[b, :p] = schema_prompt_tags(int(p), sub_seed(cfg.seed, "prompt_tags", b))
    gtags = _call_tags(cfg, 66)
    probs = tag_mix(np.concatenate([ptags[b, :P[b]] for b in range(cfg.batch)] + [gtags.ravel()]), 12)
    pol = make_policy(12, cfg.n_groups, cfg.n_layers, beta, cfg.seed, tag_probs=probs, n_sink=cfg.n_sink)
    say(f"policy expected cost {pol.expected_cost:.3f}")
    layers = (0, 9, 18, 27)
    sample = [(b, l) for b in (3, 64, 127) for l in layers]
    if beta == 0.33:
        sample += [(b, 27) for b in (17, 40, 77, 100, 115)]
    run = DeviceRun(pol, n_layers=cfg.n_layers, layers=layers, Hq=cfg.n_q_heads, Hkv=cfg.n_kv_heads,
                    D=cfg.head_dim, P=P, prompt_tags=ptags, gen_tags=gtags, sample=sample, seed=cfg.seed,
                    n_bulk=64, n_steps=2)
    run.fill()
    run.step(check=False, fused=True)
    run.step(check=True, fused=True)
    run.check_lists()
    run.check_stores()


def test_qwen3_32b_attention_batch256_one_layer_group():
    """One GPU's share of the 64-layer Qwen3-32B attention workload: 256
    sequences, prompts log-uniform over 16k..32k tokens kept HIGH, 64 query /
    8 KV heads (group 8), head_dim 128; two layers of the resident group, 256
    generated tokens bulk-appended, then two fused decode steps.  Every
    counter and list bit-exact; stores and attention of 6 sequences x 2
    layers and of 10 more sequences in the first layer."""
    from tests.fullsize_util import DeviceRun
    cfg = CONFIGS[4]
    say(f"case: {cfg.name}")
    P = prompt_lengths(cfg)
    tags = _call_tags(cfg, 258)
    pol = _calls_policy(cfg)
    layers = (0, 5)
    sample = [(b, l) for b in (0, 63, 64, 130, 200, 255) for l in layers]
    sample += [(b, layers[0]) for b in (17, 40, 90, 101, 150, 170, 190, 222, 240, 250)]
    run = DeviceRun(pol, n_layers=cfg.n_layers, layers=layers, Hq=cfg.n_q_heads, Hkv=cfg.n_kv_heads,
                    D=cfg.head_dim, P=P, prompt_tags=None, gen_tags=tags, sample=sample, seed=cfg.seed,
                    n_bulk=256, n_steps=2)
    run.fill()
    run.step(check=False, fused=True)
    run.step(check=True, fused=True)
    run.check_lists()
    run.check_stores()


def test_qwen3_4b_batch64_online_controller():
    """The timed workload's shapes under the online controller (Alg. 2): 64
    sequences, 36 layers in 4 groups, prompts U{1024..8192} kept HIGH (they
    bypass the controller), 512 generated tokens with tagger tags and parser
    states bulk-appended, then a one-token append step and two fused steps;
    R_0 from the table's beta with T_max = 515.  Every counter, list and
    remaining budget of all 64 sequences x 36 layers bit-exact; stores and
    attention of 6 sequences x the first layer of each group."""
    from bench import build_workload
    from tests.fullsize_util import DeviceRun
    from workload.policy import with_budget_controller
    from workload.tags import CRITICAL_STATES, PARSER_STATES, function_call_tags_with_states
    cfg, P, tags, pol, _ = build_workload(2)
    say(f"case: {cfg.name} with the online controller")
    n_gen = 515
    ts = [function_call_tags_with_states(cfg.gen_tokens, sub_seed(cfg.seed, "tags", b)) for b in range(cfg.batch)]
    assert all((t == tags[b]).all() for b, (t, _) in enumerate(ts))
    states = np.stack([s for _, s in ts])
    cal = [function_call_tags_with_states(n_gen, sub_seed(cfg.seed, "tags", 1000 + i)) for i in range(8)]
    pol = with_budget_controller(pol, cal, len(PARSER_STATES), CRITICAL_STATES)
    sample = [(b, l) for b in (0, 13, 31, 40, 52, 63) for l in (0, 9, 18, 27)]
    run = DeviceRun(pol, n_layers=cfg.n_layers, layers=range(cfg.n_layers), Hq=cfg.n_q_heads,
                    Hkv=cfg.n_kv_heads, D=cfg.head_dim, P=P, prompt_tags=None, gen_tags=tags, sample=sample,
                    seed=cfg.seed, n_bulk=512, n_steps=3, gen_states=states, t_max=n_gen)
    run.fill()
    run.check_lists()
    run.step(check=False)
    run.step(check=True, fused=True)
    run.step(check=True, fused=True)
    run.check_lists()
    run.check_stores()


def test_qwen3_4b_batch64_recent_window():
    """The timed workload's shapes with a protected recent window of 64
    positions (Section 3.1): 64 sequences, 36 layers, prompts U{1024..8192}
    kept HIGH (their last 64 positions pass through the window), 512
    generated tokens bulk-appended, then a one-token append step and two
    fused steps.  Every counter and list of all 64 sequences x 36 layers
    bit-exact; window contents, stores and attention of 6 sequences x the
    first layer of each group."""
    from bench import build_workload
    from tests.fullsize_util import DeviceRun
    cfg, P, tags, pol, _ = build_workload(2)
    pol.recent_window = 64
    say(f"case: {cfg.name} with a 64-position recent window")
    sample = [(b, l) for b in (1, 17, 30, 44, 58, 62) for l in (0, 9, 18, 27)]
    run = DeviceRun(pol, n_layers=cfg.n_layers, layers=range(cfg.n_layers), Hq=cfg.n_q_heads,
                    Hkv=cfg.n_kv_heads, D=cfg.head_dim, P=P, prompt_tags=None, gen_tags=tags, sample=sample,
                    seed=cfg.seed, n_bulk=512, n_steps=3)
    run.fill()
    run.check_lists()
    run.step(check=False)
    run.step(check=True, fused=True)
    run.step(check=True, fused=True)
    run.check_lists()
    run.check_stores()
