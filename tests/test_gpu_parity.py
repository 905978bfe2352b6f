"""Parity of the HIP path (through the C ABI) with the CPU oracle."""

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import Scenario, assert_attn_close, bits16, say
from workload import CONFIGS, make_policy, function_call_tags
from workload.policy import uniform_policy
from workload.tags import iid_tags, tag_mix
from workload.tensors import sub_seed

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_28276_amd.pask  # noqa: F401  (fails loudly when libpask.so is missing)


def test_tiny_config_every_step():
    """1 sequence, 2 layers in 2 groups, 8 query / 2 KV heads, head_dim 64;
    256 prompt tokens kept HIGH then 128 generated tokens with i.i.d. tags:
    fused append + attention every step, every layer."""
    cfg = CONFIGS[0]
    say("case: tiny config, every step")
    pol = make_policy(6, cfg.n_groups, cfg.n_layers, 0.33, cfg.seed)
    tags = iid_tags(cfg.gen_tokens, sub_seed(cfg.seed, "tags", 0))[None]
    sc = Scenario(pol, B=1, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[256], gen_tags=tags, seed=cfg.seed)
    sc.fill_prompt()
    worst = 0.0
    for t in range(cfg.gen_tokens):
        worst = max(worst, sc.decode_step(t))
        if t in (0, 17, 127):
            sc.check_state()
    say(f"tiny config: worst |err| {worst:.2e}")


def test_quantiser_exhaustive_absmax_on_gpu():
    """Every non-negative finite bf16 absmax (32,640 values), plus exact-tie
    groups and random groups, through both append paths (bulk and one token
    per step), codes and scales bit-exact against the oracle."""
    say("case: quantiser exhaustive")
    rng = np.random.default_rng(5)
    absmax = np.arange(0x0000, 0x7F80, dtype=np.int64)
    groups = []
    for a in absmax:
        frac = rng.uniform(-1, 1, size=31)
        av = float(torch.tensor([int(a)], dtype=torch.int16).view(torch.bfloat16).float())
        g = torch.tensor(np.concatenate([[av], frac * av]), dtype=torch.float32).to(torch.bfloat16)
        g = g[torch.as_tensor(rng.permutation(32))]
        groups.append(bits16(g))
    for k in range(-30, 20):
        s = 2.0 ** k
        h = rng.integers(-7, 7, size=31) + 0.5
        g = torch.tensor(np.concatenate([[7 * s], h * s]), dtype=torch.float32).to(torch.bfloat16)
        groups.append(bits16(g))
    x = np.stack(groups)                                        # [n_groups, 32] bf16 bits
    per_tok = 2 * 8 * 4                                         # K and V, 8 heads, 4 groups of 32
    n_tok = -(-x.shape[0] // per_tok)
    pad = n_tok * per_tok - x.shape[0]
    x = np.concatenate([x, np.zeros((pad, 32), np.uint16)])
    kv = x.reshape(n_tok, 2, 8, 128)
    k = torch.from_numpy(kv[:, 0].astype(np.int16)).view(torch.bfloat16)
    v = torch.from_numpy(kv[:, 1].astype(np.int16)).view(torch.bfloat16)
    pol = uniform_policy(6, 1, 2, oracle.LOW)
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob
    sess = PaskSession(pack_blob(pol), max_batch=1, n_layers=2, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       max_tokens_per_seq=n_tok, hi_pages=4, lo_pages=2 * (n_tok // 16 + 1))
    dev = sess.device
    tags = torch.zeros((1, n_tok), dtype=torch.uint8, device=dev)
    sess.append(0, tags, k[None].to(dev), v[None].to(dev))                      # bulk path
    q = torch.zeros((1, 32, 128), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    for i in range(n_tok):                                                     # one token per step
        sess.decode(1, q, out, None, tags[:, i].contiguous(), k[i][None].to(dev), v[i][None].to(dev))
    torch.cuda.synchronize()
    kc_ref, ks_ref = oracle.quantize_groups(bits16(k))
    vc_ref, vs_ref = oracle.quantize_groups(bits16(v))
    for layer in (0, 1):
        kc, ks, vc, vs = sess.gather_store(0, layer, 1)
        assert kc.shape[0] == n_tok
        assert (ks == ks_ref).all(), f"layer {layer}: K scales"
        assert (vs == vs_ref).all(), f"layer {layer}: V scales"
        assert (kc == kc_ref).all(), f"layer {layer}: K codes"
        assert (vc == vc_ref).all(), f"layer {layer}: V codes"


@pytest.mark.parametrize("Hq,Hkv,D", [(8, 8, 64), (16, 8, 64), (8, 2, 64), (16, 2, 64),
                                      (8, 8, 128), (16, 8, 128), (32, 8, 128), (64, 8, 128),
                                      (1, 1, 64), (6, 3, 64), (12, 3, 128), (40, 5, 128), (7, 7, 128)])
def test_geometries_mixed_policy(Hq, Hkv, D):
    """Every supported (group size, head_dim) pair, and KV head counts that
    are not powers of two (a page's chunk rows then do not divide the pack's
    256 threads; the head rotation of the pages wraps at 3, 5, 7); ragged
    prompts (not page multiples), a batch of 5, mixed HIGH / LOW / DROP decode
    tokens."""
    say(f"case: geometry Hq={Hq} Hkv={Hkv} D={D}")
    pol = make_policy(6, 2, 4, 0.33, seed=Hq * 100 + D)
    P = [1, 15, 17, 33, 300]
    T = 40
    tags = np.stack([function_call_tags(T, 50 + b) for b in range(5)])
    sc = Scenario(pol, B=5, L=4, Hq=Hq, Hkv=Hkv, D=D, prompt_lens=P, gen_tags=tags, seed=77 + D + Hq)
    sc.fill_prompt()
    sc.append_steps(0, 20)
    sc.decode_step(20)
    sc.append_steps(21, 39)
    sc.decode_step(39)
    sc.check_state()


@pytest.mark.parametrize("B", [256, 260])
def test_decode_batch_around_single_call_limit(B):
    """Up to 256 sequences a decode call with new tokens persists them in its
    own attention and merge kernels; above, it runs the one-token append
    kernel first.  Both sides of the limit: ragged short prompts (some empty),
    mixed HIGH / LOW / DROP tokens, three steps, every sequence compared."""
    say(f"case: decode batch {B}")
    pol = make_policy(6, 2, 2, 0.33, seed=900 + B)
    P = [(7 * b) % 45 for b in range(B)]
    T = 3
    tags = np.stack([function_call_tags(T, 1000 + b) for b in range(B)])
    sc = Scenario(pol, B=B, L=2, Hq=8, Hkv=2, D=64, prompt_lens=P, gen_tags=tags, seed=B)
    sc.fill_prompt()
    for t in range(T):
        sc.decode_step(t)
    sc.check_state()


@pytest.mark.parametrize("B", [8, 9])
def test_segment_count_boundary(B):
    """8 sequences x 8 KV heads = 64 segments take the few-segment path
    (pieces of 4 pages, sliced merge), 9 x 8 = 72 the general one; prompts of
    18-40 pages so every segment is cut into several pieces."""
    say(f"case: segment boundary B={B}")
    pol = make_policy(6, 2, 2, 0.33, seed=500 + B)
    P = [280 + 37 * b for b in range(B)]
    T = 6
    tags = np.stack([function_call_tags(T, 70 + b) for b in range(B)])
    sc = Scenario(pol, B=B, L=2, Hq=32, Hkv=8, D=128, prompt_lens=P, gen_tags=tags, seed=300 + B)
    sc.fill_prompt()
    sc.append_steps(0, 4)
    sc.decode_step(4)
    sc.decode_step(5)
    sc.check_state()


def test_all_drop_and_empty_history():
    """All-DROP table: a sequence with no prompt has an empty history
    (out = 0, lse = -inf); one with a prompt sees only the prompt."""
    say("case: all-DROP / empty history")
    pol = uniform_policy(6, 2, 2, oracle.DROP)
    tags = iid_tags(8, 3)[None].repeat(2, axis=0)
    sc = Scenario(pol, B=2, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[0, 40], gen_tags=tags, seed=9)
    sc.fill_prompt()
    for t in range(8):
        sc.decode_step(t)
    sc.check_state()


def test_sinks_keep_first_positions_high():
    say("case: sinks")
    pol = uniform_policy(6, 2, 2, oracle.DROP, n_sink=5)
    tags = iid_tags(30, 4)[None]
    sc = Scenario(pol, B=1, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[0], gen_tags=tags, seed=10)
    sc.append_steps(0, 3)
    for t in range(3, 30):
        sc.decode_step(t)
    sc.check_state()
    hi, lo = sc.oc.lists(0, 0)
    assert hi.tolist() == [0, 1, 2, 3, 4] and lo.size == 0


def test_prompt_side_persistence_tagged_prompt():
    """Prompt tokens governed by a 12-tag table (6 decode tags, 6 prompt
    labels) with 16 sinks, appended in bulk after prefill."""
    say("case: tagged prompt")
    from workload.tags import schema_prompt_tags
    pol = make_policy(12, 2, 2, 0.33, seed=12, n_sink=16)
    P = [700, 1030, 5]
    ptags = np.zeros((3, max(P)), np.uint8)
    for b, p in enumerate(P):
        ptags[b, :p] = schema_prompt_tags(p, 20 + b)
    tags = np.stack([function_call_tags(24, 30 + b) for b in range(3)])
    sc = Scenario(pol, B=3, L=2, Hq=8, Hkv=2, D=64, prompt_lens=P, gen_tags=tags, seed=13, prompt_tags=ptags)
    sc.fill_prompt()
    sc.decode_step(0)
    sc.append_steps(1, 23)
    sc.decode_step(23)
    sc.check_state()


def test_small_ctx_hint_grid_stride():
    """A max_ctx_hint far below the real history: a workspace with room for
    few partials per (sequence, KV head) forces larger per-block page
    ranges; results unchanged."""
    say("case: small ctx hint")
    pol = make_policy(6, 2, 2, 0.33, seed=14)
    tags = iid_tags(10, 5)[None].repeat(2, axis=0)
    sc = Scenario(pol, B=2, L=2, Hq=8, Hkv=2, D=64, prompt_lens=[1500, 2100], gen_tags=tags, seed=15,
                  max_ctx_hint=100)
    sc.fill_prompt()
    sc.decode_step(0)
    sc.check_state()


def test_batch_beyond_64_sequences():
    """150 sequences (three 64-sequence chunks in the attention work plan, the
    last ragged), about one in five with no prompt, short ragged prompts and
    three long ones (at indices 5, 70 and 140, each split over several
    blocks): the plan, the block search, the walk to the next sequence and the
    merge read counts beyond the first 64 sequences."""
    say("case: batch of 150")
    rng = np.random.default_rng(21)
    B = 150
    P = rng.integers(1, 90, size=B)
    P[rng.random(B) < 0.2] = 0
    P[[5, 70, 140]] = [700, 1000, 913]
    pol = make_policy(6, 2, 2, 0.33, seed=21)
    tags = np.stack([function_call_tags(12, 60 + b) for b in range(B)])
    sc = Scenario(pol, B=B, L=2, Hq=8, Hkv=2, D=64, prompt_lens=P, gen_tags=tags, seed=21)
    sc.fill_prompt()
    sc.decode_step(0)
    sc.append_steps(1, 11)
    sc.decode_step(11)
    sc.check_state()


def test_flags_bad_tag_capacity_and_pool_exhaustion():
    """Device anomalies set sticky flags and never write outside the pools."""
    say("case: flags")
    from paper_2608_28276_amd import pask
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob
    pol = uniform_policy(6, 1, 1, oracle.LOW)
    sess = PaskSession(pack_blob(pol), max_batch=2, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=64,
                       max_tokens_per_seq=64, hi_pages=1, lo_pages=2, extra_bytes=4096)
    dev = sess.device
    canary = sess.buf[sess.nbytes:]
    canary.fill_(0xA5)
    k = torch.randn((2, 64, 2, 64)).to(torch.bfloat16).to(dev)
    tags = torch.zeros((2, 64), dtype=torch.uint8, device=dev)
    tags[0, 3] = 200                                     # tag outside the table -> HIGH + flag
    sess.append(0, tags, k, k)                           # 2 x 64 LOW tokens, room for 32 -> exhaustion
    st, status, _ = sess.stats(batch=2)
    assert status == pask.PASK_E_DEVICE_FLAG
    assert st.device_flags & pask.PASK_FLAG_BAD_TAG
    assert st.device_flags & pask.PASK_FLAG_LO_POOL_EXHAUSTED
    assert st.n_low == 32 and st.n_lost == 128 - 32 - 1 and st.n_high == 1
    assert (canary == 0xA5).all()
    cnt = sess.counters()[:2, 0].cpu().numpy()
    assert (cnt[:, 1] % 16 == 0).all() and cnt[:, 1].sum() == 32
    # A further append beyond max_tokens_per_seq: capacity flag.
    sess.reset()
    sess.append(0, tags[:, :1].contiguous(), k[:, :1].contiguous(), k[:, :1].contiguous(), batch=1)
    big = torch.zeros((1, 64, 2, 64), dtype=torch.bfloat16, device=dev)
    sess.append(0, torch.zeros((1, 64), dtype=torch.uint8, device=dev), big, big, batch=1)
    st, status, _ = sess.stats(batch=1)
    assert st.device_flags & pask.PASK_FLAG_SEQ_CAPACITY
    assert int(sess.counters()[0, 0, 2]) == 64
    assert (canary == 0xA5).all()


def test_call_persisting_its_tokens_flags_and_page_order():
    """A decode call that persists each sequence's token itself (at most 64
    sequences, no window, no parser states): the pages one call opens are
    granted in sequence order, so the first opener takes the last page of a
    pool and the later ones are lost and flagged; a tag outside the table is
    kept HIGH (forced) and flagged; a sequence at its capacity loses the token.
    Counters, cursors and flags follow these rules exactly, the stored entries
    match the oracle bit for bit, and each sequence's attention matches the
    oracle over what was stored (zeros and -inf for a sequence with nothing)."""
    say("case: one call persisting its tokens: flags and page order")
    from paper_2608_28276_amd import pask
    from paper_2608_28276_amd.session import PaskSession
    from workload.policy import pack_blob
    from workload.tensors import bf16_normal
    from tests.gpu_util import bf16_f64, policy_dict
    pol = uniform_policy(6, 1, 1, oracle.LOW)
    P = [32, 5, 16, 0, 16]                               # HIGH pages 2 + 1 + 1 + 0 + 1 = the whole HIGH pool
    B, Hq, Hkv, D = len(P), 8, 2, 64
    sess = PaskSession(pack_blob(pol), max_batch=B, n_layers=1, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D,
                       max_tokens_per_seq=32, hi_pages=5, lo_pages=1)
    dev = sess.device
    oc = oracle.OracleCache(policy_dict(pol), Hkv, D)
    k = bf16_normal((B, 32, Hkv, D), 71)
    v = bf16_normal((B, 32, Hkv, D), 72)
    sess.append(0, None, k.to(dev), v.to(dev), n_new=torch.as_tensor(P, dtype=torch.int32, device=dev), keep_all=True)
    for b, p in enumerate(P):
        oc.append(0, b, np.zeros(p, np.uint8), bits16(k[b, :p]), bits16(v[b, :p]), keep_all=True)
    tags = np.array([0, 200, 0, 0, 200], np.uint8)
    kn, vn = bf16_normal((B, Hkv, D), 73), bf16_normal((B, Hkv, D), 74)
    q = bf16_normal((B, Hq, D), 75)
    out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    sess.decode(0, q.to(dev), out, lse, torch.as_tensor(tags, device=dev), kn.to(dev), vn.to(dev))
    torch.cuda.synchronize()
    cnt = sess.counters()[:B, 0].cpu().numpy()
    sw = sess.status_words().cpu().numpy().astype(np.uint32)
    #            hi  lo  pos drop forced lost      (the kept-all prompt tokens count as forced)
    want = [(32, 0, 32, 0, 32, 1),                       # at capacity: lost
            (6, 0, 6, 0, 6, 0),                          # tag 200: HIGH, forced, slot 5 of its page
            (16, 1, 17, 0, 16, 0),                       # LOW, opens the LOW pool's only page
            (0, 0, 1, 0, 0, 1),                          # LOW, opens a page: none left, lost
            (16, 0, 17, 0, 16, 1)]                       # tag 200: HIGH, opens a page: none left, lost
    for b in range(B):
        assert tuple(int(x) for x in cnt[b, :6]) == want[b], (b, cnt[b, :6], want[b])
    assert sw[2] == 5 + 1 and sw[3] == 0 + 2, sw         # one page per opener, granted or not
    assert sw[0] == (pask.PASK_FLAG_SEQ_CAPACITY | pask.PASK_FLAG_BAD_TAG | pask.PASK_FLAG_LO_POOL_EXHAUSTED |
                     pask.PASK_FLAG_HI_POOL_EXHAUSTED), hex(sw[0])
    for b in (1, 2):                                     # the stored tokens
        oc.append(0, b, tags[b:b + 1], bits16(kn[b:b + 1]), bits16(vn[b:b + 1]))
    il = sess.index_lists().cpu().numpy()
    assert il[1, 0, 0, 5] == 5 and il[2, 0, 1, 0] == 16
    for b in (1, 2):
        gk, gv = sess.gather_store(b, 0, 0)
        ok, ov = oc.hi_entries(b, 0)
        assert (gk == ok).all() and (gv == ov).all(), ("HIGH store", b)
    lo = oc.lo_entries(2, 0)
    glo = sess.gather_store(2, 0, 1)
    assert all(np.array_equal(x, y) for x, y in zip(glo, lo)), "LOW store of sequence 2"
    o = bf16_f64(out)
    l_gpu = lse.cpu().double().numpy()
    for b in range(B):
        o_ref, lse_ref = oc.attend(0, b, bits16(q[b]), sess.softmax_scale)
        if P[b] == 0:                                    # nothing stored: zeros, -inf
            assert (o[b] == 0).all() and np.isneginf(l_gpu[b]).all()
            continue
        assert_attn_close(o[b], o_ref, f"sequence {b}")


def test_stats_ckv_matches_oracle_counts():
    say("case: stats")
    pol = make_policy(6, 2, 4, 0.33, seed=16)
    tags = np.stack([function_call_tags(64, 60 + b) for b in range(3)])
    sc = Scenario(pol, B=3, L=4, Hq=8, Hkv=2, D=64, prompt_lens=[10, 20, 30], gen_tags=tags, seed=17)
    sc.fill_prompt()
    sc.append_steps(0, 64)
    st, status, per = sc.sess.stats(batch=3, per_seq=True)
    assert status == 0
    nh = nl = nd = nf = 0
    want = np.zeros((3, 2, 3), dtype=np.int64)
    for b in range(3):
        for layer in range(4):
            c = sc.oc.counts(b, layer)
            nh, nl, nd, nf = nh + c["hi"], nl + c["lo"], nd + c["drop"], nf + c["forced"]
            grp = int(pol.group_of_layer[layer])
            want[b, grp] += [c["drop"], c["lo"], c["hi"]]
    assert (per == want[:, :, None, :]).all()
    assert (st.n_high, st.n_low, st.n_drop, st.n_forced_high) == (nh, nl, nd, nf)
    assert st.c_kv_governed == pytest.approx(oracle.c_kv(nh - nf, nl, nd, 2, 64), rel=1e-12)
    assert (per[:, :, 0, :] == per[:, :, 1, :]).all()            # identical across KV heads
