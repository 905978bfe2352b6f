"""Pins of the oracle's protected recent window (Section 3.1): a release (and
any other action) takes effect only once the token leaves the last W
positions of its sequence; inside the window every token is attended at
full precision.  The references are torch SDPA (through `pins.sdpa_gqa`)
over explicitly chosen K/V sets, and the W = 0 cache on the prefix of the
stream that has left the window."""

import numpy as np
import pytest
import torch

import oracle
from tests import pins
from workload import make_policy
from workload.policy import uniform_policy, with_budget_controller
from workload.tags import iid_tags, function_call_tags_with_states, CRITICAL_STATES, PARSER_STATES


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).numpy().astype(np.int64) & 0xFFFF


def _rand_bf16(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(shape, generator=g).to(torch.bfloat16)


SCALE64 = float(np.float32(1.0 / np.sqrt(64)))
HQ, HKV, D = 8, 2, 64


def _pd(pol, window):
    d = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=pol.n_sink,
             rho_up=pol.rho_up, recent_window=window)
    if pol.n_states:
        d.update(n_states=pol.n_states, beta_q=pol.beta_q, reserve_q=pol.reserve_q, crit=pol.crit)
    return d


def _sdpa(q, k, v):
    return pins.sdpa_gqa(q.double().numpy(), np.asarray(k, np.float64), np.asarray(v, np.float64), SCALE64)


def test_window_covering_the_stream_is_full_kv():
    """All-DROP table, W larger than the stream: nothing has been persisted
    yet and attention equals full attention over every token at bf16."""
    n = 70
    cache = oracle.OracleCache(_pd(uniform_policy(6, 2, 2, oracle.DROP), 100), HKV, D)
    k, v, q = _rand_bf16((n, HKV, D), 1), _rand_bf16((n, HKV, D), 2), _rand_bf16((HQ, D), 3)
    cache.append(0, 0, iid_tags(n, 1), _bits(k), _bits(v))
    o, _ = cache.attend(0, 0, _bits(q), SCALE64)
    assert np.abs(o - _sdpa(q, k.double(), v.double())).max() < 1e-13
    c = cache.counts(0, 0)
    assert (c["hi"], c["lo"], c["drop"], c["window"], c["pos"]) == (0, 0, 0, n, n)


@pytest.mark.parametrize("W", [1, 5, 16, 37])
def test_all_drop_attends_exactly_the_last_w_tokens(W):
    """All-DROP table: after every append of a ragged sequence of appends,
    the visible set is the prompt (kept HIGH) and the last W generated
    positions; everything older is released."""
    p, n = 12, 90
    cache = oracle.OracleCache(_pd(uniform_policy(6, 2, 2, oracle.DROP), W), HKV, D)
    k, v = _rand_bf16((p + n, HKV, D), 4), _rand_bf16((p + n, HKV, D), 5)
    cache.append(0, 0, np.zeros(p, np.uint8), _bits(k[:p]), _bits(v[:p]), keep_all=True)
    t = p
    for i, m in enumerate([1, 3, 1, 20, 2, 40, 1, 22]):
        cache.append(0, 0, iid_tags(m, 10 + i), _bits(k[t:t + m]), _bits(v[t:t + m]))
        t += m
        q = _rand_bf16((HQ, D), 100 + i)
        keep = sorted(set(range(p)) | set(range(max(0, t - W), t)))
        o, _ = cache.attend(0, 0, _bits(q), SCALE64)
        assert np.abs(o - _sdpa(q, k[keep].double(), v[keep].double())).max() < 1e-13, (W, t)
        c = cache.counts(0, 0)
        assert c["window"] == min(W, t) and c["hi"] == min(p, max(0, t - W))
        assert c["hi"] + c["lo"] + c["drop"] + c["window"] == c["pos"] == t


def test_low_tokens_are_full_precision_until_they_leave():
    """All-LOW table with W = 7: the tokens older than the window are seen
    through their int4 codes, the last 7 at bf16."""
    n, W = 50, 7
    cache = oracle.OracleCache(_pd(uniform_policy(6, 2, 2, oracle.LOW), W), HKV, D)
    k, v, q = _rand_bf16((n, HKV, D), 6), _rand_bf16((n, HKV, D), 7), _rand_bf16((HQ, D), 8)
    cache.append(0, 0, iid_tags(n, 2), _bits(k), _bits(v))
    kc, ks = oracle.quantize_groups(_bits(k[:n - W]))
    vc, vs = oracle.quantize_groups(_bits(v[:n - W]))
    kk = np.concatenate([oracle.dequant(kc, ks), k[n - W:].double().numpy()])
    vv = np.concatenate([oracle.dequant(vc, vs), v[n - W:].double().numpy()])
    o, _ = cache.attend(0, 0, _bits(q), SCALE64)
    assert np.abs(o - _sdpa(q, kk, vv)).max() < 1e-13
    assert cache.lists(0, 0)[1].tolist() == list(range(n - W))


@pytest.mark.parametrize("W", [1, 4, 33])
def test_stores_equal_the_w0_stores_of_the_prefix_that_left(W):
    """Mixed table with sinks: after each append, the stores (lists,
    bf16 bits, codes, scales, counters) equal those of a W = 0 cache fed the
    same stream without its last W tokens; bulk and one-by-one appends agree."""
    pol = make_policy(6, 2, 4, 0.33, seed=3, n_sink=5)
    n = 160
    tags = iid_tags(n, 7)
    k, v = _rand_bf16((n, HKV, D), 9), _rand_bf16((n, HKV, D), 10)
    win = oracle.OracleCache(_pd(pol, W), HKV, D)
    one = oracle.OracleCache(_pd(pol, W), HKV, D)
    t = 0
    for m in [3, 1, 50, 7, 99]:
        win.append(2, 0, tags[t:t + m], _bits(k[t:t + m]), _bits(v[t:t + m]))
        for i in range(t, t + m):
            one.append(2, 0, tags[i:i + 1], _bits(k[i:i + 1]), _bits(v[i:i + 1]))
        t += m
        ref = oracle.OracleCache(_pd(pol, 0), HKV, D)
        left = max(0, t - W)
        ref.append(2, 0, tags[:left], _bits(k[:left]), _bits(v[:left]))
        for cache in (win, one):
            c, r = cache.counts(0, 2), ref.counts(0, 2)
            assert (c["hi"], c["lo"], c["drop"], c["forced"]) == (r["hi"], r["lo"], r["drop"], r["forced"])
            assert c["pos"] == t and c["window"] == min(W, t)
            for a, b in zip(cache.lists(0, 2), ref.lists(0, 2)):
                assert (a == b).all()
            for a, b in zip(cache.hi_entries(0, 2) + cache.lo_entries(0, 2),
                            ref.hi_entries(0, 2) + ref.lo_entries(0, 2)):
                assert a.shape == b.shape and (a == b).all()


def test_controller_charges_at_decision_time():
    """The controller decides and charges R when a token is accepted (Alg. 2);
    the window only delays the Persist step: R after every append is the
    same for W = 0 and W = 9, and so are the eventual stores."""
    T = 120
    tags, states = function_call_tags_with_states(T, 5)
    pol = make_policy(6, 2, 4, 0.33, seed=8, n_sink=2)
    pol = with_budget_controller(pol, [function_call_tags_with_states(T, 50 + i) for i in range(3)],
                                 len(PARSER_STATES), CRITICAL_STATES)
    k, v = _rand_bf16((T, HKV, D), 11), _rand_bf16((T, HKV, D), 12)
    caches = {W: oracle.OracleCache(_pd(pol, W), HKV, D) for W in (0, 9)}
    for c in caches.values():
        c.budget_init(0, [1], T // 2)
    for t in range(0, T, 10):
        for c in caches.values():
            c.append(1, 0, tags[t:t + 10], _bits(k[t:t + 10]), _bits(v[t:t + 10]), states=states[t:t + 10])
        assert caches[0].counts(0, 1)["R"] == caches[9].counts(0, 1)["R"]
    pad_tags = np.zeros(9, np.uint8)
    caches[9].append(1, 0, pad_tags, np.zeros((9, HKV, D), np.int64), np.zeros((9, HKV, D), np.int64),
                     keep_all=True)                     # push the last 9 generated tokens out
    for a, b in zip(caches[0].lists(0, 1), caches[9].lists(0, 1)):
        assert (a == b[b < T]).all()


class _QuantisedWindow(oracle.OracleCache):
    """Planted mistake: tokens inside the window are seen at their action's
    precision (LOW quantised, DROP hidden) instead of at full precision."""

    def visible_kv(self, seq, layer):
        st = self.sl(seq, layer)
        keep_pos, keep_k, keep_v = st.w_pos, st.w_k, st.w_v
        sel = st.w_act != oracle.DROP
        st.w_pos, st.w_k, st.w_v = st.w_pos[sel], st.w_k[sel].copy(), st.w_v[sel].copy()
        low = st.w_act[sel] == oracle.LOW
        if low.any():
            for arr in (st.w_k, st.w_v):
                c, s = oracle.quantize_groups(arr[low])
                arr[low] = oracle.dequant(c, s).astype(np.float32).view(np.uint32) >> 16
        try:
            return super().visible_kv(seq, layer)
        finally:
            st.w_pos, st.w_k, st.w_v = keep_pos, keep_k, keep_v


def test_planted_window_mistake_is_caught(monkeypatch):
    monkeypatch.setattr(oracle, "OracleCache", _QuantisedWindow)
    with pytest.raises(AssertionError):
        test_window_covering_the_stream_is_full_kv()
    with pytest.raises(AssertionError):
        test_low_tokens_are_full_precision_until_they_leave()
