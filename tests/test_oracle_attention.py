"""Pins of the oracle's attention over the persisted history and of C_KV
(Eq. 1; a Full-KV cache has C_KV = 1.00, Section 4.1)."""

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from tests import pins
from workload.policy import make_policy, uniform_policy
from workload.tags import iid_tags


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).numpy().astype(np.int64) & 0xFFFF


def _rand_bf16(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(shape, generator=g).to(torch.bfloat16)


SCALE64 = float(np.float32(1.0 / np.sqrt(64)))


def _policy_dict(pol):
    return dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=pol.n_sink)


def test_all_high_equals_full_attention_sdpa():
    hq, hkv, d, n = 8, 2, 64, 200
    pol = uniform_policy(6, 2, 2, oracle.HIGH)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k, v = _rand_bf16((n, hkv, d), 1), _rand_bf16((n, hkv, d), 2)
    q = _rand_bf16((hq, d), 3)
    cache.append(0, 0, iid_tags(n, 1), _bits(k), _bits(v))
    o, lse = cache.attend(0, 0, _bits(q), SCALE64)
    ref = pins.sdpa_gqa(q.double().numpy(), k.double().numpy(), v.double().numpy(), SCALE64)
    assert np.abs(o - ref).max() < 1e-13
    s = np.einsum("hd,nhd->hn", q.double().numpy(), np.repeat(k.double().numpy(), 4, axis=1)) * SCALE64
    assert np.abs(lse - scipy.special.logsumexp(s, axis=1)).max() < 1e-12


def test_all_drop_sees_only_prompt():
    hq, hkv, d, p, n = 8, 2, 64, 50, 120
    pol = uniform_policy(6, 2, 2, oracle.DROP)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k, v = _rand_bf16((p + n, hkv, d), 4), _rand_bf16((p + n, hkv, d), 5)
    q = _rand_bf16((hq, d), 6)
    cache.append(1, 0, np.zeros(p, np.uint8), _bits(k[:p]), _bits(v[:p]), keep_all=True)
    cache.append(1, 0, iid_tags(n, 2), _bits(k[p:]), _bits(v[p:]))
    hi, lo = cache.lists(0, 1)
    assert hi.tolist() == list(range(p)) and lo.size == 0
    o, _ = cache.attend(1, 0, _bits(q), SCALE64)
    ref = pins.sdpa_gqa(q.double().numpy(), k[:p].double().numpy(), v[:p].double().numpy(), SCALE64)
    assert np.abs(o - ref).max() < 1e-13


def test_all_low_equals_attention_over_dequantised():
    hq, hkv, d, n = 8, 2, 64, 90
    pol = uniform_policy(6, 2, 2, oracle.LOW)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k, v = _rand_bf16((n, hkv, d), 7), _rand_bf16((n, hkv, d), 8)
    q = _rand_bf16((hq, d), 9)
    cache.append(0, 0, iid_tags(n, 3), _bits(k), _bits(v))
    kc, ks = oracle.quantize_groups(_bits(k))
    vc, vs = oracle.quantize_groups(_bits(v))
    kh, vh = oracle.dequant(kc, ks), oracle.dequant(vc, vs)
    o, _ = cache.attend(0, 0, _bits(q), SCALE64)
    ref = pins.sdpa_gqa(q.double().numpy(), kh, vh, SCALE64)
    assert np.abs(o - ref).max() < 1e-13


def test_single_visible_token_gives_its_value():
    hq, hkv, d = 8, 2, 64
    pol = uniform_policy(6, 2, 2, oracle.DROP)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k, v = _rand_bf16((1, hkv, d), 10), _rand_bf16((1, hkv, d), 11)
    cache.append(0, 0, [0], _bits(k), _bits(v), keep_all=True)
    cache.append(0, 0, iid_tags(30, 5), np.zeros((30, hkv, d), np.int64), np.zeros((30, hkv, d), np.int64))
    o, _ = cache.attend(0, 0, _bits(_rand_bf16((hq, d), 12)), SCALE64)
    want = np.repeat(v.double().numpy()[0], hq // hkv, axis=0)
    assert (o == want).all()


def test_constant_keys_average_values_and_rows_sum_to_one():
    hq, hkv, d, n = 8, 2, 64, 77
    pol = uniform_policy(6, 2, 2, oracle.HIGH)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k = _rand_bf16((1, hkv, d), 13).expand(n, hkv, d)
    v = _rand_bf16((n, hkv, d), 14)
    cache.append(0, 0, iid_tags(n, 6), _bits(k), _bits(v))
    o, lse = cache.attend(0, 0, _bits(_rand_bf16((hq, d), 15)), SCALE64)
    mean = np.repeat(v.double().numpy().mean(axis=0), hq // hkv, axis=0)
    assert np.abs(o - mean).max() < 1e-13
    # Value vectors of all ones: every softmax row sums to one.
    cache2 = oracle.OracleCache(_policy_dict(pol), hkv, d)
    ones = torch.ones((n, hkv, d), dtype=torch.bfloat16)
    cache2.append(0, 0, iid_tags(n, 6), _bits(_rand_bf16((n, hkv, d), 16)), _bits(ones))
    o2, _ = cache2.attend(0, 0, _bits(_rand_bf16((hq, d), 17)), SCALE64)
    assert np.abs(o2 - 1.0).max() < 1e-12


def test_empty_history():
    o, lse = oracle.attention(np.ones((4, 8)), np.zeros((0, 1, 8)), np.zeros((0, 1, 8)), 0.5)
    assert (o == 0).all() and np.isneginf(lse).all()


def test_mixed_policy_matches_sdpa_on_persisted_set():
    hq, hkv, d, p, n = 8, 2, 64, 64, 128
    pol = make_policy(6, 2, 2, 0.33, seed=3)
    cache = oracle.OracleCache(_policy_dict(pol), hkv, d)
    k, v = _rand_bf16((p + n, hkv, d), 20), _rand_bf16((p + n, hkv, d), 21)
    q = _rand_bf16((hq, d), 22)
    tags = iid_tags(n, 7)
    cache.append(1, 0, np.zeros(p, np.uint8), _bits(k[:p]), _bits(v[:p]), keep_all=True)
    cache.append(1, 0, tags, _bits(k[p:]), _bits(v[p:]))
    eff = np.maximum(pol.action, pol.floor)[:, 1][tags]
    kk, vv = [], []
    for i in range(p + n):
        a = 2 if i < p else eff[i - p]
        if a == 2:
            kk.append(k[i].double().numpy()); vv.append(v[i].double().numpy())
        elif a == 1:
            kc, ks = oracle.quantize_groups(_bits(k[i]))
            vc, vs = oracle.quantize_groups(_bits(v[i]))
            kk.append(oracle.dequant(kc, ks)); vv.append(oracle.dequant(vc, vs))
    o, _ = cache.attend(1, 0, _bits(q), SCALE64)
    ref = pins.sdpa_gqa(q.double().numpy(), np.stack(kk), np.stack(vv), SCALE64)
    assert np.abs(o - ref).max() < 1e-13


def test_planted_gqa_mapping_mistake_is_caught():
    """Query head h reading KV head h % Hkv instead of h // G fails the SDPA pin."""
    hq, hkv, d, n = 8, 2, 64, 50
    k, v = _rand_bf16((n, hkv, d), 30), _rand_bf16((n, hkv, d), 31)
    q = _rand_bf16((hq, d), 32)
    kd, vd = k.double().numpy(), v.double().numpy()
    perm = [h % hkv for h in range(hq)]
    o, _ = _per_head(q.double().numpy(), kd[:, perm, :], vd[:, perm, :], SCALE64)
    ref = pins.sdpa_gqa(q.double().numpy(), kd, vd, SCALE64)
    assert np.abs(o - ref).max() > 1e-3
    good, _ = oracle.attention(q.double().numpy(), kd, vd, SCALE64)
    assert np.abs(good - ref).max() < 1e-13


def _per_head(q, k, v, scale):
    """Attention with one KV head per query head (k, v [n, Hq, D])."""
    hq = q.shape[0]
    o = np.zeros_like(q)
    for h in range(hq):
        s = k[:, h, :] @ q[h] * scale
        w = np.exp(s - s.max())
        o[h] = (w / w.sum()) @ v[:, h, :]
    return o, None


def test_ckv_closed_forms():
    assert oracle.c_kv(100, 0, 0, 8, 128) == 1.0            # Full KV (Section 4.1)
    assert oracle.c_kv(0, 100, 0, 8, 128) == 0.28125
    assert oracle.c_kv(0, 0, 100, 8, 128) == 0.0
    m = oracle.entry_bytes(8, 128)
    assert m[oracle.HIGH] == 4096 and m[oracle.LOW] == 1152 and m[oracle.DROP] == 0
    m0 = oracle.entry_bytes(2, 64)
    assert m0[oracle.HIGH] == 512 and m0[oracle.LOW] == 144
