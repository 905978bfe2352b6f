"""Pins of the oracle's attention-output distortion D(q, a) (Eq. 4, Section 3.3).

References that do not reuse the oracle's arithmetic:
  * a = HIGH: the intervened run equals the reference, so D = 0 exactly;
  * two positions (one prompt token, one generated token of the bucket),
    DROP: o_full = (1 - p) v0 + p v1 with p the logistic of the score
    difference and o_a = v0, so D = max_h p_h^2 ||v1 - v0||^2 (closed form);
  * brute force: torch scaled-dot-product attention in fp64 over explicit key
    sets (DROP removes the bucket's positions, LOW replaces their K / V by an
    int4 round trip written with torch / numpy library rounding), the steps
    of S(q) and the layers of the group enumerated directly;
  * a bucket that never occurs: S(q) is empty, D = 0.
Planted mistakes in a copy of the outer loop (sum instead of max over heads,
no square, S(q) taken over every step, S(q) starting after the first
occurrence, the intervention applied in every group) each fail one of them.
"""

import math

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _bf16(shape, rng, scale=1.0):
    x = torch.from_numpy(rng.standard_normal(shape) * scale).to(torch.bfloat16)
    return x.view(torch.int16).numpy().view(np.uint16)


def _f64(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).double()


def _int4_round_trip(x):
    """Symmetric int4, one fp16 scale per 32 contiguous elements, with library
    rounding: fp16 cast of absmax / 7 (round to nearest even), codes
    rint(x / s) clamped to [-7, 7], 0 when s = 0."""
    shp = x.shape
    g = x.reshape(shp[:-1] + (shp[-1] // 32, 32))
    s = (g.abs().amax(-1, keepdim=True) / 7.0).to(torch.float16).double()
    q = torch.where(s > 0, torch.clamp(torch.round(g / torch.where(s > 0, s, 1.0)), -7, 7), 0.0)
    return (q * s).reshape(shp)


def _sdpa(q, k, v, scale):
    """q [Hq, D], k / v [n, Hkv, D] fp64 -> o [Hq, D] (GQA by repeat_interleave)."""
    hq, hkv = q.shape[0], k.shape[1]
    kk = k.permute(1, 0, 2).repeat_interleave(hq // hkv, dim=0)
    vv = v.permute(1, 0, 2).repeat_interleave(hq // hkv, dim=0)
    return torch.nn.functional.scaled_dot_product_attention(q[:, None, :], kk, vv, scale=scale)[:, 0, :]


def _brute_force(tags, kb, vb, qb, P, gol, tag, group, action, scale):
    R, T = tags.shape
    layers = [l for l in range(len(gol)) if gol[l] == group]
    tot, n_s = 0.0, 0
    for r in range(R):
        first = np.flatnonzero(tags[r] == tag)
        if first.size == 0:
            continue
        for u in range(int(first[0]), T):
            n_s += 1
            n = P + u + 1
            is_z = np.zeros(n, bool)
            is_z[P:] = tags[r, :u + 1] == tag
            for l in layers:
                k, v, q = _f64(kb[r, l, :n]), _f64(vb[r, l, :n]), _f64(qb[r, l, u])
                o_full = _sdpa(q, k, v, scale)
                if action == oracle.DROP:
                    keep = torch.from_numpy(~is_z)
                    o_a = _sdpa(q, k[keep], v[keep], scale)
                elif action == oracle.LOW:
                    zz = torch.from_numpy(is_z)
                    k2, v2 = k.clone(), v.clone()
                    k2[zz], v2[zz] = _int4_round_trip(k[zz]), _int4_round_trip(v[zz])
                    o_a = _sdpa(q, k2, v2, scale)
                else:
                    o_a = o_full
                tot += float(((o_full - o_a) ** 2).sum(-1).max())
    return (tot / n_s if n_s else 0.0), n_s


def _inputs(seed, R=2, L=2, T=6, P=3, Hq=4, Hkv=2, D=64, n_tags=3):
    rng = np.random.default_rng(seed)
    tags = rng.integers(0, n_tags, size=(R, T)).astype(np.uint8)
    kb = _bf16((R, L, P + T, Hkv, D), rng)
    vb = _bf16((R, L, P + T, Hkv, D), rng)
    qb = _bf16((R, L, T, Hq, D), rng)
    return tags, kb, vb, qb


SCALE = float(np.float32(1 / math.sqrt(64)))


def test_high_intervention_is_exactly_zero():
    tags, kb, vb, qb = _inputs(1)
    gol = np.array([0, 1])
    for tag in range(3):
        d, n_s = oracle.distortion(tags, kb, vb, qb, 3, gol, 3, tag, 1, oracle.HIGH, SCALE)
        assert d == 0.0
        assert n_s > 0


def _two_token(seed, Hq=4, Hkv=2, D=64):
    rng = np.random.default_rng(seed)
    tags = np.array([[1]], np.uint8)
    kb = _bf16((1, 1, 2, Hkv, D), rng)
    vb = _bf16((1, 1, 2, Hkv, D), rng, scale=2.0)
    qb = _bf16((1, 1, 1, Hq, D), rng, scale=3.0)     # spread the per-head weights
    k, v, q = _f64(kb[0, 0]).numpy(), _f64(vb[0, 0]).numpy(), _f64(qb[0, 0, 0]).numpy()
    want = 0.0
    for h in range(Hq):
        g = h // (Hq // Hkv)
        s0, s1 = SCALE * float(q[h] @ k[0, g]), SCALE * float(q[h] @ k[1, g])
        p1 = 1.0 / (1.0 + math.exp(s0 - s1))
        want = max(want, p1 * p1 * float(((v[1, g] - v[0, g]) ** 2).sum()))
    return tags, kb, vb, qb, want


@pytest.mark.parametrize("seed", [3, 4, 5])
def test_two_positions_drop_closed_form(seed):
    tags, kb, vb, qb, want = _two_token(seed)
    d, n_s = oracle.distortion(tags, kb, vb, qb, 1, np.array([0]), 2, 1, 0, oracle.DROP, SCALE)
    assert n_s == 1
    assert d == pytest.approx(want, rel=1e-12, abs=0)


@pytest.mark.parametrize("action", [oracle.DROP, oracle.LOW])
@pytest.mark.parametrize("seed", [11, 12, 13])
def test_brute_force_masked_attention(action, seed):
    tags, kb, vb, qb = _inputs(seed)
    tags[0, :2] = 0                    # trajectory 0: the bucket first occurs at step 2
    tags[0, 2] = 2
    gol = np.array([0, 1])
    for group in (0, 1):
        d, n_s = oracle.distortion(tags, kb, vb, qb, 3, gol, 3, 2, group, action, SCALE)
        want, want_n = _brute_force(tags, kb, vb, qb, 3, gol, 2, group, action, SCALE)
        assert n_s == want_n
        assert d == pytest.approx(want, rel=1e-10, abs=1e-14)
        assert d > 0


def test_absent_bucket_has_no_positions():
    tags, kb, vb, qb = _inputs(21)
    tags[:] = 0
    d, n_s = oracle.distortion(tags, kb, vb, qb, 3, np.array([0, 1]), 3, 2, 0, oracle.DROP, SCALE)
    assert (d, n_s) == (0.0, 0)


# -- planted mistakes --------------------------------------------------------

def _planted(mistake, tags, kb, vb, qb, P, gol, n_tags, tag, group, action, scale):
    """The oracle's outer loop with one mistake planted."""
    R, T = tags.shape
    hkv, d = kb.shape[-2], kb.shape[-1]
    n_groups = int(gol.max()) + 1
    layers = [l for l in range(len(gol)) if gol[l] == group or mistake == "all_groups"]
    full_a = np.full((n_tags, n_groups), oracle.HIGH, np.uint8)
    int_a, _ = oracle.intervention_table(n_tags, n_groups, tag, group, action)
    if mistake == "all_groups":
        int_a[tag, :] = action
    pol = lambda a: dict(action=a, floor=np.zeros_like(a), group_of_layer=gol, n_sink=0)
    tot, n_s = 0.0, 0
    for r in range(R):
        ref, itv = oracle.OracleCache(pol(full_a), hkv, d), oracle.OracleCache(pol(int_a), hkv, d)
        for l in layers:
            for c in (ref, itv):
                c.append(l, 0, np.zeros(P, np.uint8), kb[r, l, :P], vb[r, l, :P], keep_all=True)
        seen = False
        for u in range(T):
            hit = int(tags[r, u]) == tag
            for l in layers:
                for c in (ref, itv):
                    c.append(l, 0, tags[r, u:u + 1], kb[r, l, P + u][None], vb[r, l, P + u][None])
            in_s = {"every_step": True, "after_first": seen}.get(mistake, seen or hit)
            seen |= hit
            if not in_s:
                continue
            n_s += 1
            for l in layers:
                o_f, _ = ref.attend(l, 0, qb[r, l, u], scale)
                o_a, _ = itv.attend(l, 0, qb[r, l, u], scale)
                dd = ((o_f - o_a) ** 2).sum(-1)
                if mistake == "sum_heads":
                    tot += float(dd.sum())
                elif mistake == "no_square":
                    tot += float(np.sqrt(dd).max())
                else:
                    tot += float(dd.max())
    return (tot / n_s if n_s else 0.0), n_s


def test_planted_copy_without_mistake_agrees():
    tags, kb, vb, qb = _inputs(31)
    gol = np.array([0, 1])
    got = _planted(None, tags, kb, vb, qb, 3, gol, 3, 1, 1, oracle.DROP, SCALE)
    want = oracle.distortion(tags, kb, vb, qb, 3, gol, 3, 1, 1, oracle.DROP, SCALE)
    assert got[1] == want[1] and got[0] == pytest.approx(want[0], rel=1e-12)


@pytest.mark.parametrize("mistake", ["sum_heads", "no_square", "after_first"])
def test_planted_mistakes_fail_the_closed_form(mistake):
    tags, kb, vb, qb, want = _two_token(3)
    d, _ = _planted(mistake, tags, kb, vb, qb, 1, np.array([0]), 2, 1, 0, oracle.DROP, SCALE)
    assert d != pytest.approx(want, rel=1e-6)


@pytest.mark.parametrize("mistake", ["every_step", "all_groups"])
def test_planted_mistakes_fail_the_brute_force(mistake):
    tags, kb, vb, qb = _inputs(11)
    tags[0, :2] = 0
    tags[0, 2] = 2
    gol = np.array([0, 1])
    want, _ = _brute_force(tags, kb, vb, qb, 3, gol, 2, 1, oracle.DROP, SCALE)
    d, _ = _planted(mistake, tags, kb, vb, qb, 3, gol, 3, 2, 1, oracle.DROP, SCALE)
    assert d != pytest.approx(want, rel=1e-6)
