"""CPU oracle for the PASK decode hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never imports it.

What it computes, each piece following the passage named in its docstring:
  * the per-token, per-layer-group action: a = max(a0[z][c], a-[z][c]) under
    the order DROP < RETAIN-LOW < RETAIN-HIGH (Section 3.1; Eq. 10, the max step
    of the online lookup, Alg. 2);
  * persistence of each entry (the Persist step of Alg. 2): DROP entries are
    released from future attention (Section 3.1), LOW / HIGH entries are kept
    in two compacted stores in position order;
  * RETAIN-LOW storage: symmetric int4 with one fp16 scale per 32 elements.  The
    paper names no low-bit format; this is the format chosen for the build,
    computed here in exact integer arithmetic on bf16 bit patterns;
  * decode attention over the persisted history, by the textbook definition
    softmax(q k^T * scale) v, in fp64;
  * the normalised KV cost C_KV of Eq. 1;
  * the online budget controller of Alg. 2 (Eq. 9-10): the remaining budget
    R_t, B_t = max(0, R_t - Gamma(s_t)), demotions above the floors in
    ascending upgrade score, promotions in critical states in descending
    score, R_{t+1} = R_t - sum_c m(a_c, c), all in integer bytes;
  * the protected recent window of Section 3.1: the last W positions of a
    sequence stay visible at full precision whatever their action, which
    takes effect when a token leaves the window (release then removes it from
    the attention that follows);
  * the attention-output distortion D(q, a) of Eq. 4 (Section 3.3): one
    bucket q = (z, c) intervened with action a while every other bucket stays
    HIGH, the squared L2 distance of the attention outputs maximised over
    query heads, averaged over the decode positions the bucket affects and
    summed over the layers of group c.

Everything is plain numpy.  The attention is the definition written out
(exact, up to fp64 rounding order); the decisions, compaction and codes are
exact integer results.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

DROP, LOW, HIGH = 0, 1, 2        # R < L < H (Section 3.1)
QGROUP = 32                      # elements per fp16 scale of a RETAIN-LOW entry
QMAX = 7                         # symmetric int4 code range [-7, 7]
FP16_MAX_BITS = 0x7BFF           # 65504


# --------------------------------------------------------------------------
# Decisions (Eq. 10; Alg. 2, lookup and max steps)
# --------------------------------------------------------------------------

def decide(tags, positions, group: int, action, floor, n_sink: int, keep_all: bool):
    """Actions for a run of tokens of one sequence in layer group `group`.

    The table gives the selected action a0 = action[z][c] and the floor
    a- = floor[z][c]; the online action is their maximum under R < L < H.
    Overrides: the first n_sink positions of a sequence and tokens appended
    in keep-all mode (prompt tokens not governed by the table) are HIGH; a tag
    outside the table is HIGH and reported (fail-safe).

    Returns (actions uint8 [n], forced bool [n], bad_tag bool [n])."""
    tags = np.asarray(tags, dtype=np.int64)
    positions = np.asarray(positions, dtype=np.int64)
    action = np.asarray(action)
    floor = np.asarray(floor)
    n_tags = action.shape[0]
    out = np.empty(tags.shape, dtype=np.uint8)
    forced = np.zeros(tags.shape, dtype=bool)
    bad = tags >= n_tags
    for i in range(tags.size):
        z = int(tags[i])
        if keep_all or positions[i] < n_sink or z >= n_tags:
            out[i] = HIGH
            forced[i] = True
        else:
            out[i] = max(int(action[z, group]), int(floor[z, group]))
    return out, forced, bad


def compact(actions, positions):
    """The two persisted stores of one (sequence, layer): the positions whose
    action is HIGH and those whose action is LOW, each in increasing position
    order.  A DROP position appears in neither (release, Section 3.1).  The
    slot of an entry is its rank in its store."""
    actions = np.asarray(actions)
    positions = np.asarray(positions, dtype=np.int64)
    order = np.argsort(positions, kind="stable")
    a, p = actions[order], positions[order]
    return p[a == HIGH].copy(), p[a == LOW].copy()


# --------------------------------------------------------------------------
# RETAIN-LOW format: int4, symmetric absmax / 7, fp16 scale per 32 elements.
# Exact integer arithmetic on bit patterns.
# --------------------------------------------------------------------------

def bf16_mag(bits):
    """Split bf16 bit patterns into sign and an exact magnitude M * 2**E.
    Normal: M = 128 + mantissa, E = exponent - 134.  Subnormal: M = mantissa,
    E = -133.  Inputs must be finite."""
    bits = np.asarray(bits, dtype=np.int64) & 0xFFFF
    sign = bits >> 15
    ex = (bits >> 7) & 0xFF
    man = bits & 0x7F
    if np.any(ex == 0xFF):
        raise ValueError("non-finite bf16 input")
    m = np.where(ex == 0, man, man | 0x80)
    e = np.where(ex == 0, -133, ex - 134)
    return sign, m, e


def _rne_div(num, den):
    """Round-half-to-even of num/den for non-negative int64 arrays, den > 0."""
    q, r = np.divmod(num, den)
    up = (2 * r > den) | ((2 * r == den) & ((q & 1) == 1))
    return q + up.astype(np.int64)


def _floor_log2_ratio(m, e, d: int):
    """floor(log2(m * 2**e / d)) for integer m >= 1 and small odd d, exactly."""
    m = np.asarray(m, dtype=np.int64)
    f = np.zeros(m.shape, dtype=np.int64)
    # Largest f with d * 2**f <= m, searched over the small range m allows.
    for cand in range(-4, 9):
        ok = (m >= d * (1 << cand)) if cand >= 0 else (m * (1 << -cand) >= d)
        f = np.where(ok, cand, f)
    return f + e


def fp16_scale_bits(absmax_bits):
    """fp16 bit pattern of the group scale s = RNE_fp16(absmax / 7), saturated
    at 65504.  absmax_bits are non-negative finite bf16 patterns."""
    _, m, e = bf16_mag(absmax_bits)
    m = np.asarray(m, dtype=np.int64)
    e = np.asarray(e, dtype=np.int64)
    zero = m == 0
    m1 = np.where(zero, 1, m)
    # Exponent k such that the significand S = a/7 / 2**k lies in [1024, 2048);
    # fp16 normal numbers are S * 2**k with k in [-24, 5]; below, k = -24 and
    # S < 1024 (subnormals).
    k = _floor_log2_ratio(m1, e, QMAX) - 10
    k = np.maximum(k, -24)
    sh = e - k                                 # S = m * 2**sh / 7
    sh_c = np.clip(sh, -62, 40)
    num = np.where(sh_c >= 0, m1 << np.maximum(sh_c, 0), m1)
    den = np.where(sh_c >= 0, QMAX, QMAX << np.maximum(-sh_c, 0))
    tiny = sh < -40                            # quotient far below 1/2
    s = np.where(tiny, 0, _rne_div(np.where(tiny, 0, num), np.where(tiny, 1, den)))
    carry = s == 2048                          # rounding reached the next binade
    s = np.where(carry, 1024, s)
    k = np.where(carry, k + 1, k)
    over = k > 5                               # beyond 65504: saturate
    bits = np.where(s >= 1024, ((k + 25) << 10) | (s - 1024), s)
    bits = np.where(over, FP16_MAX_BITS, bits)
    bits = np.where(zero, 0, bits)
    return bits.astype(np.uint16)


def fp16_mag(bits):
    """fp16 pattern -> (S, k) with value S * 2**k (finite, non-negative)."""
    bits = np.asarray(bits, dtype=np.int64)
    ex = (bits >> 10) & 0x1F
    man = bits & 0x3FF
    s = np.where(ex == 0, man, man | 0x400)
    k = np.where(ex == 0, -24, ex - 25)
    return s, k


def quantize_groups(x_bits):
    """Quantise bf16 vectors group-wise along the last axis (length a multiple
    of 32).  Returns (codes int8 [..., n], scale_bits uint16 [..., n/32]).

    Per group: absmax a = max |x_i|; s = RNE_fp16(a / 7) saturated at 65504;
    q_i = clamp(RNE(x_i / s), -7, 7), and q = 0 for the whole group when s = 0.
    RNE of the quotient is symmetric, so q_i = sign(x_i) * RNE(|x_i| / s)."""
    x = np.asarray(x_bits, dtype=np.int64) & 0xFFFF
    shape = x.shape
    n = shape[-1]
    assert n % QGROUP == 0
    g = x.reshape(-1, n // QGROUP, QGROUP)
    absmax = (g & 0x7FFF).max(axis=-1)          # order of finite magnitudes = order of bits
    sbits = fp16_scale_bits(absmax)
    S, k = fp16_mag(sbits)
    sign, m, e = bf16_mag(g)
    S_ = S[..., None]
    sh = e - k[..., None]                       # |x| / s = m * 2**sh / S
    big = sh > 15                               # quotient >= 2**15 / 2047 > 7.5
    tiny = sh < -40                             # quotient < 2**-29
    sh_c = np.clip(sh, -40, 15)
    num = np.where(sh_c >= 0, m << np.maximum(sh_c, 0), m)
    den = np.where(sh_c >= 0, S_, S_ << np.maximum(-sh_c, 0))
    safe_den = np.where(den == 0, 1, den)
    q = _rne_div(num, safe_den)
    q = np.where(big, QMAX, np.where(tiny, 0, q))
    q = np.minimum(q, QMAX)
    q = np.where(S_ == 0, 0, q)
    q = np.where(sign == 1, -q, q)
    return q.reshape(shape).astype(np.int8), sbits.reshape(shape[:-1] + (n // QGROUP,))


def pack_nibbles(codes):
    """Two's-complement nibbles, element 2j in the low nibble of byte j."""
    c = np.asarray(codes, dtype=np.int64) & 0xF
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def unpack_nibbles(packed):
    p = np.asarray(packed, dtype=np.int64)
    lo, hi = p & 0xF, (p >> 4) & 0xF
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int64)
    out[..., 0::2], out[..., 1::2] = lo, hi
    return np.where(out >= 8, out - 16, out).astype(np.int8)


def fp16_to_f64(bits):
    s, k = fp16_mag(np.asarray(bits, dtype=np.int64) & 0x7FFF)
    v = s.astype(np.float64) * np.exp2(k.astype(np.float64))
    return np.where((np.asarray(bits, dtype=np.int64) >> 15) == 1, -v, v)


def bf16_to_f64(bits):
    sign, m, e = bf16_mag(bits)
    v = m.astype(np.float64) * np.exp2(e.astype(np.float64))
    return np.where(sign == 1, -v, v)


def dequant(codes, scale_bits):
    """x_hat = q * s (exact in fp64)."""
    c = np.asarray(codes, dtype=np.float64)
    s = fp16_to_f64(scale_bits)
    n = c.shape[-1]
    return (c.reshape(c.shape[:-1] + (n // QGROUP, QGROUP)) * s[..., None]).reshape(c.shape)


# --------------------------------------------------------------------------
# Attention over the persisted history (textbook definition, fp64)
# --------------------------------------------------------------------------

def attention(q, k, v, scale: float):
    """o_h = sum_j softmax_j(scale * q_h . k_j) v_j for every query head h,
    with grouped-query sharing: query head h reads KV head h // G.

    q [Hq, D], k and v [n, Hkv, D] (fp64).  Returns (o [Hq, D], lse [Hq]) with
    lse = m + ln(sum_j exp(s_j - m)).  An empty history gives o = 0, lse = -inf."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    hq, d = q.shape
    n, hkv, _ = k.shape
    g = hq // hkv
    o = np.zeros((hq, d))
    lse = np.full(hq, -np.inf)
    if n == 0:
        return o, lse
    for h in range(hq):
        kv = h // g
        s = (k[:, kv, :] @ q[h]) * scale
        m = s.max()
        w = np.exp(s - m)
        tot = w.sum()
        o[h] = (w / tot) @ v[:, kv, :]
        lse[h] = m + math.log(tot)
    return o, lse


# --------------------------------------------------------------------------
# Persisted-history model of one cache (Alg. 2 Persist step, replayed)
# --------------------------------------------------------------------------

@dataclass
class _SeqLayer:
    n_pos: int = 0
    hi_pos: list = field(default_factory=list)
    lo_pos: list = field(default_factory=list)
    hi_k: list = field(default_factory=list)     # bf16 bits [n, Hkv, D] per append
    hi_v: list = field(default_factory=list)
    lo_kc: list = field(default_factory=list)    # int8 codes [n, Hkv, D] per append
    lo_ks: list = field(default_factory=list)    # fp16 scale bits [n, Hkv, D/32] per append
    lo_vc: list = field(default_factory=list)
    lo_vs: list = field(default_factory=list)
    n_forced: int = 0
    n_drop: int = 0
    R: int = 0                                    # remaining budget (bytes) of the online controller
    # tokens inside the protected recent window, in position order: decided,
    # not yet persisted (positions, actions, forced flags, bf16 bits of K, V)
    w_pos: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    w_act: np.ndarray = field(default_factory=lambda: np.zeros(0, np.uint8))
    w_forced: np.ndarray = field(default_factory=lambda: np.zeros(0, bool))
    w_k: np.ndarray = None
    w_v: np.ndarray = None


class OracleCache:
    """The persisted history of a set of sequences, replayed append by append.

    policy: dict with action [T][C], floor [T][C], group_of_layer [L], n_sink,
    and optionally recent_window W (Section 3.1), rho_up and the controller's
    n_states, beta_q, reserve_q, crit."""

    def __init__(self, policy: dict, n_kv_heads: int, head_dim: int):
        self.action = np.asarray(policy["action"])
        self.floor = np.asarray(policy["floor"])
        self.group_of_layer = np.asarray(policy["group_of_layer"])
        self.n_sink = int(policy.get("n_sink", 0))
        self.window = int(policy.get("recent_window", 0))
        self.hkv = n_kv_heads
        self.d = head_dim
        self.state: dict = {}
        self.bad_tag = False
        self.bad_state = False
        # online controller (Alg. 2), when the table carries it
        self.rho_up = np.asarray(policy.get("rho_up", np.zeros(self.action.shape + (2,), np.float32)),
                                 dtype=np.float32)
        n_groups = self.action.shape[1]
        self.m = group_costs(self.group_of_layer, n_groups, n_kv_heads, head_dim)
        self.n_states = int(policy.get("n_states", 0))
        self.beta_q = int(policy.get("beta_q", 0))
        self.crit = np.asarray(policy.get("crit", np.zeros(0, np.uint8)))
        self.gamma = reserve_bytes(policy.get("reserve_q", np.zeros(0, np.uint32)), self.m)

    def budget_init(self, seq: int, layers, t_max: int):
        """R_0 for one sequence in the given layers (each layer keeps its copy)."""
        for layer in layers:
            self.sl(seq, layer).R = initial_budget(self.beta_q, t_max, self.m)

    def sl(self, seq: int, layer: int) -> _SeqLayer:
        return self.state.setdefault((seq, layer), _SeqLayer())

    def append(self, layer: int, seq: int, tags, k_bits, v_bits, keep_all: bool = False, states=None):
        """Persist n new tokens of one sequence in one layer.
        k_bits, v_bits: bf16 bit patterns [n, Hkv, D].  states: parser states
        [n] (the online controller decides, token after token) or None (the
        static lookup of Eq. 10).  Keep-all appends bypass the controller."""
        st = self.sl(seq, layer)
        tags = np.asarray(tags).reshape(-1)
        n = tags.size
        k_bits = (np.asarray(k_bits).astype(np.int64) & 0xFFFF).astype(np.uint16).reshape(n, self.hkv, self.d)
        v_bits = (np.asarray(v_bits).astype(np.int64) & 0xFFFF).astype(np.uint16).reshape(n, self.hkv, self.d)
        pos = st.n_pos + np.arange(n)
        c = int(self.group_of_layer[layer])
        acts, forced, bad = decide(tags, pos, c, self.action, self.floor, self.n_sink, keep_all)
        if states is not None and not keep_all:
            states = np.asarray(states).reshape(-1)
            for i in range(n):
                s = int(states[i])
                known = s < self.n_states
                self.bad_state |= not known
                a, cost = online_actions(int(tags[i]), s, st.R, self.action, self.floor, self.rho_up, self.m,
                                         self.gamma[s] if known else 0, bool(self.crit[s]) if known else False,
                                         bool(forced[i]))
                acts[i] = a[c]
                st.R -= cost
        self.bad_tag |= bool(bad.any())
        if self.window == 0:
            self._persist(st, pos, acts, forced, k_bits, v_bits)
        else:
            # Section 3.1: the decision is taken now; it takes effect when the
            # token leaves the last W positions of the sequence.
            if st.w_k is None:
                st.w_k = np.zeros((0, self.hkv, self.d), np.uint16)
                st.w_v = np.zeros((0, self.hkv, self.d), np.uint16)
            wp = np.concatenate([st.w_pos, pos])
            wa = np.concatenate([st.w_act, acts])
            wf = np.concatenate([st.w_forced, forced])
            wk = np.concatenate([st.w_k, k_bits])
            wv = np.concatenate([st.w_v, v_bits])
            out = wp < st.n_pos + n - self.window
            self._persist(st, wp[out], wa[out], wf[out], wk[out], wv[out])
            st.w_pos, st.w_act, st.w_forced, st.w_k, st.w_v = wp[~out], wa[~out], wf[~out], wk[~out], wv[~out]
        st.n_pos += n
        return acts

    def _persist(self, st: _SeqLayer, pos, acts, forced, k_bits, v_bits):
        """The Persist step of Alg. 2 for entries in position order: HIGH keeps
        the bf16 bits, LOW the int4 codes and fp16 scales, DROP nothing."""
        st.n_forced += int(np.asarray(forced).sum())
        hi = acts == HIGH
        lo = acts == LOW
        st.hi_pos.extend(pos[hi].tolist())
        st.hi_k.append(k_bits[hi])
        st.hi_v.append(v_bits[hi])
        if lo.any():
            kc, ks = quantize_groups(k_bits[lo])
            vc, vs = quantize_groups(v_bits[lo])
            st.lo_pos.extend(pos[lo].tolist())
            st.lo_kc.append(kc)
            st.lo_ks.append(ks)
            st.lo_vc.append(vc)
            st.lo_vs.append(vs)
        st.n_drop += int((acts == DROP).sum())

    def lists(self, seq: int, layer: int):
        st = self.sl(seq, layer)
        return np.asarray(st.hi_pos, dtype=np.int64), np.asarray(st.lo_pos, dtype=np.int64)

    def lo_entries(self, seq: int, layer: int):
        """(k codes, k scale bits, v codes, v scale bits) of the LOW store, by slot."""
        st = self.sl(seq, layer)
        shp_c = (0, self.hkv, self.d)
        shp_s = (0, self.hkv, self.d // QGROUP)
        f = lambda xs, shp, dt: (np.concatenate(xs).astype(dt) if xs else np.zeros(shp, dt))
        return (f(st.lo_kc, shp_c, np.int8), f(st.lo_ks, shp_s, np.uint16),
                f(st.lo_vc, shp_c, np.int8), f(st.lo_vs, shp_s, np.uint16))

    def hi_entries(self, seq: int, layer: int):
        """(k bits, v bits) of the HIGH store, by slot (uint16 bf16 patterns)."""
        st = self.sl(seq, layer)
        shp = (0, self.hkv, self.d)
        f = lambda xs: np.concatenate(xs) if xs else np.zeros(shp, np.uint16)
        return f(st.hi_k), f(st.hi_v)

    def visible_kv(self, seq: int, layer: int):
        """K and V of every visible entry in position order, in fp64: the
        persisted stores and the tokens still inside the recent window."""
        hk, hv = self.hi_entries(seq, layer)
        kc, ks, vc, vs = self.lo_entries(seq, layer)
        hi_pos, lo_pos = self.lists(seq, layer)
        pos = np.concatenate([hi_pos, lo_pos])
        k = np.concatenate([bf16_to_f64(hk), dequant(kc, ks)])
        v = np.concatenate([bf16_to_f64(hv), dequant(vc, vs)])
        st = self.sl(seq, layer)
        if st.w_pos.size:
            pos = np.concatenate([pos, st.w_pos])
            k = np.concatenate([k, bf16_to_f64(st.w_k)])
            v = np.concatenate([v, bf16_to_f64(st.w_v)])
        order = np.argsort(pos, kind="stable")
        return k[order], v[order]

    def attend(self, layer: int, seq: int, q_bits, scale: float):
        """Decode attention of one sequence's query (bf16 bits [Hq, D]) over the
        history persisted so far in `layer`.  `scale` is the fp32 softmax scale
        widened to fp64."""
        k, v = self.visible_kv(seq, layer)
        return attention(bf16_to_f64(q_bits), k, v, scale)

    def counts(self, seq: int, layer: int):
        st = self.sl(seq, layer)
        return dict(hi=len(st.hi_pos), lo=len(st.lo_pos), pos=st.n_pos, drop=st.n_drop,
                    forced=st.n_forced, R=st.R, window=int(st.w_pos.size))


# --------------------------------------------------------------------------
# Normalised KV cost (Eq. 1)
# --------------------------------------------------------------------------

def entry_bytes(n_kv_heads: int, head_dim: int):
    """Stored bytes of one (token, layer) entry per action: K and V of every KV
    head; bf16 for HIGH; int4 codes plus fp16 scales per 32 elements for LOW."""
    hi = 2 * n_kv_heads * head_dim * 2
    lo = 2 * n_kv_heads * (head_dim // 2 + 2 * (head_dim // QGROUP))
    return {DROP: 0, LOW: lo, HIGH: hi}


# --------------------------------------------------------------------------
# Online budget controller (Eq. 9-10; Alg. 2)
# --------------------------------------------------------------------------

def group_costs(group_of_layer, n_groups: int, n_kv_heads: int, head_dim: int) -> np.ndarray:
    """m(a, c): bytes one token persists in layer group c under action a, the
    stored bytes of one (token, layer) entry times the layers of the group
    (the cost accounting of Eq. 1).  int64 [n_groups][3]."""
    layers = np.bincount(np.asarray(group_of_layer, dtype=np.int64), minlength=n_groups)
    e = entry_bytes(n_kv_heads, head_dim)
    return np.array([[layers[c] * e[a] for a in (DROP, LOW, HIGH)] for c in range(n_groups)], dtype=np.int64)


def initial_budget(beta_q: int, t_max: int, m) -> int:
    """R_0 = beta * T_max * sum_c m(H, c) bytes, beta = beta_q / 65536, rounded
    down (the paper gives no R_0: the budget fraction of the bytes of T_max
    tokens kept HIGH in every layer is the reading taken here)."""
    full = int(np.asarray(m)[:, HIGH].sum())
    return (int(beta_q) * int(t_max) * full) // 65536


def reserve_bytes(reserve_q, m) -> np.ndarray:
    """Gamma(s) (Eq. 9) in bytes: reserve_q[s] sixteenths of sum_c m(H, c),
    rounded down."""
    full = int(np.asarray(m)[:, HIGH].sum())
    return np.array([(int(r) * full) // 16 for r in np.asarray(reserve_q)], dtype=np.int64)


def online_actions(z: int, s: int, R: int, action, floor, rho_up, m, gamma, crit, forced: bool):
    """The actions of one accepted token in every layer group, and their bytes.

    Follows Alg. 2 after the lookup: a_c = max(a0_c, a-_c) (Eq. 10); the budget
    available now is B = max(0, R - Gamma(s)) (Eq. 10); while the actions cost
    more than B, the group whose current action sits above its floor and whose
    last upgrade has the smallest score rho_D (Eq. 7, distortion loss per saved
    byte) is demoted one step, lower group first on ties, until the cost fits
    or only floors remain (the floors take priority); then, in a critical or
    lookahead-critical state, the eligible promotion (action below HIGH,
    positive score, fits in B) with the largest score is applied, lower group
    first on ties, until none fits.  A forced token (a sink, a tag outside the
    table) is HIGH in every group and is neither demoted nor promoted.
    Returns (actions uint8 [C], bytes)."""
    C = len(m)
    if forced:
        a = [HIGH] * C
    else:
        a = [max(int(action[z][c]), int(floor[z][c])) for c in range(C)]
    cost = sum(int(m[c][a[c]]) for c in range(C))
    if forced:
        return np.asarray(a, dtype=np.uint8), cost
    B = max(0, int(R) - int(gamma))
    while cost > B:                                                     # Demote
        best = None
        for c in range(C):
            if a[c] > int(floor[z][c]):
                loss = float(rho_up[z][c][a[c] - 1])
                if best is None or loss < best[0]:
                    best = (loss, c)
        if best is None:
            break
        c = best[1]
        cost -= int(m[c][a[c]]) - int(m[c][a[c] - 1])
        a[c] -= 1
    if crit:                                                            # Promote
        while True:
            best = None
            for c in range(C):
                if a[c] < HIGH:
                    gain = float(rho_up[z][c][a[c]])
                    extra = int(m[c][a[c] + 1]) - int(m[c][a[c]])
                    if gain > 0.0 and cost + extra <= B and (best is None or gain > best[0]):
                        best = (gain, c, extra)
            if best is None:
                break
            cost += best[2]
            a[best[1]] += 1
    return np.asarray(a, dtype=np.uint8), cost


def c_kv(n_high: int, n_low: int, n_drop: int, n_kv_heads: int, head_dim: int) -> float:
    """C_KV = sum of m(a) over (token, layer) entries / the same with every a = H."""
    m = entry_bytes(n_kv_heads, head_dim)
    tot = n_high + n_low + n_drop
    if tot == 0:
        return float("nan")
    return (n_high * m[HIGH] + n_low * m[LOW]) / (tot * m[HIGH])


# --------------------------------------------------------------------------
# Attention-output distortion (Eq. 4, Section 3.3)
# --------------------------------------------------------------------------

def output_distortion(o_full, o_int) -> float:
    """max over query heads h of ||o_full[h] - o_int[h]||_2^2: the quantity
    inside the expectation of Eq. 4 for one layer and one decode position."""
    d = np.asarray(o_full, dtype=np.float64) - np.asarray(o_int, dtype=np.float64)
    return float(np.max(np.sum(d * d, axis=-1)))


def intervention_table(n_tags: int, n_groups: int, tag: int, group: int, action: int):
    """(action, floor) tables of a one-bucket intervention (Section 3.3):
    bucket (tag, group) gets `action`, every other bucket HIGH, floors at
    DROP so the lookup returns exactly those actions."""
    a = np.full((n_tags, n_groups), HIGH, dtype=np.uint8)
    a[tag, group] = action
    return a, np.zeros_like(a)


def distortion(tags, k_bits, v_bits, q_bits, prompt_len: int, group_of_layer, n_tags: int, tag: int, group: int,
               action: int, scale: float):
    """D(q, a) of Eq. 4 for bucket q = (tag, group) on reference trajectories.

    tags [R, T]: tags of the T generated tokens of R trajectories; k_bits,
    v_bits [R, L, P + T, Hkv, D]: bf16 K / V of every position and layer (the
    P prompt positions first, kept HIGH in both runs); q_bits [R, L, T, Hq, D]:
    the query of every decode step.  Step u appends position P + u, then
    attends with its query (the token sees itself at its persisted precision).

    The reference run keeps every bucket HIGH; the intervened run gives
    bucket (tag, group) the action `action`.  S(q) holds the steps (r, u)
    whose history contains a generated token with tag `tag`, i.e. the steps
    from the bucket's first occurrence in r on.  Returns
    sum over layers l of group `group` of the mean over S(q) of
    max_h ||o_full - o_a||^2, and |S(q)|; D = 0 when S(q) is empty."""
    tags = np.asarray(tags)
    R, T = tags.shape
    gol = np.asarray(group_of_layer)
    L = gol.size
    hkv, d = k_bits.shape[-2], k_bits.shape[-1]
    layers = [l for l in range(L) if gol[l] == group]
    full = dict(action=np.full((n_tags, int(gol.max()) + 1), HIGH, np.uint8), group_of_layer=gol, n_sink=0)
    full["floor"] = np.zeros_like(full["action"])
    a_int, f_int = intervention_table(n_tags, int(gol.max()) + 1, tag, group, action)
    inter = dict(action=a_int, floor=f_int, group_of_layer=gol, n_sink=0)
    total, n_s = 0.0, 0
    for r in range(R):
        ref, itv = OracleCache(full, hkv, d), OracleCache(inter, hkv, d)
        for l in layers:
            for c in (ref, itv):
                c.append(l, 0, np.zeros(prompt_len, np.uint8), k_bits[r, l, :prompt_len], v_bits[r, l, :prompt_len],
                         keep_all=True)
        seen = False
        for u in range(T):
            seen |= int(tags[r, u]) == tag
            for l in layers:
                for c in (ref, itv):
                    c.append(l, 0, tags[r, u:u + 1], k_bits[r, l, prompt_len + u][None],
                             v_bits[r, l, prompt_len + u][None])
            if not seen:
                continue
            n_s += 1
            for l in layers:
                o_full, _ = ref.attend(l, 0, q_bits[r, l, u], scale)
                o_int, _ = itv.attend(l, 0, q_bits[r, l, u], scale)
                total += output_distortion(o_full, o_int)
    return (total / n_s if n_s else 0.0), n_s
