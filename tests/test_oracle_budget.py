"""Pins of the oracle's online budget controller (Alg. 2; Eq. 9-10).

Hand-worked cases on a three-group table fix the demotion order (ascending
upgrade score of the step being undone, lower group on ties), the floors'
priority, the reserve Gamma(s) and the promotions of critical states; random
tables check the invariants the algorithm guarantees; planted mistakes in the
controller each fail one of the pins."""

import itertools

import numpy as np
import pytest

import oracle
from oracle.pask_oracle import HIGH, LOW, DROP

# m(a, c) in bytes for three groups; one tag (z = 0).
M = np.array([[0, 3, 10], [0, 6, 20], [0, 3, 10]], dtype=np.int64)
ACTION = np.array([[HIGH, HIGH, LOW]], dtype=np.uint8)
FLOOR = np.array([[LOW, DROP, DROP]], dtype=np.uint8)
RHO = np.array([[[5.0, 1.0], [2.0, 0.5], [4.0, 3.0]]], dtype=np.float32)   # per group: (R->L, L->H)
GAMMA = np.array([0, 8], dtype=np.int64)      # state 0: no reserve, state 1: 8 bytes
CRIT = np.array([0, 1], dtype=np.uint8)        # state 1 is critical


def run(R, s, action=ACTION, floor=FLOOR, rho=RHO, m=M, gamma=GAMMA, crit=CRIT, forced=False, fn=None):
    fn = fn or oracle.online_actions
    a, cost = fn(0, s, R, action, floor, rho, m, int(gamma[s]), bool(crit[s]), forced)
    return [int(x) for x in a], int(cost)


# Worked by hand from the algorithm (actions per group, bytes):
#  (a) R=100, s=0: B=100 >= 33: no change.
#  (b) R=25: B=25 < 33; losses c0 1.0 (H->L), c1 0.5 (H->L), c2 4.0 (L->R): demote c1 -> 19 <= 25.
#  (c) R=10: after c1: losses c0 1.0, c1 2.0 (L->R), c2 4.0: demote c0 -> 12; then c1 2.0 -> 6 <= 10.
#  (d) R=0: c1, c0, c1, c2 in that order; c0 stops at its floor L: cost 3 > B = 0 (floors win).
#  (e) R=40, s=1: B=32 < 33: demote c1 -> 19; critical: promote c2 (score 3.0, +7 -> 26);
#      c1's promotion (+14 -> 40) does not fit.
#  (g) R=60, s=1: B=52 >= 33: promote c2 -> 40; every group at HIGH.
CASES = [
    (100, 0, [HIGH, HIGH, LOW], 33),
    (25, 0, [HIGH, LOW, LOW], 19),
    (10, 0, [LOW, DROP, LOW], 6),
    (0, 0, [LOW, DROP, DROP], 3),
    (40, 1, [HIGH, LOW, HIGH], 26),
    (60, 1, [HIGH, HIGH, HIGH], 40),
]


@pytest.mark.parametrize("R,s,want,cost", CASES)
def test_worked_cases(R, s, want, cost):
    assert run(R, s) == (want, cost)


def test_ties_go_to_the_lower_group():
    """Equal scores everywhere, every action HIGH, floors DROP, R=25: c0 is
    demoted twice (40 -> 33 -> 30), then c1 once (-> 16 <= 25)."""
    act = np.full((1, 3), HIGH, np.uint8)
    flo = np.zeros((1, 3), np.uint8)
    rho = np.ones((1, 3, 2), np.float32)
    assert run(25, 0, action=act, floor=flo, rho=rho) == ([DROP, LOW, HIGH], 16)


def test_forced_token_is_high_everywhere():
    assert run(0, 1, forced=True) == ([HIGH, HIGH, HIGH], 40)


def test_costs_budget_and_reserve_units():
    """m(a, c) = layers of c x entry bytes: groups of 2 and 1 layers, 2 KV heads,
    head_dim 64: HIGH 512 B, LOW 2*2*(32+4) = 144 B per (token, layer)."""
    m = oracle.group_costs([0, 0, 1], 2, 2, 64)
    assert m.tolist() == [[0, 288, 1024], [0, 144, 512]]
    # R_0 = floor(beta_q * T_max * sum_c m(H, c) / 65536); beta_q = 21627 (~0.33), T_max = 1024
    assert oracle.initial_budget(21627, 1024, m) == 519048
    # Gamma = floor(reserve_q * sum_c m(H, c) / 16); 1755 sixteenths
    assert oracle.reserve_bytes([1755, 0], m).tolist() == [168480, 0]


def _random_table(rng, T, C):
    action = rng.integers(0, 3, size=(T, C)).astype(np.uint8)
    floor = rng.integers(0, 3, size=(T, C)).astype(np.uint8)
    rho = (rng.integers(0, 6, size=(T, C, 2)) * 0.25).astype(np.float32)   # ties are common
    layers = rng.integers(1, 5, size=C)
    m = np.stack([np.zeros(C), 9 * layers, 32 * layers], axis=1).astype(np.int64)
    return action, floor, rho, m


def test_invariants_on_random_tables():
    rng = np.random.default_rng(3)
    for _ in range(3000):
        T, C = int(rng.integers(1, 4)), int(rng.integers(1, 6))
        action, floor, rho, m = _random_table(rng, T, C)
        z = int(rng.integers(0, T))
        R = int(rng.integers(-50, 400))
        gamma = int(rng.integers(0, 100))
        crit = bool(rng.integers(0, 2))
        a, cost = oracle.online_actions(z, 0, R, action, floor, rho, m, gamma, crit, False)
        a = a.astype(int)
        eq10 = np.maximum(action[z], floor[z]).astype(int)
        B = max(0, R - gamma)
        assert (a >= floor[z]).all(), "never below the floor"
        assert cost == sum(int(m[c][a[c]]) for c in range(C))
        if not crit:
            assert (a <= eq10).all(), "only demotions outside critical states"
            assert cost <= B or (a == np.minimum(eq10, floor[z])).all(), "fits, or only floors remain"
        if cost > B:
            assert (a == floor[z]).all()
        # more budget never lowers an action outside critical states
        if not crit:
            a2, _ = oracle.online_actions(z, 0, R + 37, action, floor, rho, m, gamma, False, False)
            assert (a2.astype(int) >= a).all()


def test_ample_budget_no_reserve_is_the_static_lookup():
    """With a budget no token can exhaust, no reserve and no critical state,
    the controller returns Eq. 10's max for every bucket."""
    for vals in itertools.product(range(3), repeat=4):
        action = np.array(vals[:2], np.uint8).reshape(1, 2)
        floor = np.array(vals[2:], np.uint8).reshape(1, 2)
        a, _ = oracle.online_actions(0, 0, 10**9, action, floor, np.ones((1, 2, 2), np.float32),
                                     M[:2], 0, False, False)
        assert a.tolist() == np.maximum(action[0], floor[0]).tolist()


def _budget_cache(beta_q=21627, reserve=(1755, 400, 900), crit=(0, 1, 1)):
    from workload import make_policy
    pol = make_policy(6, 2, 4, 0.33, seed=5)
    d = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=0,
             rho_up=pol.rho_up, n_states=len(reserve), beta_q=beta_q,
             reserve_q=np.array(reserve, np.uint32), crit=np.array(crit, np.uint8))
    return oracle.OracleCache(d, 2, 64), pol


def test_cache_bulk_equals_one_by_one_and_layers_of_a_group_agree():
    rng = np.random.default_rng(11)
    n = 300
    tags = rng.integers(0, 6, size=n)
    states = rng.integers(0, 3, size=n)
    kv = np.zeros((n, 2, 64), np.uint16)
    a, _ = _budget_cache()
    b, _ = _budget_cache()
    a.budget_init(0, range(4), 200)
    b.budget_init(0, range(4), 200)
    for layer in range(4):
        a.append(layer, 0, tags, kv, kv, states=states)
        for i in range(n):
            b.append(layer, 0, tags[i:i + 1], kv[i:i + 1], kv[i:i + 1], states=states[i:i + 1])
    for layer in range(4):
        assert [x.tolist() for x in a.lists(0, layer)] == [x.tolist() for x in b.lists(0, layer)]
        assert a.counts(0, layer)["R"] == b.counts(0, layer)["R"]
    # layers 0, 1 form group 0 and layers 2, 3 group 1 (contiguous groups)
    assert [x.tolist() for x in a.lists(0, 0)] == [x.tolist() for x in a.lists(0, 1)]
    assert [x.tolist() for x in a.lists(0, 2)] == [x.tolist() for x in a.lists(0, 3)]
    assert len({a.counts(0, layer)["R"] for layer in range(4)}) == 1


def test_cache_budget_accounting_matches_the_stored_decisions():
    """R_0 - R_T equals the bytes of the actions that the stores hold, summed
    over groups (one layer per group read back)."""
    rng = np.random.default_rng(12)
    n = 400
    tags, states = rng.integers(0, 6, size=n), rng.integers(0, 3, size=n)
    kv = np.zeros((n, 2, 64), np.uint16)
    oc, pol = _budget_cache()
    oc.budget_init(0, range(4), 300)
    for layer in range(4):
        oc.append(layer, 0, tags, kv, kv, states=states)
    spent = 0
    for c, layer in enumerate((0, 2)):
        hi, lo = oc.lists(0, layer)
        spent += hi.size * int(oc.m[c][HIGH]) + lo.size * int(oc.m[c][LOW])
    assert oracle.initial_budget(21627, 300, oc.m) - oc.counts(0, 0)["R"] == spent
    # the controller bit: a tight budget demotes, so the stores differ from Eq. 10
    static, _ = _budget_cache()
    for layer in range(4):
        static.append(layer, 0, tags, kv, kv)
    assert sum(x.size for x in oc.lists(0, 0)) < sum(x.size for x in static.lists(0, 0)) or \
        oc.lists(0, 0)[0].size < static.lists(0, 0)[0].size


@pytest.mark.parametrize("mutant", ["descending_demotion", "ties_to_higher_group", "promote_everywhere",
                                    "score_of_wrong_step", "reserve_ignored"])
def test_planted_controller_mistakes_are_caught(mutant):
    good = oracle.online_actions

    def bad(z, s, R, action, floor, rho, m, gamma, crit, forced):
        if mutant == "descending_demotion":
            return good(z, s, R, action, floor, -rho if not crit else rho, m, gamma, crit, forced)
        if mutant == "ties_to_higher_group":
            a, cost = good(z, s, R, action[:, ::-1], floor[:, ::-1], rho[:, ::-1], m[::-1], gamma, crit, forced)
            return a[::-1], cost
        if mutant == "promote_everywhere":
            return good(z, s, R, action, floor, rho, m, gamma, True, forced)
        if mutant == "score_of_wrong_step":
            return good(z, s, R, action, floor, rho[..., ::-1], m, gamma, crit, forced)
        return good(z, s, R, action, floor, rho, m, 0, crit, forced)

    caught = any(run(R, s, fn=bad) != (want, cost) for R, s, want, cost in CASES)
    act = np.full((1, 3), HIGH, np.uint8)
    caught |= run(25, 0, action=act, floor=np.zeros((1, 3), np.uint8), rho=np.ones((1, 3, 2), np.float32),
                  fn=bad) != ([DROP, LOW, HIGH], 16)
    assert caught, mutant
