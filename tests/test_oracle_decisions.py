"""Pins of the oracle's decisions and compaction (Section 3.1 action order;
Eq. 10 / Alg. 2 lookup-and-max; release semantics)."""

import itertools

import numpy as np
import pytest

import oracle
from workload.policy import contiguous_groups, make_policy, uniform_policy
from workload.tags import iid_tags, function_call_tags

# The paper's order R < L < H written as a truth table of "the higher of two".
PAPER_MAX = {("R", "R"): "R", ("R", "L"): "L", ("R", "H"): "H",
             ("L", "R"): "L", ("L", "L"): "L", ("L", "H"): "H",
             ("H", "R"): "H", ("H", "L"): "H", ("H", "H"): "H"}
CODE = {"R": oracle.DROP, "L": oracle.LOW, "H": oracle.HIGH}


def test_max_follows_paper_order():
    for (a0, am), want in PAPER_MAX.items():
        action = np.array([[CODE[a0]]], dtype=np.uint8)
        floor = np.array([[CODE[am]]], dtype=np.uint8)
        got, forced, bad = oracle.decide([0], [5], 0, action, floor, n_sink=0, keep_all=False)
        assert got[0] == CODE[want] and not forced[0] and not bad[0]


def test_overrides():
    action = np.zeros((6, 2), dtype=np.uint8)
    floor = np.zeros((6, 2), dtype=np.uint8)
    # sinks
    got, forced, _ = oracle.decide([1, 1, 1, 1], [0, 1, 2, 3], 1, action, floor, n_sink=2, keep_all=False)
    assert got.tolist() == [2, 2, 0, 0] and forced.tolist() == [True, True, False, False]
    # keep-all (prompt not governed by the table)
    got, forced, _ = oracle.decide([1, 2, 3], [10, 11, 12], 0, action, floor, n_sink=0, keep_all=True)
    assert (got == 2).all() and forced.all()
    # tag outside the table: HIGH and flagged
    got, forced, bad = oracle.decide([6, 0], [10, 11], 0, action, floor, n_sink=0, keep_all=False)
    assert got.tolist() == [2, 0] and bad.tolist() == [True, False]


def _bruteforce_visible(tags, group, action, floor):
    """Mask-based brute force: position p is visible at precision a iff the
    (tag, group) bucket's higher-of(selected, floor) action is a; built by
    scanning every bucket's mask instead of per-token lookup."""
    tags = np.asarray(tags)
    n_tags = action.shape[0]
    hi = np.zeros(tags.size, dtype=bool)
    lo = np.zeros(tags.size, dtype=bool)
    for z in range(n_tags):
        mask = tags == z
        a = PAPER_MAX[("RLH"[action[z, group]], "RLH"[floor[z, group]])]
        if a == "H":
            hi |= mask
        elif a == "L":
            lo |= mask
    pos = np.arange(tags.size)
    return pos[hi], pos[lo]


def test_exhaustive_tiny_tables():
    """Every (selected, floor) table for T=2, C=1 and for T=1, C=2 (3^4 each)."""
    rng = np.random.default_rng(0)
    for T, C in [(2, 1), (1, 2)]:
        for vals in itertools.product(range(3), repeat=2 * T * C):
            action = np.array(vals[:T * C], dtype=np.uint8).reshape(T, C)
            floor = np.array(vals[T * C:], dtype=np.uint8).reshape(T, C)
            tags = rng.integers(0, T, size=13)
            for c in range(C):
                acts, _, _ = oracle.decide(tags, np.arange(13), c, action, floor, 0, False)
                hi, lo = oracle.compact(acts, np.arange(13))
                bhi, blo = _bruteforce_visible(tags, c, action, floor)
                assert hi.tolist() == bhi.tolist() and lo.tolist() == blo.tolist()


def test_counts_closed_form_from_table():
    """n_H, n_L, n_R per group equal tag counts weighted by the table."""
    pol = make_policy(6, 4, 36, 0.33, seed=11)
    tags = function_call_tags(5000, 3)
    counts = np.bincount(tags, minlength=6)
    eff = np.maximum(pol.action, pol.floor)
    cache = oracle.OracleCache(dict(action=pol.action, floor=pol.floor,
                                    group_of_layer=pol.group_of_layer, n_sink=0), 1, 32)
    kv = np.zeros((tags.size, 1, 32), dtype=np.int64)
    for layer in range(0, 36, 9):
        c = int(pol.group_of_layer[layer])
        cache.append(layer, 0, tags, kv, kv)
        got = cache.counts(0, layer)
        assert got["hi"] == int(counts[eff[:, c] == 2].sum())
        assert got["lo"] == int(counts[eff[:, c] == 1].sum())
        assert got["drop"] == int(counts[eff[:, c] == 0].sum())
        assert got["hi"] + got["lo"] + got["drop"] == got["pos"] == tags.size


def test_lists_partition_and_order():
    pol = make_policy(6, 2, 2, 0.33, seed=5)
    tags = iid_tags(300, 4)
    acts, _, _ = oracle.decide(tags, np.arange(300), 1, pol.action, pol.floor, 0, False)
    hi, lo = oracle.compact(acts, np.arange(300))
    assert (np.diff(hi) > 0).all() and (np.diff(lo) > 0).all()
    assert not set(hi) & set(lo)
    dropped = set(np.nonzero(acts == 0)[0].tolist())
    assert set(hi) | set(lo) | dropped == set(range(300))


def test_incremental_equals_bulk_append():
    """Persisting tokens one call at a time equals persisting them in one call."""
    rng = np.random.default_rng(1)
    pol = make_policy(6, 2, 2, 0.33, seed=6)
    p = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=3)
    a, b = oracle.OracleCache(p, 2, 64), oracle.OracleCache(p, 2, 64)
    tags = iid_tags(40, 2)
    kv = rng.integers(0, 0x7F00, size=(40, 2, 64)) | (rng.integers(0, 2, size=(40, 2, 64)) << 15)
    a.append(1, 0, tags, kv, kv)
    for i in range(40):
        b.append(1, 0, tags[i:i + 1], kv[i:i + 1], kv[i:i + 1])
    assert [x.tolist() for x in a.lists(0, 1)] == [x.tolist() for x in b.lists(0, 1)]
    for x, y in zip(a.lo_entries(0, 1), b.lo_entries(0, 1)):
        assert (x == y).all()


def test_lists_identical_across_layers_of_a_group():
    pol = make_policy(6, 4, 36, 0.33, seed=2)
    p = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=0)
    cache = oracle.OracleCache(p, 1, 32)
    tags = function_call_tags(400, 9)
    kv = np.zeros((400, 1, 32), dtype=np.int64)
    for layer in range(36):
        cache.append(layer, 0, tags, kv, kv)
    for c in range(4):
        layers = np.nonzero(pol.group_of_layer == c)[0]
        ref = [x.tolist() for x in cache.lists(0, layers[0])]
        for layer in layers[1:]:
            assert [x.tolist() for x in cache.lists(0, layer)] == ref


@pytest.mark.parametrize("mutant", ["min_instead_of_max", "floor_ignored", "group_from_layer_mod"])
def test_planted_decision_mistakes_are_caught(mutant, monkeypatch):
    import oracle.pask_oracle as po
    good = po.decide

    if mutant == "min_instead_of_max":
        def bad(tags, positions, group, action, floor, n_sink, keep_all):
            return good(tags, positions, group, np.minimum(action, floor), np.minimum(action, floor),
                        n_sink, keep_all)
    elif mutant == "floor_ignored":
        def bad(tags, positions, group, action, floor, n_sink, keep_all):
            return good(tags, positions, group, action, np.zeros_like(floor), n_sink, keep_all)
    else:
        def bad(tags, positions, group, action, floor, n_sink, keep_all):
            return good(tags, positions, (group + 1) % action.shape[1], action, floor, n_sink, keep_all)
    monkeypatch.setattr(po, "decide", bad)
    rng = np.random.default_rng(0)
    caught = False
    for T, C in [(2, 1), (1, 2)]:
        for vals in itertools.product(range(3), repeat=2 * T * C):
            action = np.array(vals[:T * C], dtype=np.uint8).reshape(T, C)
            floor = np.array(vals[T * C:], dtype=np.uint8).reshape(T, C)
            tags = rng.integers(0, T, size=13)
            for c in range(C):
                acts, _, _ = po.decide(tags, np.arange(13), c, action, floor, 0, False)
                hi, lo = po.compact(acts, np.arange(13))
                bhi, blo = _bruteforce_visible(tags, c, action, floor)
                caught |= hi.tolist() != bhi.tolist() or lo.tolist() != blo.tolist()
    assert caught


def test_contiguous_groups():
    assert contiguous_groups(36, 4).tolist() == [0] * 9 + [1] * 9 + [2] * 9 + [3] * 9
    assert uniform_policy(6, 2, 2, 2).action.min() == 2
