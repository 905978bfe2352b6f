"""The seeded input generators: determinism, shapes and the tag mix."""

import struct

import numpy as np

from workload import CONFIGS, make_policy, pack_blob, prompt_lengths, tag_mix, function_call_tags
from workload.policy import fnv1a32
from workload.tags import schema_prompt_tags
from workload.tensors import bf16_normal


def test_call_tags_deterministic_and_mix():
    a = function_call_tags(50000, 17)
    assert (a == function_call_tags(50000, 17)).all() and a.size == 50000
    m = tag_mix(a, 6)
    # ~35% scaffold+boundary, 25% keys, 30% argument values, 10% free text.
    assert abs(m[3] + m[4] - 0.35) < 0.07
    assert abs(m[0] - 0.25) < 0.05
    assert abs(m[1] + m[2] - 0.30) < 0.05
    assert abs(m[5] - 0.10) < 0.04


def test_schema_prompt_labels_in_range():
    t = schema_prompt_tags(20000, 3)
    assert t.min() >= 6 and t.max() <= 11 and t.size == 20000


def test_policy_budget_and_blob_layout():
    for cfg in CONFIGS:
        pol = make_policy(cfg.n_tags, cfg.n_groups, cfg.n_layers, 0.33, cfg.seed)
        assert abs(pol.expected_cost - 0.33) < 0.02 or pol.expected_cost < 0.33
        blob = pack_blob(pol)
        magic, ver, hdr, T, C, L, sink, win, body = struct.unpack_from("<4sHHIIIIII", blob)
        assert magic == b"PASK" and ver == 1 and hdr == 32 and (T, C, L) == (cfg.n_tags, cfg.n_groups, cfg.n_layers)
        assert len(blob) == 32 + body + 4
        assert struct.unpack_from("<I", blob, len(blob) - 4)[0] == fnv1a32(blob[:-4])


def test_prompt_lengths_ranges():
    for cfg in CONFIGS:
        p = prompt_lengths(cfg)
        assert p.shape == (cfg.batch,)
        assert p.min() >= cfg.prompt_min and p.max() <= cfg.prompt_max


def test_bf16_normal_seeded():
    a = bf16_normal((4, 8), 5)
    b = bf16_normal((4, 8), 5)
    assert (a == b).all() and a.shape == (4, 8)


def test_tagger_states_align_with_tags_and_reserve_follows_eq8():
    """Parser states come with the same tag stream: free text is read outside
    calls, enum values and keys inside their strings or right at their end;
    Gamma(s) is the median future floor cost, so it shrinks toward the end
    of a trace and a state that never occurs reserves nothing."""
    from paper_2608_28276_amd import tagger as tg
    from workload.tags import (function_call_tags_with_states, CRITICAL_STATES, PARSER_STATES, REQUIRED_KEY,
                               ENUM_VALUE, FREE_TEXT)
    from workload.policy import with_budget_controller, pack_blob, floor_cost
    tags, states = function_call_tags_with_states(5000, 17)
    assert (tags == function_call_tags(5000, 17)).all()
    assert states.max() < len(PARSER_STATES) == tg.N_STATES
    lex = states // 3
    assert set(lex[tags == FREE_TEXT]) <= {tg.S_TEXT}
    assert set(lex[tags == REQUIRED_KEY]) <= {tg.S_IN_KEY, tg.S_EXPECT_COLON, tg.S_EXPECT_VALUE, tg.S_IN_STRING,
                                             tg.S_IN_ENUM}
    assert set(lex[tags == ENUM_VALUE]) <= {tg.S_IN_ENUM, tg.S_AFTER_VALUE, tg.S_EXPECT_KEY, tg.S_EXPECT_VALUE,
                                           tg.S_END}
    assert (lex[tags == REQUIRED_KEY] == tg.S_IN_KEY).mean() > 0.9
    pol = make_policy(6, 2, 4, 0.33, seed=3)
    trace = (tags[:200], states[:200])
    bp = with_budget_controller(pol, [trace], len(PARSER_STATES) + 1, CRITICAL_STATES)
    f = floor_cost(pol, trace[0])
    future = np.array([f[u + 1:].sum() for u in range(200)])
    for s in range(len(PARSER_STATES)):
        sel = trace[1] == s
        if sel.any():
            assert bp.reserve_q[s] == int(round(16 * np.quantile(future[sel], 0.5)))
    assert bp.reserve_q[len(PARSER_STATES)] == 0
    assert bp.crit.tolist()[:len(PARSER_STATES)] == [int(s in CRITICAL_STATES) for s in range(len(PARSER_STATES))]
    blob = pack_blob(bp)
    assert blob[4:6] == (2).to_bytes(2, "little") and len(blob) > len(pack_blob(pol))
