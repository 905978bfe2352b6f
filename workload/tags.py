"""Structural-tag streams.

The paper derives a tag for every generated token from the accepted parser
transition of a grammar-constrained decoder (Section 3.2, Eq. 3), and labels
prompt tokens by input-derived semantic classes for its prefill companion
(Section 3.5).  Generated tokens: seeded tool-call output (workload.calls)
read by the tagger's pushdown automaton (paper_2608_28276_amd.tagger), which
gives each token its tag and parser state.  Prompt tokens: a seeded labeller
with the shape of tool-schema prompts.  No model, grammar package or
benchmark data is used; nothing is taken from any benchmark.
"""

from __future__ import annotations

import numpy as np

from paper_2608_28276_amd import tagger as _tagger

from .calls import function_call_output

# Six decode tags (generated tokens; the tagger's map from z_t) and six prompt
# labels (prompt tokens).
DECODE_TAGS = _tagger.TAG_NAMES
PROMPT_TAGS = ("protected_content", "function_name", "param_key", "constraint",
               "schema_scaffold", "instruction_text")
REQUIRED_KEY, ENUM_VALUE, ARG_VALUE, BOUNDARY, SCAFFOLD, FREE_TEXT = range(6)
PROTECTED, FUNC_NAME, PARAM_KEY, CONSTRAINT, SCHEMA_SCAFFOLD, INSTRUCTION = range(6, 12)


# Parser states and Crit(s) of the tagger's automaton (the s_t of the online
# lookup, Section 3.4): the parser position after a token combined with what
# the frontier must produce next.
PARSER_STATES = tuple(f"{lex}/{nxt}" for lex in _tagger.LEX for nxt in _tagger.NEXTS)
CRITICAL_STATES = _tagger.CRITICAL_STATES


def iid_tags(n: int, seed: int, n_tags: int = 6) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_tags, size=n).astype(np.uint8)


def function_call_tags_with_states(n: int, seed: int):
    """(tags, parser states) of n generated tokens of back-to-back calls to a
    seeded set of invented tools: the token stream of workload.calls, read by
    the tagger's pushdown automaton (structural tag z_t -> decode tag id;
    parser state id for the controller)."""
    tools, toks = function_call_output(n, seed)
    tags, states = _tagger.tag_stream(tools, toks[:n])
    return np.asarray(tags, dtype=np.uint8), np.asarray(states, dtype=np.uint8)


def function_call_tags(n: int, seed: int) -> np.ndarray:
    """Decode tags of n generated tokens (function_call_tags_with_states)."""
    return function_call_tags_with_states(n, seed)[0]


def schema_prompt_tags(n: int, seed: int) -> np.ndarray:
    """Labels of an n-token prompt: tool schemas (function name, parameter keys,
    constraints, schema scaffold) interleaved with instruction text that
    carries protected content (user-supplied values)."""
    rng = np.random.default_rng(seed)
    out: list[int] = []

    def emit(tag, k):
        out.extend([tag] * int(k))

    while len(out) < n:
        if rng.random() < 0.35:              # instruction paragraph
            for _ in range(int(rng.integers(1, 5))):
                emit(INSTRUCTION, rng.integers(5, 30))
                if rng.random() < 0.5:
                    emit(PROTECTED, rng.integers(1, 8))
        else:                                # one tool schema
            emit(SCHEMA_SCAFFOLD, rng.integers(3, 8))
            emit(FUNC_NAME, rng.integers(1, 5))
            emit(SCHEMA_SCAFFOLD, rng.integers(2, 5))
            emit(INSTRUCTION, rng.integers(5, 25))   # description
            for _ in range(int(rng.integers(1, 7))):
                emit(SCHEMA_SCAFFOLD, rng.integers(2, 5))
                emit(PARAM_KEY, rng.integers(1, 4))
                emit(SCHEMA_SCAFFOLD, rng.integers(2, 6))
                emit(CONSTRAINT, rng.integers(1, 8))
                if rng.random() < 0.5:
                    emit(INSTRUCTION, rng.integers(3, 15))
            emit(SCHEMA_SCAFFOLD, rng.integers(2, 5))
    return np.asarray(out[:n], dtype=np.uint8)


def tag_mix(tags: np.ndarray, n_tags: int) -> np.ndarray:
    """Empirical tag frequencies."""
    counts = np.bincount(np.asarray(tags, dtype=np.int64), minlength=n_tags)[:n_tags]
    return counts / max(1, counts.sum())
