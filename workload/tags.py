"""Structural-tag streams.

The paper derives a tag for every generated token from the accepted parser
transition of a grammar-constrained decoder (Section 3.2, Eq. 3), and labels
prompt tokens by input-derived semantic classes for its prefill companion
(Section 3.5).  No decoder, grammar engine or benchmark data is used here:
these seeded generators emit tag ids with the shape of function-call output
(a JSON object per call, keys, enum / string / number arguments, nested
objects) and of tool-schema prompts.  Nothing is taken from any benchmark.
"""

from __future__ import annotations

import numpy as np

# Six decode tags (generated tokens) and six prompt labels (prompt tokens).
DECODE_TAGS = ("required_key", "enum_value", "arg_value", "boundary", "scaffold", "free_text")
PROMPT_TAGS = ("protected_content", "function_name", "param_key", "constraint",
               "schema_scaffold", "instruction_text")
REQUIRED_KEY, ENUM_VALUE, ARG_VALUE, BOUNDARY, SCAFFOLD, FREE_TEXT = range(6)
PROTECTED, FUNC_NAME, PARAM_KEY, CONSTRAINT, SCHEMA_SCAFFOLD, INSTRUCTION = range(6, 12)


# Parser states of the synthetic function-call grammar (the s_t of the online
# lookup, Section 3.4): where the parser frontier is when a token is accepted.
PARSER_STATES = ("text", "expect_key", "key", "expect_value", "enum", "argument", "close")
ST_TEXT, ST_EXPECT_KEY, ST_KEY, ST_EXPECT_VALUE, ST_ENUM, ST_ARG, ST_CLOSE = range(7)
# Critical or lookahead-critical states: a key or an enumerated value is being
# produced, or the next token must be one.
CRITICAL_STATES = (ST_EXPECT_KEY, ST_KEY, ST_EXPECT_VALUE, ST_ENUM)


def iid_tags(n: int, seed: int, n_tags: int = 6) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_tags, size=n).astype(np.uint8)


class _Walker:
    """Emits the tags of back-to-back function calls.

    Each call is an optional free-text preamble followed by
    {"name": <function>, "arguments": {k1: v1, ...}} with 1-6 keys; values are
    enum, string or number tokens or a nested object (depth <= 3).  Quotes and
    fixed template words are scaffold, delimiters are boundary."""

    def __init__(self, rng: np.random.Generator):
        self.rng = rng
        self.out: list[int] = []
        self.states: list[int] = []

    def emit(self, tag: int, state: int, n: int = 1):
        self.out.extend([tag] * n)
        self.states.extend([state] * n)

    def value(self, depth: int):
        r = self.rng.random()
        if depth < 3 and r < 0.10:
            self.obj(depth + 1, int(self.rng.integers(1, 4)))
        elif r < 0.40:                       # enum value, quoted
            self.emit(SCAFFOLD, ST_ENUM)
            self.emit(ENUM_VALUE, ST_ENUM, int(self.rng.integers(1, 3)))
        elif r < 0.80:                       # string argument, quoted
            self.emit(SCAFFOLD, ST_ARG)
            self.emit(ARG_VALUE, ST_ARG, int(self.rng.integers(1, 11)))
        else:                                # number argument
            self.emit(ARG_VALUE, ST_ARG, int(self.rng.integers(1, 4)))

    def obj(self, depth: int, n_keys: int):
        self.emit(BOUNDARY, ST_EXPECT_KEY)   # {
        for i in range(n_keys):
            if i:
                self.emit(BOUNDARY, ST_EXPECT_KEY)   # ,
            if self.rng.random() < 0.5:
                self.emit(SCAFFOLD, ST_KEY)  # opening quote as its own token
            self.emit(REQUIRED_KEY, ST_KEY, int(self.rng.integers(1, 6)))
            self.emit(BOUNDARY, ST_EXPECT_VALUE)     # ":
            self.value(depth)
        self.emit(BOUNDARY, ST_CLOSE)        # }

    def call(self):
        if self.rng.random() < 0.7:
            self.emit(FREE_TEXT, ST_TEXT, int(self.rng.integers(3, 16)))
        self.emit(BOUNDARY, ST_EXPECT_KEY)   # {
        self.emit(SCAFFOLD, ST_KEY, 2)       # "name":
        self.emit(ENUM_VALUE, ST_ENUM, int(self.rng.integers(1, 4)))
        self.emit(BOUNDARY, ST_EXPECT_KEY)   # ,
        self.emit(SCAFFOLD, ST_KEY, 2)       # "arguments":
        self.obj(1, int(self.rng.integers(1, 7)))
        self.emit(BOUNDARY, ST_CLOSE)        # }


def walk_function_calls(n: int, seed: int) -> np.ndarray:
    """Tags of n generated tokens from back-to-back synthetic function calls."""
    return walk_function_calls_with_states(n, seed)[0]


def walk_function_calls_with_states(n: int, seed: int):
    """(tags, parser states) of n generated tokens; the tags are those of
    walk_function_calls with the same seed."""
    w = _Walker(np.random.default_rng(seed))
    while len(w.out) < n:
        w.call()
    return np.asarray(w.out[:n], dtype=np.uint8), np.asarray(w.states[:n], dtype=np.uint8)


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
