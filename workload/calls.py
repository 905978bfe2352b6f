"""Seeded synthetic tool-calling output: tool schemas, schema-valid call text
and a deterministic sub-word tokenizer.

The paper's decode tags come from the parser of a grammar-constrained decoder
running a model on function-calling tasks (Section 4.1).  Neither the model
nor the benchmark is used here: tools are invented from a seeded syllable
vocabulary (no benchmark item, name or text), their calls are drawn as JSON
that satisfies the schema, and the text is cut into tokens the way a
byte-pair tokenizer cuts JSON (merged punctuation such as `{"` or `": "`,
words in pieces of a few letters with a leading space).  The structural tags
are then read off the token stream by the parser in
paper_2608_28276_amd.tagger.

Shape of the output (tuned so that the tag mix is near the serving
workloads' 35% scaffold + boundary, 25% keys, 30% argument and enum values,
10% free text): back-to-back calls, each an optional free-text preamble and
{"name": <tool>, "arguments": {...}} with 1-6 parameters whose values are
enums, strings, numbers, booleans, nested objects (depth <= 3) or short
arrays.
"""

from __future__ import annotations

import json
import re
import zlib

import numpy as np

_ONSETS = ("b", "c", "d", "f", "g", "h", "k", "l", "m", "n", "p", "r", "s", "t", "v", "z", "br", "st", "tr",
           "pl", "gr", "sh", "ch")
_NUCLEI = ("a", "e", "i", "o", "u", "ai", "ou", "ei")
_CODAS = ("", "", "", "n", "r", "s", "l", "t", "m", "x")


def _word(rng: np.random.Generator, lo: int = 1, hi: int = 3) -> str:
    n = int(rng.integers(lo, hi + 1))
    return "".join(str(rng.choice(_ONSETS)) + str(rng.choice(_NUCLEI)) + str(rng.choice(_CODAS)) for _ in range(n))


def _ident(rng: np.random.Generator, lo: int = 1, hi: int = 3) -> str:
    return "_".join(_word(rng, 1, 2) for _ in range(int(rng.integers(lo, hi + 1))))


def _param_schema(rng: np.random.Generator, depth: int) -> dict:
    r = rng.random()
    if depth < 3 and r < 0.08:
        return _object_schema(rng, depth + 1, int(rng.integers(1, 4)))
    if r < 0.12:
        return {"type": "array", "items": _param_schema(rng, 3)}
    if r < 0.45:
        return {"type": "string", "enum": sorted({_ident(rng, 1, 2) for _ in range(int(rng.integers(2, 7)))})}
    if r < 0.80:
        return {"type": "string"}
    if r < 0.90:
        return {"type": "integer"}
    if r < 0.95:
        return {"type": "number"}
    return {"type": "boolean"}


def _object_schema(rng: np.random.Generator, depth: int, n_props: int) -> dict:
    props = {}
    while len(props) < n_props:
        props[_ident(rng)] = _param_schema(rng, depth)
    keys = list(props)
    n_req = int(rng.integers(1, len(keys) + 1))
    required = [k for k in keys if k in set(rng.choice(keys, size=n_req, replace=False).tolist())]
    return {"type": "object", "properties": props, "required": required}


def make_tools(rng: np.random.Generator, n_tools: int) -> dict:
    """{tool name: parameters schema} for n_tools invented tools."""
    tools = {}
    while len(tools) < n_tools:
        tools[_ident(rng, 2, 3)] = _object_schema(rng, 1, int(rng.integers(1, 7)))
    return tools


def _value(rng: np.random.Generator, schema: dict):
    t = schema.get("type")
    if "enum" in schema:
        return str(rng.choice(schema["enum"]))
    if t == "string":
        return " ".join(_word(rng) for _ in range(int(rng.integers(1, 6))))
    if t == "integer":
        return int(rng.integers(-50, 5000))
    if t == "number":
        return round(float(rng.uniform(-100, 1000)), int(rng.integers(1, 4)))
    if t == "boolean":
        return bool(rng.random() < 0.5)
    if t == "array":
        return [_value(rng, schema["items"]) for _ in range(int(rng.integers(1, 4)))]
    if t == "object":
        props = schema["properties"]
        keys = [k for k in props if k in schema["required"] or rng.random() < 0.5]
        rng.shuffle(keys)
        return {k: _value(rng, props[k]) for k in keys}
    raise ValueError(t)


def call_text(rng: np.random.Generator, tools: dict) -> str:
    """One call: an optional free-text preamble, then the JSON object."""
    name = str(rng.choice(list(tools)))
    text = ""
    if rng.random() < 0.4:
        words = [_word(rng) for _ in range(int(rng.integers(3, 12)))]
        text = " ".join(words).capitalize() + ".\n"
    call = {"name": name, "arguments": _value(rng, tools[name])}
    return text + json.dumps(call, separators=(", ", ": ")) + "\n"


# Punctuation pieces the tokenizer merges (longest first).
_PUNCT = sorted({'{"', '"}', '"}}', '":', '": ', '",', '["', '"]', ']}', '],', '},', '}}', ' "', ' {"', ' [',
                 ' {', ', ', '"', '{', '}', '[', ']', ',', ':', '.\n', '\n', '.', ' '}, key=len, reverse=True)
_TOKEN = re.compile("|".join([r" ?[A-Za-z]+", r"-?[0-9]+"] + [re.escape(p) for p in _PUNCT] + [r"."]), re.S)


def _pieces(word: str):
    """A word in sub-word pieces of 2-5 letters (the first keeps the leading
    space), fixed by a hash of the word, as a learned vocabulary would cut it."""
    core = word.lstrip(" ")
    lead = word[: len(word) - len(core)]
    h = zlib.crc32(core.encode())
    out, i = [], 0
    while i < len(core):
        n = 2 + (h % 4)
        h //= 4
        out.append(core[i:i + n])
        i += n
    if len(out) > 1 and len(out[-1]) == 1:
        last = out.pop()
        out[-1] += last
    out[0] = lead + out[0]
    return out


def tokenize(text: str):
    toks = []
    for m in _TOKEN.finditer(text):
        t = m.group(0)
        if t.strip(" ").isalpha():
            toks.extend(_pieces(t))
        elif t.lstrip("-").isdigit() and len(t) > 3:
            toks.extend(t[i:i + 3] for i in range(0, len(t), 3))
        else:
            toks.append(t)
    assert "".join(toks) == text
    return toks


def function_call_output(n_tokens: int, seed: int, n_tools: int = 4):
    """(tools, tokens): at least n_tokens tokens of back-to-back calls to a
    seeded set of tools."""
    rng = np.random.default_rng(seed)
    tools = make_tools(rng, n_tools)
    toks: list[str] = []
    while len(toks) < n_tokens:
        toks.extend(tokenize(call_text(rng, tools)))
    return tools, toks
