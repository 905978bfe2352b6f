"""The structural tagger (Section 3.2, Eq. 3; Crit of Alg. 2): a pushdown
automaton over tool-call output that gives every accepted token its
z_t = (class, role, state, next), decode tag and parser state.

Pinned by hand: the expected rows below were derived token by token from the
definitions (class priority string > number > literal > text > punct > quote
> space; the role of the element the dominant characters belong to; the
parser position after the token; what the frontier must produce next), not
read off the program."""

import json

import numpy as np
import pytest

from paper_2608_28276_amd import tagger as tg
from workload.calls import function_call_output, make_tools, tokenize

FORECAST = {"get_forecast": {"type": "object", "properties": {
    "city": {"type": "string"}, "unit": {"type": "string", "enum": ["metric", "imperial"]},
    "days": {"type": "integer"}}, "required": ["city", "unit"]}}

# token, class, role, parser position after it, next, decode tag, Crit(s)
FORECAST_ROWS = [
    ("Let", "text", "none", "text", "none", "free_text", False),
    (" me", "text", "none", "text", "none", "free_text", False),
    (" check", "text", "none", "text", "none", "free_text", False),
    (".", "text", "none", "text", "none", "free_text", False),
    ("\n", "space", "none", "text", "none", "scaffold", False),
    ('{"', "punct", "structure", "in_template_key", "none", "boundary", False),
    ("name", "string", "template", "in_template_key", "none", "scaffold", False),
    ('":', "punct", "structure", "expect_value", "enum", "boundary", True),        # the function name comes next
    (' "', "quote", "function_name", "in_enum", "none", "scaffold", True),
    ("get", "string", "function_name", "in_enum", "none", "enum_value", True),
    ("_fore", "string", "function_name", "in_enum", "none", "enum_value", True),
    ("cast", "string", "function_name", "in_enum", "none", "enum_value", True),
    ('",', "punct", "structure", "expect_key", "none", "boundary", False),
    (' "', "quote", "template", "in_template_key", "none", "scaffold", False),
    ("arguments", "string", "template", "in_template_key", "none", "scaffold", False),
    ('":', "punct", "structure", "expect_value", "key", "boundary", True),         # an object with required keys
    (' {"', "punct", "structure", "in_key", "none", "boundary", True),
    ("ci", "string", "required_key", "in_key", "none", "required_key", True),      # prefix "ci": only city
    ("ty", "string", "required_key", "in_key", "none", "required_key", True),
    ('":', "punct", "structure", "expect_value", "none", "boundary", False),       # a free string next
    (' "', "quote", "argument", "in_string", "none", "scaffold", False),
    ("Par", "string", "argument", "in_string", "none", "arg_value", False),
    ("is", "string", "argument", "in_string", "none", "arg_value", False),
    ('",', "punct", "structure", "expect_key", "key", "boundary", True),           # unit still missing
    (' "', "quote", "none", "in_key", "none", "scaffold", True),
    ("unit", "string", "required_key", "in_key", "none", "required_key", True),
    ('":', "punct", "structure", "expect_value", "enum", "boundary", True),
    (' "', "quote", "enum", "in_enum", "none", "scaffold", True),
    ("met", "string", "enum", "in_enum", "none", "enum_value", True),
    ("ric", "string", "enum", "in_enum", "none", "enum_value", True),
    ('",', "punct", "structure", "expect_key", "none", "boundary", False),         # every required key seen
    (' "', "quote", "none", "in_key", "none", "scaffold", True),
    ("days", "string", "optional_key", "in_key", "none", "required_key", True),
    ('":', "punct", "structure", "expect_value", "none", "boundary", False),
    (" ", "space", "none", "expect_value", "none", "scaffold", False),
    ("3", "number", "argument", "in_number", "none", "arg_value", False),
    ("}}", "punct", "structure", "end", "none", "boundary", False),
]

ALARM = {"set_alarm": {"type": "object", "properties": {
    "time": {"type": "string"},
    "tags": {"type": "array", "items": {"type": "string", "enum": ["work", "home"]}},
    "repeat": {"type": "boolean"},
    "target": {"type": "object", "properties": {"room": {"type": "string"}, "level": {"type": "integer"}},
               "required": ["room"]}},
    "required": ["time", "target"]}}

ALARM_ROWS = [
    ('{"', "punct", "structure", "in_template_key", "none", "boundary", False),
    ("name", "string", "template", "in_template_key", "none", "scaffold", False),
    ('": ', "punct", "structure", "expect_value", "enum", "boundary", True),
    ('"', "quote", "function_name", "in_enum", "none", "scaffold", True),
    ("set", "string", "function_name", "in_enum", "none", "enum_value", True),
    ("_alarm", "string", "function_name", "in_enum", "none", "enum_value", True),
    ('",', "punct", "structure", "expect_key", "none", "boundary", False),
    (' "', "quote", "template", "in_template_key", "none", "scaffold", False),
    ("arguments", "string", "template", "in_template_key", "none", "scaffold", False),
    ('": ', "punct", "structure", "expect_value", "key", "boundary", True),
    ('{"', "punct", "structure", "in_key", "none", "boundary", True),
    ("t", "string", "optional_key", "in_key", "none", "required_key", True),        # time, tags, target: not all required
    ("ags", "string", "optional_key", "in_key", "none", "required_key", True),      # tags
    ('": ', "punct", "structure", "expect_value", "none", "boundary", False),       # an array next
    ('["', "punct", "structure", "in_enum", "none", "boundary", True),              # enum items
    ("work", "string", "enum", "in_enum", "none", "enum_value", True),
    ('"]', "punct", "structure", "after_value", "key", "boundary", True),           # time and target missing
    (', "', "punct", "structure", "in_key", "none", "boundary", True),
    ("ta", "string", "required_key", "in_key", "none", "required_key", True),       # only target left with "ta"
    ("rget", "string", "required_key", "in_key", "none", "required_key", True),
    ('": ', "punct", "structure", "expect_value", "key", "boundary", True),         # object with a required key
    ('{"', "punct", "structure", "in_key", "none", "boundary", True),
    ("room", "string", "required_key", "in_key", "none", "required_key", True),
    ('": ', "punct", "structure", "expect_value", "none", "boundary", False),
    ('"', "quote", "argument", "in_string", "none", "scaffold", False),
    ("hall", "string", "argument", "in_string", "none", "arg_value", False),
    ('"}', "punct", "structure", "after_value", "key", "boundary", True),           # time still missing
    (', "', "punct", "structure", "in_key", "none", "boundary", True),
    ("time", "string", "required_key", "in_key", "none", "required_key", True),
    ('": "', "punct", "structure", "in_string", "none", "boundary", False),
    ("now", "string", "argument", "in_string", "none", "arg_value", False),
    ('",', "punct", "structure", "expect_key", "none", "boundary", False),
    (' "', "quote", "none", "in_key", "none", "scaffold", True),
    ("repeat", "string", "optional_key", "in_key", "none", "required_key", True),
    ('": ', "punct", "structure", "expect_value", "none", "boundary", False),
    ("true", "literal", "argument", "after_value", "none", "arg_value", False),
    ("}}", "punct", "structure", "end", "none", "boundary", False),
    ("\n", "space", "none", "text", "none", "scaffold", False),
]


@pytest.mark.parametrize("tools,rows", [(FORECAST, FORECAST_ROWS), (ALARM, ALARM_ROWS)], ids=["forecast", "alarm"])
def test_hand_derived_tags(tools, rows):
    p = tg.CallParser(tools)
    for i, (tok, cls, role, lex, nxt, tag, is_crit) in enumerate(rows):
        z = p.feed(tok)
        assert z.names() == (cls, role, lex, nxt), (i, tok, z.names())
        assert tg.TAG_NAMES[z.tag] == tag, (i, tok)
        assert tg.crit(z.state) == is_crit, (i, tok)
        assert z.state == tg.LEX.index(lex) * 3 + tg.NEXTS.index(nxt)
    assert p.finished()


def test_text_equals_tokens_and_is_valid_json():
    """The hand examples are the JSON the rows describe."""
    text = "".join(r[0] for r in ALARM_ROWS)
    obj = json.loads(text)
    assert obj["name"] == "set_alarm" and obj["arguments"]["target"] == {"room": "hall"}
    assert json.loads("".join(r[0] for r in FORECAST_ROWS)[len("Let me check.\n"):])["arguments"]["days"] == 3


@pytest.mark.parametrize("text", [
    '{"name": "nope", "arguments": {}}',                                   # unknown tool
    '{"arguments": {}, "name": "get_forecast"}',                           # name must come first
    '{"name": "get_forecast", "arguments": {"city": "x"}}',                # unit missing at close
    '{"name": "get_forecast", "arguments": {"city": "x", "unit": "kelvin"}}',   # not an enum value
    '{"name": "get_forecast", "arguments": {"city": 3, "unit": "metric"}}',      # number for a string
    '{"name": "get_forecast", "arguments": {"city": "x", "city": "y", "unit": "metric"}}',   # duplicate key
    '{"name": "get_forecast", "arguments": {"town": "x"}}',                # key not in the schema
    '{"name": "get_forecast", "arguments": {"city": "x", "unit": "metric", "days": 2.5}}',  # not an integer
    '{"name": "get_forecast", "arguments": {"city": "x", "unit": "metric",}}',   # trailing comma
    '{"name": "get_forecast", "arguments": {"city": "x", "unit": "metric", "days": tru}}',  # bad literal
])
def test_rejects_output_outside_the_grammar(text):
    p = tg.CallParser(FORECAST)
    with pytest.raises(tg.GrammarError):
        for ch in text:
            p.feed(ch)
        assert p.finished()


def test_state_after_a_token_does_not_depend_on_segmentation():
    """Characters one at a time or the tokenizer's pieces: the parser ends every
    token in the same position, with the same frontier."""
    tools, toks = function_call_output(3000, 5)
    a, b = tg.CallParser(tools), tg.CallParser(tools)
    for tok in toks:
        za = a.feed(tok)
        for ch in tok:
            zb = b.feed(ch)
        assert (za.lex, za.next) == (zb.lex, zb.next)
        assert len(a.stack) == len(b.stack)


def test_generated_calls_are_schema_valid():
    """Every generated call is JSON that the parser accepts for its tool set,
    and every tag and state is in range."""
    tools, toks = function_call_output(20000, 11)
    text = "".join(toks)
    calls = [line for line in text.split("\n") if line.startswith("{")]
    assert len(calls) > 50
    for line in calls:
        obj = json.loads(line)
        assert obj["name"] in tools
    tags, states = tg.tag_stream(tools, toks)
    assert max(tags) < 6 and max(states) < tg.N_STATES <= 64
    assert tokenize(text) == toks


def test_crit_states():
    for s in range(tg.N_STATES):
        lex, nxt = divmod(s, 3)
        assert tg.crit(s) == (tg.LEX[lex] in ("in_key", "in_enum") or tg.NEXTS[nxt] != "none")
    assert set(tg.CRITICAL_STATES) == {s for s in range(tg.N_STATES) if tg.crit(s)}


def test_tools_are_seeded():
    a = make_tools(np.random.default_rng(3), 4)
    assert a == make_tools(np.random.default_rng(3), 4) and len(a) == 4
