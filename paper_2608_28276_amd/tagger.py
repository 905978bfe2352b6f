"""Structural tags of generated tokens from parser transitions (Section 3.2).

A constrained decoder keeps a parser state s_t and, once token y_t is
accepted, knows the transition s_{t-1} -> s_t before the token's KV is
persisted (Section 3.1).  PASK reads that transition as a structural tag
z_t = (class_t, role_t, state_t, next_t) (Eq. 3) and combines it with the
layer group to look up the persistence action; Crit(s_t) (critical or
lookahead-critical, Alg. 2 and Section 3.4) gates the controller's
promotions.  This module is that front end for function-call output: a
pushdown automaton over the characters of the output that follows a set of
tool schemas (a JSON-schema subset), fed token by token.

Grammar accepted (the output of a tool-calling model):
    output   := (text call)*          text: free text without '{'
    call     := {"name": <tool name>, "arguments": <object of the tool's
                 parameters>}  ("name" first; the name selects the schema)
Parameters: string, string enum, integer, number, boolean, object (nested
properties, required keys), array (items of one schema).  Objects accept
each property at most once, in any order, and close only when every
required key is present.  Whitespace between JSON tokens is free.

The four components of z_t, for the token just accepted:
  class  the broad type of the token's characters, by priority string >
         number > literal > text > punctuation > quote > space (a token
         like `"city` is string content, `":` is punctuation);
  role   the schema responsibility of the element those characters belong
         to: template key ("name", "arguments"), function name, required or
         optional parameter key, enum value, free argument value, structure;
  state  the parser's position after the token (LEX below);
  next   whether the frontier, after the token, must next produce a
         critical element: a key (the open object still lacks a required
         key, or the next value is an object that does) or an enum value
         (the next value is an enum or the function name).
The parser state s_t given to the online controller is (state, next) as one
id, STATE_ID = lex * 3 + next; Crit(s_t) holds inside a parameter key or an
enum value / function name, and wherever next is a key or an enum value.

The map from z_t to the six decode tag ids of the policy table
(TAG_NAMES) is tag_of() below.
"""

from __future__ import annotations

from dataclasses import dataclass

# -- components of z_t -------------------------------------------------------
CLASSES = ("text", "punct", "quote", "string", "number", "literal", "space")
C_TEXT, C_PUNCT, C_QUOTE, C_STRING, C_NUMBER, C_LITERAL, C_SPACE = range(7)
ROLES = ("none", "template", "function_name", "required_key", "optional_key", "enum", "argument", "structure")
R_NONE, R_TEMPLATE, R_FNAME, R_REQ_KEY, R_OPT_KEY, R_ENUM, R_ARG, R_STRUCT = range(8)
LEX = ("text", "expect_key", "in_template_key", "in_key", "expect_colon", "expect_value", "in_enum",
       "in_string", "in_number", "in_literal", "after_value", "end")
(S_TEXT, S_EXPECT_KEY, S_IN_TEMPLATE, S_IN_KEY, S_EXPECT_COLON, S_EXPECT_VALUE, S_IN_ENUM, S_IN_STRING,
 S_IN_NUMBER, S_IN_LITERAL, S_AFTER_VALUE, S_END) = range(12)
NEXTS = ("none", "key", "enum")
N_NONE, N_KEY, N_ENUM = range(3)

N_STATES = len(LEX) * len(NEXTS)
# Class priority when one token spans several kinds of characters.
_PRIORITY = (C_STRING, C_NUMBER, C_LITERAL, C_TEXT, C_PUNCT, C_QUOTE, C_SPACE)

# -- decode tags (the policy table's rows) ------------------------------------
TAG_NAMES = ("required_key", "enum_value", "arg_value", "boundary", "scaffold", "free_text")
T_KEY, T_ENUM, T_ARG, T_BOUNDARY, T_SCAFFOLD, T_FREE = range(6)


def state_id(lex: int, nxt: int) -> int:
    return lex * len(NEXTS) + nxt


def crit(state: int) -> bool:
    """Crit(s): inside a parameter key or an enum value (function names are
    an enum over the tools), or the frontier must produce one next."""
    lex, nxt = divmod(state, len(NEXTS))
    return lex in (S_IN_KEY, S_IN_ENUM) or nxt != N_NONE


CRITICAL_STATES = tuple(s for s in range(N_STATES) if crit(s))


def tag_of(cls: int, role: int) -> int:
    """Decode tag id of a structural tag: parameter-key content ->
    required_key; function-name or enum content -> enum_value; free argument
    content -> arg_value; JSON punctuation -> boundary; quotes, spaces and
    the call template's keys -> scaffold; text outside calls -> free_text.
    (state and next reach the table through the controller's state id.)"""
    if cls == C_TEXT:
        return T_FREE
    if cls == C_PUNCT:
        return T_BOUNDARY
    if cls in (C_STRING, C_NUMBER, C_LITERAL):
        if role in (R_REQ_KEY, R_OPT_KEY):
            return T_KEY
        if role in (R_FNAME, R_ENUM):
            return T_ENUM
        if role == R_ARG:
            return T_ARG
    return T_SCAFFOLD


class GrammarError(ValueError):
    """The output left the language of the tool schemas."""


@dataclass
class Tag:
    cls: int
    role: int
    lex: int
    next: int

    @property
    def state(self) -> int:
        return state_id(self.lex, self.next)

    @property
    def tag(self) -> int:
        return tag_of(self.cls, self.role)

    def names(self):
        return CLASSES[self.cls], ROLES[self.role], LEX[self.lex], NEXTS[self.next]


# -- the pushdown automaton ----------------------------------------------------
_CALL = {"kind": "call"}     # schema marker of the call wrapper object


class _Frame:
    """An open object or array: its schema, the keys seen, the current key."""

    def __init__(self, schema, kind):
        self.schema, self.kind = schema, kind
        self.seen: set = set()
        self.key = None              # key whose value comes next (objects)
        self.count = 0               # values so far (arrays)


def _is_enum(schema) -> bool:
    return schema is not None and "enum" in schema


class CallParser:
    """Character-level pushdown automaton for the output grammar above.

    tools: {name: parameters schema (type object)}.  feed(token) consumes the
    token's characters, raises GrammarError when one is not legal, and
    returns its Tag."""

    def __init__(self, tools: dict):
        self.tools = tools
        self.lex = S_TEXT
        self.stack: list[_Frame] = []
        self.buf = ""                # characters of the open string / number / literal
        self.value_schema = None     # schema of the value being read (or expected)
        self.escape = False

    # -- schema lookups ------------------------------------------------------
    def _role_of_value(self, schema) -> int:
        if schema is _FNAME:
            return R_FNAME
        return R_ENUM if _is_enum(schema) else R_ARG

    def _expected_schema(self):
        """Schema of the value the frontier expects next (after ':' in an
        object, or after '[' / ',' in an array)."""
        top = self.stack[-1]
        if top.kind == "array":
            return top.schema.get("items", {})
        if top.schema is _CALL:
            return _FNAME if top.key == "name" else self._args_schema(top)
        return top.schema.get("properties", {}).get(top.key, {})

    def _args_schema(self, top):
        return self.tools[top.fname]

    def _missing_required(self, top) -> bool:
        if top.kind != "object":
            return False
        if top.schema is _CALL:
            return len(top.seen) < 2
        return bool(set(top.schema.get("required", ())) - top.seen)

    def _next_of(self) -> int:
        """next_t: what the frontier must produce next, if it is critical."""
        if self.lex in (S_EXPECT_KEY, S_AFTER_VALUE):
            top = self.stack[-1] if self.stack else None
            if top is not None and top.kind == "object" and top.schema is not _CALL and self._missing_required(top):
                return N_KEY
            return N_NONE
        if self.lex in (S_EXPECT_COLON, S_EXPECT_VALUE):
            sch = self._expected_schema()
            if sch is _FNAME or _is_enum(sch):
                return N_ENUM
            if sch.get("type") == "object" and sch.get("required"):
                return N_KEY
            return N_NONE
        return N_NONE

    # -- transitions ----------------------------------------------------------
    def _open_value(self, ch) -> tuple:
        """First character of a value in S_EXPECT_VALUE: (class, role)."""
        sch = self._expected_schema()
        self.value_schema = sch
        if ch == '"':
            if sch is _FNAME or _is_enum(sch) or sch.get("type") == "string":
                self.lex = S_IN_ENUM if (sch is _FNAME or _is_enum(sch)) else S_IN_STRING
                self.buf = ""
                return C_QUOTE, self._role_of_value(sch)
            raise GrammarError(f"string where the schema wants {sch.get('type')}")
        if ch == "{":
            if sch is _FNAME or sch.get("type") != "object":
                raise GrammarError("object not allowed here")
            self.stack.append(_Frame(sch, "object"))
            self.lex = S_EXPECT_KEY
            return C_PUNCT, R_STRUCT
        if ch == "[":
            if sch is _FNAME or sch.get("type") != "array":
                raise GrammarError("array not allowed here")
            self.stack.append(_Frame(sch, "array"))
            self.lex = S_EXPECT_VALUE
            return C_PUNCT, R_STRUCT
        if ch in "-0123456789":
            if sch is _FNAME or sch.get("type") not in ("integer", "number"):
                raise GrammarError("number not allowed here")
            self.lex, self.buf = S_IN_NUMBER, ch
            return C_NUMBER, R_ARG
        if ch in "tfn":
            if sch is _FNAME or sch.get("type") not in ("boolean",):
                raise GrammarError("literal not allowed here")
            self.lex, self.buf = S_IN_LITERAL, ch
            return C_LITERAL, R_ARG
        raise GrammarError(f"{ch!r} cannot start a value")

    def _close_value(self):
        """A scalar or container value is complete: back to its parent."""
        top = self.stack[-1] if self.stack else None
        if top is None:
            self.lex = S_END
            return
        if top.kind == "array":
            top.count += 1
        self.lex = S_AFTER_VALUE

    def _finish_key(self):
        top = self.stack[-1]
        key = self.buf
        if top.schema is _CALL:
            want = "name" if not top.seen else "arguments"
            if key != want or key in top.seen:
                raise GrammarError(f"call wrapper wants key {want!r}, got {key!r}")
        elif key not in top.schema.get("properties", {}) or key in top.seen:
            raise GrammarError(f"key {key!r} not allowed here")
        top.seen.add(key)
        top.key = key
        self.lex = S_EXPECT_COLON

    def _finish_string(self):
        sch = self.value_schema
        top = self.stack[-1]
        if sch is _FNAME:
            if self.buf not in self.tools:
                raise GrammarError(f"unknown tool {self.buf!r}")
            top.fname = self.buf
        elif _is_enum(sch) and self.buf not in sch["enum"]:
            raise GrammarError(f"{self.buf!r} is not one of the enum values")
        self._close_value()

    def _step(self, ch) -> tuple:
        """Consume one character; returns its (class, role)."""
        lex = self.lex
        if lex in (S_TEXT, S_END):
            if ch == "{":
                call = _Frame(_CALL, "object")
                call.fname = None
                self.stack = [call]
                self.lex = S_EXPECT_KEY
                return C_PUNCT, R_STRUCT
            self.lex = S_TEXT
            return (C_SPACE if ch.isspace() else C_TEXT), R_NONE
        if lex in (S_IN_KEY, S_IN_TEMPLATE, S_IN_ENUM, S_IN_STRING):
            role = (R_TEMPLATE if lex == S_IN_TEMPLATE else self._key_role() if lex == S_IN_KEY
                    else self._role_of_value(self.value_schema))
            if self.escape:
                self.escape = False
                self.buf += ch
                return C_STRING, role
            if ch == "\\":
                self.escape = True
                return C_STRING, role
            if ch == '"':
                if lex in (S_IN_KEY, S_IN_TEMPLATE):
                    self._finish_key()
                else:
                    self._finish_string()
                return C_QUOTE, role
            self.buf += ch
            return C_STRING, role
        if lex == S_IN_NUMBER:
            if ch in "0123456789." or (ch in "eE+-" and self.buf and self.buf[-1] in "eE"):
                self.buf += ch
                return C_NUMBER, R_ARG
            self._check_number()
            self._close_value()
            return self._step(ch)
        if lex == S_IN_LITERAL:
            for word in ("true", "false", "null"):
                if word.startswith(self.buf + ch):
                    self.buf += ch
                    if self.buf == word:
                        if word == "null":
                            raise GrammarError("null is not a parameter value here")
                        self._close_value()
                    return C_LITERAL, R_ARG
            raise GrammarError(f"bad literal {self.buf + ch!r}")
        if ch.isspace():
            return C_SPACE, R_NONE
        top = self.stack[-1]
        if lex == S_EXPECT_KEY:
            if ch == '"':
                self.buf = ""
                self.lex = S_IN_TEMPLATE if top.schema is _CALL else S_IN_KEY
                return C_QUOTE, (R_TEMPLATE if top.schema is _CALL else R_NONE)
            if ch == "}" and not top.seen:
                return self._close_container(top)
            raise GrammarError(f"{ch!r} where a key is expected")
        if lex == S_EXPECT_COLON:
            if ch == ":":
                self.lex = S_EXPECT_VALUE
                return C_PUNCT, R_STRUCT
            raise GrammarError("':' expected")
        if lex == S_EXPECT_VALUE:
            if ch == "]" and top.kind == "array" and top.count == 0:
                return self._close_container(top)
            return self._open_value(ch)
        if lex == S_AFTER_VALUE:
            if ch == ",":
                self.lex = S_EXPECT_KEY if top.kind == "object" else S_EXPECT_VALUE
                return C_PUNCT, R_STRUCT
            if ch in "}]":
                return self._close_container(top, ch)
            raise GrammarError(f"{ch!r} after a value")
        raise GrammarError(f"unexpected {ch!r}")

    def _key_role(self) -> int:
        top = self.stack[-1]
        return R_REQ_KEY if self._key_required(top) else R_OPT_KEY

    def _key_required(self, top) -> bool:
        """Whether the key being read (self.buf so far) can only be a required
        key: every property of the object that extends the prefix read so far
        is required (decided by the grammar alone, character by character)."""
        props = top.schema.get("properties", {})
        req = set(top.schema.get("required", ()))
        cands = [k for k in props if k.startswith(self.buf) and k not in top.seen]
        return bool(cands) and all(k in req for k in cands)

    def _close_container(self, top, ch="}"):
        want = "}" if top.kind == "object" else "]"
        if ch != want:
            raise GrammarError(f"{ch!r} closes a {top.kind}")
        if self._missing_required(top):
            raise GrammarError("object closed before its required keys")
        self.stack.pop()
        self._close_value()
        return C_PUNCT, R_STRUCT

    def _check_number(self):
        s = self.buf
        try:
            float(s)
        except ValueError:
            raise GrammarError(f"bad number {s!r}") from None
        if self.value_schema.get("type") == "integer" and not s.lstrip("-").isdigit():
            raise GrammarError(f"{s!r} is not an integer")

    # -- tokens ------------------------------------------------------------------
    def feed(self, token: str) -> Tag:
        """Accept one token: the transition s_{t-1} -> s_t over its characters
        and the structural tag z_t it yields."""
        if not token:
            raise GrammarError("empty token")
        seen = {}
        for ch in token:
            cls, role = self._step(ch)
            seen[cls] = role         # the last character of a class knows the most (key prefixes)
        cls = next(c for c in _PRIORITY if c in seen)
        return Tag(cls, seen[cls], self.lex, self._next_of())

    def finished(self) -> bool:
        """True between calls (every call closed)."""
        return not self.stack


class _FnameMarker(dict):
    """Schema marker of the call wrapper's "name" value: an enum over tools."""


_FNAME = _FnameMarker()


def tag_stream(tools: dict, tokens):
    """Tags (decode tag ids) and parser-state ids of an accepted token stream."""
    p = CallParser(tools)
    tags, states = [], []
    for tok in tokens:
        z = p.feed(tok)
        tags.append(z.tag)
        states.append(z.state)
    return tags, states
