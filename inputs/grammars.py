"""The grammars of the five workloads, written with the builder in grammar.py.

* arithmetic: the textbook expression grammar with NUM and ignored spaces;
* json: objects, arrays, strings with escapes, numbers, literals, whitespace;
* schema-conformant JSON: generated from a seeded random schema (schema.py);
* python-like: statements and 14 precedence levels (pylike.py).
"""
from __future__ import annotations

from .grammar import Grammar, GrammarTables

# JSON lexical syntax on bytes: bytes >= 0x80 are allowed inside strings
# without UTF-8 validation; control bytes < 0x20 are not.
JSON_STRING = r'"([^"\\\x00-\x1f]|\\(["\\/bfnrt]|u[0-9a-fA-F]{4}))*"'
JSON_NUMBER = r"-?(0|[1-9][0-9]*)(\.[0-9]+)?([eE][+-]?[0-9]+)?"
JSON_WS = r"[ \t\n\r]+"


def arithmetic() -> GrammarTables:
    """E -> E+T | T, T -> T*F | F, F -> (E) | NUM; NUM = [0-9]+; spaces ignored."""
    g = Grammar("expr")
    g.regex("NUM", "[0-9]+")
    g.ignore("WS", " +")
    g.rule("expr", 'expr "+" term', "term")
    g.rule("term", 'term "*" factor', "factor")
    g.rule("factor", '"(" expr ")"', "NUM")
    return g.compile()


def json_grammar() -> GrammarTables:
    """Generic JSON (RFC 8259 shapes) over bytes."""
    g = Grammar("value")
    g.regex("STRING", JSON_STRING)
    g.regex("NUMBER", JSON_NUMBER)
    g.ignore("WS", JSON_WS)
    g.rule("value", "object", "array", "STRING", "NUMBER", '"true"', '"false"', '"null"')
    g.rule("object", '"{" "}"', '"{" members "}"')
    g.rule("members", "pair", 'members "," pair')
    g.rule("pair", 'STRING ":" value')
    g.rule("array", '"[" "]"', '"[" elements "]"')
    g.rule("elements", "value", 'elements "," value')
    return g.compile()
