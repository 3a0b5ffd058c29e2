"""The core of the Python-like grammar, its programs and vocabularies: the
stress workload's language (deep nesting at a 262,144-token vocabulary).

The full grammar (`pylike.py`, 143 nonterminals) adds match statements,
comprehensions, async, decorators, type parameters and more; at this
vocabulary its classifier construction takes too long for a test session, so
this workload keeps the core (88 terminals, 80 nonterminals, 382 LR states).
Its documents, vocabulary and seeds are unchanged from when it was the only
Python-like grammar.

Grammar: def/class/if/elif/else/while/for/try/with/return/... statements;
blocks are NEWLINE INDENT stmts DEDENT, with INDENT and DEDENT spelled as the
reserved bytes 0x0E and 0x0F (a non-contextual lexer cannot count columns);
spaces, tabs and comments are ignored.  Expressions have a conditional
expression, lambda, 14 stratified binary-operator levels (left-recursive,
power right-recursive), unary operators, calls, subscripts/slices,
attributes and list/dict/tuple literals.  The grammar is LALR(1) as written.
"""
from __future__ import annotations

import functools

import numpy as np

from .grammar import Grammar, GrammarTables
from .vocab import Vocab, piece_vocab

INDENT = "\x0e"
DEDENT = "\x0f"

KEYWORDS = ["def", "class", "if", "elif", "else", "while", "for", "in", "return", "pass", "break",
            "continue", "lambda", "and", "or", "not", "is", "None", "True", "False", "import", "from",
            "as", "global", "try", "except", "finally", "raise", "assert", "del", "with", "yield"]

# the 14 binary levels, lowest precedence first
BINARY_LEVELS = [
    ["|>"],                 # pipe
    ["??"],                 # coalesce
    ["or"],
    ["and"],
    ["==", "!="],
    ["<", ">", "<=", ">=", "in", "is"],
    ["|"],
    ["^"],
    ["&"],
    ["<<", ">>"],
    [".."],                 # range
    ["+", "-"],
    ["*", "/", "//", "%", "@"],
    ["**"],                 # power (right-associative)
]
AUGASSIGN = ["+=", "-=", "*=", "/=", "//=", "%=", "&=", "|=", "^=", "<<=", ">>=", "**="]


def pylike_grammar() -> GrammarTables:
    g = Grammar("file")
    g.regex("NAME", r"[A-Za-z_][A-Za-z0-9_]*")
    g.regex("NUMBER", r"[0-9]+(\.[0-9]+)?([eE][+-]?[0-9]+)?|0[xX][0-9a-fA-F]+")
    g.regex("STRING", r'"([^"\\\n]|\\.)*"' + "|" + r"'([^'\\\n]|\\.)*'")
    g.ignore("WS", r"[ \t]+")
    g.ignore("COMMENT", r"#[^\n\x0e\x0f]*")
    for k in KEYWORDS:
        g.literal(k)
    NL, IND, DED = g.literal("\n"), g.literal(INDENT), g.literal(DEDENT)

    # ---- file and statements
    g.rule("file", [], ["file", "line"])
    g.rule("line", [NL], ["stmt"])
    g.rule("stmts", ["stmt"], ["stmts", "stmt"], ["stmts", NL])
    g.rule("suite", [NL, IND, "stmts", DED])
    g.rule("stmt", ["simple_stmt"], ["compound_stmt"])
    g.rule("simple_stmt", ["small_stmts", NL], ["small_stmts", '";"', NL])
    g.rule("small_stmts", ["small_stmt"], ["small_stmts", '";"', "small_stmt"])
    g.rule("small_stmt", ["expr_stmt"], ["return_stmt"], ['"pass"'], ['"break"'], ['"continue"'],
           ["global_stmt"], ["del_stmt"], ["import_stmt"], ["assert_stmt"], ["raise_stmt"],
           ["yield_stmt"])
    g.rule("expr_stmt", ["testlist"], ["testlist", '"="', "assign_rhs"], ["testlist", "augassign", "testlist"])
    g.rule("assign_rhs", ["testlist"], ["testlist", '"="', "assign_rhs"])
    g.rule("augassign", *[[f'"{op}"'] for op in AUGASSIGN])
    g.rule("return_stmt", ['"return"'], ['"return"', "testlist"])
    g.rule("yield_stmt", ['"yield"'], ['"yield"', "testlist"])
    g.rule("global_stmt", ['"global"', "names"])
    g.rule("names", ["NAME"], ["names", '","', "NAME"])
    g.rule("del_stmt", ['"del"', "testlist"])
    g.rule("import_stmt", ['"import"', "dotted_as_names"],
           ['"from"', "dotted_name", '"import"', "import_targets"])
    g.rule("import_targets", ['"*"'], ["import_as_names"], ['"("', "import_as_names", '")"'])
    g.rule("import_as_names", ["import_as_name"], ["import_as_names", '","', "import_as_name"])
    g.rule("import_as_name", ["NAME"], ["NAME", '"as"', "NAME"])
    g.rule("dotted_as_names", ["dotted_as_name"], ["dotted_as_names", '","', "dotted_as_name"])
    g.rule("dotted_as_name", ["dotted_name"], ["dotted_name", '"as"', "NAME"])
    g.rule("dotted_name", ["NAME"], ["dotted_name", '"."', "NAME"])
    g.rule("assert_stmt", ['"assert"', "test"], ['"assert"', "test", '","', "test"])
    g.rule("raise_stmt", ['"raise"'], ['"raise"', "test"], ['"raise"', "test", '"from"', "test"])

    g.rule("compound_stmt", ["if_stmt"], ["while_stmt"], ["for_stmt"], ["funcdef"], ["classdef"],
           ["try_stmt"], ["with_stmt"])
    g.rule("if_stmt", ['"if"', "test", '":"', "suite", "elifs", "else_opt"])
    g.rule("elifs", [], ["elifs", '"elif"', "test", '":"', "suite"])
    g.rule("else_opt", [], ['"else"', '":"', "suite"])
    g.rule("while_stmt", ['"while"', "test", '":"', "suite", "else_opt"])
    g.rule("for_stmt", ['"for"', "targets", '"in"', "testlist", '":"', "suite", "else_opt"])
    g.rule("targets", ["target"], ["targets", '","', "target"])
    g.rule("target", ["NAME"], ['"("', "targets", '")"'], ['"["', "targets", '"]"'])
    g.rule("funcdef", ["decorators_opt", '"def"', "NAME", '"("', "params_opt", '")"', "returns_opt", '":"', "suite"])
    g.rule("decorators_opt", [], ["decorators_opt", '"@"', "dotted_name", NL],
           ["decorators_opt", '"@"', "dotted_name", '"("', "args_opt", '")"', NL])
    g.rule("returns_opt", [], ['"->"', "test"])
    g.rule("params_opt", [], ["params"], ["params", '","'])
    g.rule("params", ["param"], ["params", '","', "param"])
    g.rule("param", ["NAME"], ["NAME", '":"', "test"], ["NAME", '"="', "test"],
           ["NAME", '":"', "test", '"="', "test"], ['"*"', "NAME"], ['"**"', "NAME"])
    g.rule("classdef", ['"class"', "NAME", '":"', "suite"], ['"class"', "NAME", '"("', "args_opt", '")"', '":"', "suite"])
    g.rule("try_stmt", ['"try"', '":"', "suite", "excepts", "else_opt", "finally_opt"],
           ['"try"', '":"', "suite", '"finally"', '":"', "suite"])
    g.rule("excepts", ["except_clause"], ["excepts", "except_clause"])
    g.rule("except_clause", ['"except"', '":"', "suite"], ['"except"', "test", '":"', "suite"],
           ['"except"', "test", '"as"', "NAME", '":"', "suite"])
    g.rule("finally_opt", [], ['"finally"', '":"', "suite"])
    g.rule("with_stmt", ['"with"', "with_items", '":"', "suite"])
    g.rule("with_items", ["with_item"], ["with_items", '","', "with_item"])
    g.rule("with_item", ["test"], ["test", '"as"', "target"])

    # ---- expressions
    g.rule("testlist", ["test"], ["test", '","'], ["test", '","', "testlist_tail"])
    g.rule("testlist_tail", ["test"], ["test", '","'], ["test", '","', "testlist_tail"])
    g.rule("test", ["lvl0"], ["lvl0", '"if"', "lvl0", '"else"', "test"], ["lambdef"])
    g.rule("lambdef", ['"lambda"', '":"', "test"], ['"lambda"', "names", '":"', "test"])
    n = len(BINARY_LEVELS)
    for i, ops in enumerate(BINARY_LEVELS[:-1]):
        nxt = f"lvl{i + 1}" if i + 1 < n - 1 else "unary"
        if ops == ["or"] or ops == ["and"]:
            # boolean levels take "not" operands
            pass
        if i == 3:      # after "and": the "not" level
            nxt = "notexpr"
            g.rule("notexpr", ['"not"', "notexpr"], ["lvl4"])
        alts = [[nxt]] + [[f"lvl{i}", f'"{op}"', nxt] for op in ops]
        if ops == ["<", ">", "<=", ">=", "in", "is"]:
            alts += [[f"lvl{i}", '"not"', '"in"', nxt], [f"lvl{i}", '"is"', '"not"', nxt]]
        g.rule(f"lvl{i}", *alts)
    g.rule("unary", ['"-"', "unary"], ['"+"', "unary"], ['"~"', "unary"], ["power"])
    g.rule("power", ["primary"], ["primary", '"**"', "unary"])
    g.rule("primary", ["atom"], ["primary", '"("', "args_opt", '")"'], ["primary", '"["', "subscripts", '"]"'],
           ["primary", '"."', "NAME"])
    g.rule("args_opt", [], ["args"], ["args", '","'])
    g.rule("args", ["arg"], ["args", '","', "arg"])
    g.rule("arg", ["test"], ["test", '"="', "test"], ['"*"', "test"], ['"**"', "test"])
    g.rule("subscripts", ["subscript"], ["subscripts", '","', "subscript"])
    g.rule("subscript", ["test"], ["slice"])
    g.rule("slice", ['":"'], ["test", '":"'], ['":"', "test"], ["test", '":"', "test"],
           ['":"', "test", '":"', "test"], ["test", '":"', "test", '":"', "test"])
    g.rule("atom", ["NAME"], ["NUMBER"], ["strings"], ['"None"'], ['"True"'], ['"False"'],
           ['"("', '")"'], ['"("', "testlist", '")"'],
           ['"["', '"]"'], ['"["', "items", '"]"'], ['"["', "test", '"for"', "targets", '"in"', "lvl2", '"]"'],
           ['"{"', '"}"'], ['"{"', "dict_items", '"}"'])
    g.rule("strings", ["STRING"], ["strings", "STRING"])
    g.rule("items", ["test"], ["items", '","', "test"], ["items", '","'])
    g.rule("dict_items", ["dict_item"], ["dict_items", '","', "dict_item"], ["dict_items", '","'])
    g.rule("dict_item", ["test", '":"', "test"], ['"**"', "test"])
    return g.compile()


# ----------------------------------------------------------------- programs

_NAMES = ["x", "y", "i", "j", "n", "data", "value", "result", "items", "key", "node", "self", "count",
          "total", "buf", "line", "path", "obj", "cfg", "fn", "acc", "left", "right", "idx", "tmp"]
_BIN_OPS = [op for lvl in BINARY_LEVELS for op in lvl] + ["not in", "is not"]


class ProgramGen:
    """Random programs; `depth_budget` bounds statement and expression nesting."""

    def __init__(self, rng: np.random.Generator, expr_depth: int = 4, block_depth: int = 4):
        self.r = rng
        self.expr_depth = expr_depth
        self.block_depth = block_depth
        self.out: list[str] = []

    def name(self) -> str:
        r = self.r
        if r.random() < 0.2:
            return _NAMES[int(r.integers(len(_NAMES)))] + str(int(r.integers(0, 100)))
        return _NAMES[int(r.integers(len(_NAMES)))]

    def atom(self, d: int) -> str:
        r = self.r
        k = r.random()
        if k < 0.35 or d <= 0:
            return self.name() if r.random() < 0.7 else str(int(r.integers(0, 1000)))
        if k < 0.45:
            return '"' + "".join("abcdefgh "[int(c)] for c in r.integers(0, 9, size=int(r.integers(0, 8)))) + '"'
        if k < 0.6:
            return "(" + self.expr(d - 1) + ")"
        if k < 0.7:
            return "[" + ", ".join(self.expr(d - 1) for _ in range(int(r.integers(0, 4)))) + "]"
        if k < 0.78:
            return "{" + ", ".join(self.expr(d - 1) + ": " + self.expr(d - 1) for _ in range(int(r.integers(0, 3)))) + "}"
        if k < 0.92:
            return self.name() + "(" + ", ".join(self.expr(d - 1) for _ in range(int(r.integers(0, 4)))) + ")"
        if k < 0.97:
            return self.name() + "[" + self.expr(d - 1) + "]"
        return self.name() + "." + self.name()

    def expr(self, d: int | None = None) -> str:
        r = self.r
        d = self.expr_depth if d is None else d
        s = self.atom(d)
        for _ in range(int(r.integers(0, 3)) if d > 0 else 0):
            op = _BIN_OPS[int(r.integers(len(_BIN_OPS)))]
            s = s + " " + op + " " + self.atom(d - 1)
        if d > 0 and r.random() < 0.05:
            s = s + " if " + self.atom(d - 1) + " else " + self.atom(d - 1)
        if d > 0 and r.random() < 0.05:
            s = "not " + s
        return s

    def simple(self) -> str:
        r = self.r
        k = r.random()
        if k < 0.45:
            return self.name() + " = " + self.expr()
        if k < 0.55:
            return self.name() + " += " + self.expr()
        if k < 0.7:
            return self.expr()
        if k < 0.8:
            return "return " + self.expr()
        return ["pass", "break", "continue", "global " + self.name(), "import os", "assert " + self.expr(),
                "raise " + self.name() + "()", "del " + self.name()][int(r.integers(8))]

    def block(self, level: int):
        r = self.r
        self.out.append(":\n" + INDENT)
        n = int(r.integers(1, 4))
        for _ in range(n):
            self.stmt(level + 1)
        self.out.append(DEDENT)

    def stmt(self, level: int):
        r = self.r
        k = r.random()
        if level >= self.block_depth or k < 0.55:
            self.out.append(self.simple() + "\n")
            return
        if k < 0.65:
            self.out.append("if " + self.expr())
            self.block(level)
            if r.random() < 0.3:
                self.out.append("else")
                self.block(level)
        elif k < 0.72:
            self.out.append("while " + self.expr())
            self.block(level)
        elif k < 0.8:
            self.out.append("for " + self.name() + " in " + self.expr())
            self.block(level)
        elif k < 0.9:
            self.out.append("def " + self.name() + "(" + ", ".join(self.name() for _ in range(int(r.integers(0, 3)))) + ")")
            self.block(level)
        elif k < 0.95:
            self.out.append("class " + self.name().capitalize())
            self.block(level)
        else:
            self.out.append("try")
            self.block(level)
            self.out.append("except " + self.name())
            self.block(level)

    def program(self, n_stmts: int) -> bytes:
        self.out = []
        for _ in range(n_stmts):
            self.stmt(0)
        return "".join(self.out).encode()


def program(rng: np.random.Generator) -> bytes:
    """A moderate random program (C4 prefixes; stack depth well under 200)."""
    return ProgramGen(rng, expr_depth=int(rng.integers(2, 6)), block_depth=int(rng.integers(2, 6))).program(
        int(rng.integers(3, 12)))


_OPENERS = [
    ("(", 1), ("[", 1), ("f(", 1), ("g(x, ", 1), ("a[", 1), ("{k: ", 1), ("x + (", 1), ("y * (", 1),
    ("-(", 1), ("not (", 1), ("z if (", 1), ("[i for i in (", 1), ("h(a=", 1), ("q ** (", 1),
]
_BLOCK_OPENERS = ["if x:\n" + INDENT, "while y:\n" + INDENT, "for i in z:\n" + INDENT,
                  "def f(a):\n" + INDENT, "class K:\n" + INDENT, "try:\n" + INDENT]


def deep_program(rng: np.random.Generator, approx_chars: int = 6000) -> bytes:
    """A prefix that nests blocks and expressions ever deeper (never closes
    them), interleaved with complete statements, so the parser stack keeps
    growing (C5 prefixes, up to ~1,000 stack symbols)."""
    gen = ProgramGen(rng, expr_depth=2, block_depth=1)
    out: list[str] = []
    size = 0
    in_expr = False
    while size < approx_chars:
        r = rng.random()
        if not in_expr and r < 0.25:
            s = gen.simple() + "\n" + _BLOCK_OPENERS[int(rng.integers(len(_BLOCK_OPENERS)))]
        elif not in_expr and r < 0.35:
            s = gen.simple() + "\n"
        else:
            if not in_expr:
                s = gen.name() + " = "
                in_expr = True
            else:
                s = ""
            op, _ = _OPENERS[int(rng.integers(len(_OPENERS)))]
            s += op
            if rng.random() < 0.3:
                s += gen.expr(1) + ", "
        out.append(s)
        size += len(s)
    return "".join(out).encode()


def pylike_vocab(rng: np.random.Generator, V: int) -> Vocab:
    """Bytes + Zipf-length strings over identifiers, keywords, operators and
    whitespace runs."""
    idents = [n.encode() for n in _NAMES] + [f"{n}_{k}".encode() for n in _NAMES[:10] for k in range(10)]
    kws = [k.encode() for k in KEYWORDS] + [b" " + k.encode() for k in KEYWORDS]
    ops = [op.encode() for lvl in BINARY_LEVELS for op in lvl] + [op.encode() for op in AUGASSIGN]
    ops += [b"(", b")", b"[", b"]", b"{", b"}", b",", b":", b".", b";", b"=", b"->", b"):", b"()", b"],",
            b"\n", INDENT.encode(), DEDENT.encode(), b'"', b"'", b"#"]
    ws = [b" ", b"  ", b"    ", b"        ", b"\t", b"\n    "]
    digits = [bytes([c]) for c in b"0123456789"]
    pieces = idents + kws + ops + ws + digits
    weights = ([0.6] * len(idents) + [0.5] * len(kws) + [1.2] * len(ops) + [3.0] * len(ws)
               + [0.8] * len(digits))
    return piece_vocab(rng, V, pieces, weights, zipf_s=1.2, lo=2, hi=16)


@functools.lru_cache(maxsize=None)
def grammar() -> GrammarTables:
    return pylike_grammar()
