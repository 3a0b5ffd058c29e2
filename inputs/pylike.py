"""Python-like statement/expression grammar, programs and vocabularies.

Stand-in for the paper's programming-language workloads (Java/Go/SQL from
The Stack, Sec. 4.1), whose grammars and data are not available.

Grammar (96 terminals, 144 nonterminals counting the augmented start, 591
LR(0) states): def/class with type parameters, decorators, async def/for/with,
if/elif/else, while, for, try/except/except*/finally, with, match/case
(literal, capture, value, class, sequence, mapping, or- and as-patterns,
guards), and the simple statements (annotated and starred assignment,
augmented assignment, return, yield/yield from, raise from, global,
nonlocal, del, import/from-import with relative dots, assert, type aliases).
Blocks are NEWLINE INDENT stmts DEDENT, with INDENT and DEDENT spelled as the
reserved bytes 0x0E and 0x0F (a non-contextual lexer cannot count columns),
or one simple statement on the same line; spaces, tabs and comments are
ignored.  Expressions have a conditional expression, lambda with default and
starred parameters, assignment expressions, 14 stratified binary-operator
levels (left-recursive, power right-recursive), unary operators, await,
calls with keyword and unpacked arguments, subscripts/slices, attributes,
starred expressions, list/set/dict/tuple displays and their comprehensions,
and prefixed (f/r/b) strings.  Keywords are reserved.  The grammar is
LALR(1) as written.
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
            "as", "global", "try", "except", "finally", "raise", "assert", "del", "with", "yield",
            "async", "await", "match", "case", "nonlocal", "type"]

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
    g.regex("STRING", r'[fFrRbB]?"([^"\\\n]|\\.)*"' + "|" + r"[fFrRbB]?'([^'\\\n]|\\.)*'")
    g.ignore("WS", r"[ \t]+")
    g.ignore("COMMENT", r"#[^\n\x0e\x0f]*")
    for k in KEYWORDS:
        g.literal(k)
    NL, IND, DED = g.literal("\n"), g.literal(INDENT), g.literal(DEDENT)

    # ---- file and statements
    g.rule("file", [], ["file", "line"])
    g.rule("line", [NL], ["stmt"])
    g.rule("stmts", ["stmt"], ["stmts", "stmt"], ["stmts", NL])
    g.rule("suite", [NL, IND, "stmts", DED], ["simple_stmt"])
    g.rule("stmt", ["simple_stmt"], ["compound_stmt"])
    g.rule("simple_stmt", ["small_stmts", NL], ["small_stmts", '";"', NL])
    g.rule("small_stmts", ["small_stmt"], ["small_stmts", '";"', "small_stmt"])
    g.rule("small_stmt", ["expr_stmt"], ["flow_stmt"], ["pass_stmt"], ["global_stmt"], ["nonlocal_stmt"],
           ["del_stmt"], ["import_stmt"], ["assert_stmt"], ["type_stmt"])
    g.rule("expr_stmt", ["testlist"], ["testlist", '"="', "assign_rhs"], ["testlist", "augassign", "testlist"],
           ["testlist", "annassign"])
    g.rule("annassign", ['":"', "test"], ['":"', "test", '"="', "testlist"])
    g.rule("assign_rhs", ["testlist"], ["testlist", '"="', "assign_rhs"])
    g.rule("augassign", *[[f'"{op}"'] for op in AUGASSIGN])
    g.rule("pass_stmt", ['"pass"'])
    g.rule("flow_stmt", ["break_stmt"], ["continue_stmt"], ["return_stmt"], ["raise_stmt"], ["yield_stmt"])
    g.rule("break_stmt", ['"break"'])
    g.rule("continue_stmt", ['"continue"'])
    g.rule("return_stmt", ['"return"'], ['"return"', "testlist"])
    g.rule("yield_stmt", ['"yield"'], ['"yield"', "yield_arg"])
    g.rule("yield_arg", ["testlist"], ['"from"', "test"])
    g.rule("global_stmt", ['"global"', "names"])
    g.rule("nonlocal_stmt", ['"nonlocal"', "names"])
    g.rule("names", ["NAME"], ["names", '","', "NAME"])
    g.rule("del_stmt", ['"del"', "testlist"])
    g.rule("type_stmt", ['"type"', "NAME", "type_params_opt", '"="', "test"])
    g.rule("type_params_opt", [], ['"["', "type_params", '"]"'])
    g.rule("type_params", ["type_param"], ["type_params", '","', "type_param"])
    g.rule("type_param", ["NAME"], ["NAME", '":"', "test"], ['"*"', "NAME"], ['"**"', "NAME"])
    g.rule("import_stmt", ["import_name"], ["import_from"])
    g.rule("import_name", ['"import"', "dotted_as_names"])
    g.rule("import_from", ['"from"', "import_src", '"import"', "import_targets"])
    g.rule("import_src", ["dotted_name"], ["dots"], ["dots", "dotted_name"])
    g.rule("dots", ['"."'], ['".."'], ['"..."'], ["dots", '"."'], ["dots", '".."'], ["dots", '"..."'])
    g.rule("import_targets", ['"*"'], ["import_as_names"], ['"("', "import_as_names", '")"'])
    g.rule("import_as_names", ["import_as_name"], ["import_as_names", '","', "import_as_name"])
    g.rule("import_as_name", ["NAME"], ["NAME", '"as"', "NAME"])
    g.rule("dotted_as_names", ["dotted_as_name"], ["dotted_as_names", '","', "dotted_as_name"])
    g.rule("dotted_as_name", ["dotted_name"], ["dotted_name", '"as"', "NAME"])
    g.rule("dotted_name", ["NAME"], ["dotted_name", '"."', "NAME"])
    g.rule("assert_stmt", ['"assert"', "test"], ['"assert"', "test", '","', "test"])
    g.rule("raise_stmt", ['"raise"'], ['"raise"', "test"], ['"raise"', "test", '"from"', "test"])

    g.rule("compound_stmt", ["if_stmt"], ["while_stmt"], ["for_stmt"], ["funcdef"], ["classdef"],
           ["try_stmt"], ["with_stmt"], ["async_stmt"], ["decorated"], ["match_stmt"])
    g.rule("if_stmt", ['"if"', "named_expr", '":"', "suite", "elifs", "else_opt"])
    g.rule("elifs", [], ["elifs", "elif_clause"])
    g.rule("elif_clause", ['"elif"', "named_expr", '":"', "suite"])
    g.rule("else_opt", [], ["else_clause"])
    g.rule("else_clause", ['"else"', '":"', "suite"])
    g.rule("while_stmt", ['"while"', "named_expr", '":"', "suite", "else_opt"])
    g.rule("for_stmt", ['"for"', "targets", '"in"', "testlist", '":"', "suite", "else_opt"])
    g.rule("targets", ["target"], ["targets", '","', "target"])
    g.rule("target", ["NAME"], ['"("', "targets", '")"'], ['"["', "targets", '"]"'], ["star_target"])
    g.rule("star_target", ['"*"', "target"])
    g.rule("funcdef", ['"def"', "NAME", "type_params_opt", '"("', "params_opt", '")"', "returns_opt", '":"',
                       "suite"])
    g.rule("async_stmt", ['"async"', "funcdef"], ['"async"', "for_stmt"], ['"async"', "with_stmt"])
    g.rule("decorated", ["decorators", "funcdef"], ["decorators", "classdef"], ["decorators", '"async"', "funcdef"])
    g.rule("decorators", ["decorator"], ["decorators", "decorator"])
    g.rule("decorator", ['"@"', "dotted_name", NL], ['"@"', "dotted_name", '"("', "args_opt", '")"', NL])
    g.rule("returns_opt", [], ['"->"', "test"])
    g.rule("params_opt", [], ["params"], ["params", '","'])
    g.rule("params", ["param"], ["params", '","', "param"])
    g.rule("param", ["param_plain"], ["param_default"], ["star_param"], ["kwargs_param"], ['"/"'])
    g.rule("param_plain", ["NAME"], ["NAME", '":"', "test"])
    g.rule("param_default", ["param_plain", '"="', "test"])
    g.rule("star_param", ['"*"'], ['"*"', "param_plain"])
    g.rule("kwargs_param", ['"**"', "param_plain"])
    g.rule("classdef", ['"class"', "NAME", "type_params_opt", '":"', "suite"],
           ['"class"', "NAME", "type_params_opt", '"("', "args_opt", '")"', '":"', "suite"])
    g.rule("try_stmt", ['"try"', '":"', "suite", "excepts", "else_opt", "finally_opt"],
           ['"try"', '":"', "suite", '"finally"', '":"', "suite"])
    g.rule("excepts", ["except_clause"], ["excepts", "except_clause"])
    g.rule("except_clause", ['"except"', '":"', "suite"], ['"except"', "test", '":"', "suite"],
           ['"except"', "test", '"as"', "NAME", '":"', "suite"], ['"except"', '"*"', "test", '":"', "suite"])
    g.rule("finally_opt", [], ['"finally"', '":"', "suite"])
    g.rule("with_stmt", ['"with"', "with_items", '":"', "suite"])
    g.rule("with_items", ["with_item"], ["with_items", '","', "with_item"])
    g.rule("with_item", ["test"], ["test", '"as"', "target"])

    # ---- match statement
    g.rule("match_stmt", ['"match"', "named_expr", '":"', NL, IND, "case_blocks", DED])
    g.rule("case_blocks", ["case_block"], ["case_blocks", "case_block"])
    g.rule("case_block", ['"case"', "patterns", "guard_opt", '":"', "suite"])
    g.rule("guard_opt", [], ['"if"', "named_expr"])
    g.rule("patterns", ["seq_item"], ["patterns", '","', "seq_item"])
    g.rule("seq_item", ["as_pattern"], ['"*"', "NAME"])
    g.rule("as_pattern", ["or_pattern"], ["or_pattern", '"as"', "NAME"])
    g.rule("or_pattern", ["closed_pattern"], ["or_pattern", '"|"', "closed_pattern"])
    g.rule("closed_pattern", ["literal_pattern"], ["name_or_attr"],
           ["name_or_attr", '"("', "pattern_args_opt", '")"'], ['"("', '")"'], ['"("', "patterns", '")"'],
           ['"["', '"]"'], ['"["', "patterns", '"]"'], ["mapping_pattern"])
    g.rule("literal_pattern", ["NUMBER"], ['"-"', "NUMBER"], ["strings"], ['"None"'], ['"True"'], ['"False"'])
    g.rule("name_or_attr", ["NAME"], ["name_or_attr", '"."', "NAME"])
    g.rule("mapping_pattern", ['"{"', '"}"'], ['"{"', "mapping_items", '"}"'])
    g.rule("mapping_items", ["mapping_item"], ["mapping_items", '","', "mapping_item"])
    g.rule("mapping_item", ["key_pattern", '":"', "as_pattern"], ['"**"', "NAME"])
    g.rule("key_pattern", ["literal_pattern"], ["name_or_attr"])
    g.rule("pattern_args_opt", [], ["pattern_args"], ["pattern_args", '","'])
    g.rule("pattern_args", ["pattern_arg"], ["pattern_args", '","', "pattern_arg"])
    g.rule("pattern_arg", ["as_pattern"], ["NAME", '"="', "as_pattern"])

    # ---- expressions
    g.rule("testlist", ["tstar"], ["tstar", '","'], ["tstar", '","', "testlist_tail"])
    g.rule("testlist_tail", ["tstar"], ["tstar", '","'], ["tstar", '","', "testlist_tail"])
    g.rule("tstar", ["test"], ["star_expr"])
    g.rule("star_expr", ['"*"', "lvl6"])
    g.rule("named_expr", ["test"], ["NAME", '":="', "test"])
    g.rule("test", ["lvl0"], ["lvl0", '"if"', "lvl0", '"else"', "test"], ["lambdef"])
    g.rule("lambdef", ['"lambda"', '":"', "test"], ['"lambda"', "lambda_params", '":"', "test"])
    g.rule("lambda_params", ["lambda_param"], ["lambda_params", '","', "lambda_param"])
    g.rule("lambda_param", ["NAME"], ["NAME", '"="', "test"], ['"*"', "NAME"], ['"**"', "NAME"], ['"*"'])
    n = len(BINARY_LEVELS)
    for i, ops in enumerate(BINARY_LEVELS[:-1]):
        nxt = f"lvl{i + 1}" if i + 1 < n - 1 else "unary"
        if i == 3:      # after "and": the "not" level
            nxt = "notexpr"
            g.rule("notexpr", ['"not"', "notexpr"], ["lvl4"])
        if ops == ["<", ">", "<=", ">=", "in", "is"]:
            g.rule("comp_op", *[[f'"{op}"'] for op in ops], ['"not"', '"in"'], ['"is"', '"not"'])
            g.rule(f"lvl{i}", [nxt], [f"lvl{i}", "comp_op", nxt])
            continue
        g.rule(f"lvl{i}", [nxt], *[[f"lvl{i}", f'"{op}"', nxt] for op in ops])
    g.rule("unary", ['"-"', "unary"], ['"+"', "unary"], ['"~"', "unary"], ["power"])
    g.rule("power", ["await_primary"], ["await_primary", '"**"', "unary"])
    g.rule("await_primary", ["primary"], ['"await"', "primary"])
    g.rule("primary", ["atom"], ["primary", "trailer"])
    g.rule("trailer", ["call_trailer"], ["index_trailer"], ["attr_trailer"])
    g.rule("call_trailer", ['"("', "args_opt", '")"'])
    g.rule("index_trailer", ['"["', "subscripts", '"]"'])
    g.rule("attr_trailer", ['"."', "NAME"])
    g.rule("args_opt", [], ["args"], ["args", '","'])
    g.rule("args", ["arg"], ["args", '","', "arg"])
    g.rule("arg", ["named_expr"], ["test", "comp_clauses"], ["kwarg"], ["starred_arg"], ["kwstar_arg"])
    g.rule("kwarg", ["NAME", '"="', "test"])
    g.rule("starred_arg", ['"*"', "test"])
    g.rule("kwstar_arg", ['"**"', "test"])
    g.rule("subscripts", ["subscript"], ["subscripts", '","', "subscript"])
    g.rule("subscript", ["test"], ["slice"])
    # [lower] ":" [upper] [":" [step]], every part optional
    g.rule("slice", *[[*lo, '":"', *up, *st] for lo in ([], ["test"]) for up in ([], ["test"])
                      for st in ([], ['":"'], ['":"', "test"])])
    g.rule("atom", ["NAME"], ["literal_atom"], ["list_display"], ["dict_display"], ["set_display"],
           ["paren_display"], ['"..."'])
    g.rule("literal_atom", ["NUMBER"], ["strings"], ['"None"'], ['"True"'], ['"False"'])
    g.rule("list_display", ['"["', '"]"'], ['"["', "items", '"]"'], ['"["', "test", "comp_clauses", '"]"'])
    g.rule("dict_display", ['"{"', '"}"'], ['"{"', "dict_items", '"}"'],
           ['"{"', "test", '":"', "test", "comp_clauses", '"}"'])
    g.rule("set_display", ['"{"', "items", '"}"'], ['"{"', "test", "comp_clauses", '"}"'])
    g.rule("paren_display", ['"("', '")"'], ['"("', "testlist", '")"'], ['"("', "test", "comp_clauses", '")"'],
           ['"("', "NAME", '":="', "test", '")"'])
    g.rule("comp_clauses", ["comp_for"], ["comp_clauses", "comp_for"], ["comp_clauses", '"if"', "lvl2"])
    g.rule("comp_for", ['"for"', "targets", '"in"', "lvl2"], ['"async"', '"for"', "targets", '"in"', "lvl2"])
    g.rule("strings", ["STRING"], ["strings", "STRING"])
    g.rule("items", ["tstar"], ["items", '","', "tstar"], ["items", '","'])
    g.rule("dict_items", ["dict_item"], ["dict_items", '","', "dict_item"], ["dict_items", '","'])
    g.rule("dict_item", ["test", '":"', "test"], ['"**"', "lvl6"])
    return g.compile()


# ----------------------------------------------------------------- programs

_NAMES = ["x", "y", "i", "j", "n", "data", "value", "result", "items", "key", "node", "self", "count",
          "total", "buf", "line", "path", "obj", "cfg", "fn", "acc", "left", "right", "idx", "tmp"]
_TYPES = ["int", "str", "float", "bool", "list", "dict", "Node", "Any", "T", "K"]
_BIN_OPS = [op for lvl in BINARY_LEVELS for op in lvl] + ["not in", "is not"]


class ProgramGen:
    """Random programs over the whole grammar; `expr_depth` and
    `block_depth` bound expression and statement nesting."""

    def __init__(self, rng: np.random.Generator, expr_depth: int = 4, block_depth: int = 4):
        self.r = rng
        self.expr_depth = expr_depth
        self.block_depth = block_depth
        self.out: list[str] = []

    def pick(self, seq):
        return seq[int(self.r.integers(len(seq)))]

    def name(self) -> str:
        r = self.r
        if r.random() < 0.2:
            return self.pick(_NAMES) + str(int(r.integers(0, 100)))
        return self.pick(_NAMES)

    def string(self) -> str:
        r = self.r
        body = "".join("abcdefgh "[int(c)] for c in r.integers(0, 9, size=int(r.integers(0, 8))))
        pre = self.pick(["", "", "", "f", "r", "b"])
        if pre == "f" and r.random() < 0.6:
            body += "{" + self.name() + "}"
        return pre + ('"' + body + '"' if r.random() < 0.7 else "'" + body + "'")

    def annotation(self) -> str:
        r = self.r
        t = self.pick(_TYPES)
        if r.random() < 0.3:
            t += "[" + ", ".join(self.pick(_TYPES) for _ in range(int(r.integers(1, 3)))) + "]"
        if r.random() < 0.15:
            t += " | None"
        return t

    def comp(self, d: int) -> str:
        """ for-clauses (and if-clauses) of a comprehension."""
        r = self.r
        s = ""
        for k in range(int(r.integers(1, 3))):
            s += (" async" if r.random() < 0.05 else "") + " for " + self.targets() + " in " + self.atom(d)
            if r.random() < 0.3:
                s += " if " + self.atom(d) + " " + self.pick(["<", ">", "==", "!=", "in", "is not"]) + " " + \
                    self.atom(d)
        return s

    def targets(self) -> str:
        r = self.r
        k = r.random()
        if k < 0.6:
            return self.name()
        if k < 0.85:
            return ", ".join(self.name() for _ in range(int(r.integers(2, 4))))
        if k < 0.95:
            return "(" + self.name() + ", " + self.name() + ")"
        return self.name() + ", *" + self.name()

    def call_args(self, d: int) -> str:
        r = self.r
        args = []
        for _ in range(int(r.integers(0, 4))):
            k = r.random()
            if k < 0.6:
                args.append(self.expr(d))
            elif k < 0.8:
                args.append(self.name() + "=" + self.expr(d))
            elif k < 0.9:
                args.append("*" + self.atom(d))
            else:
                args.append("**" + self.atom(d))
        if len(args) == 1 and r.random() < 0.1:
            return self.expr(d) + self.comp(d)        # a bare generator argument
        return ", ".join(args)

    def lambdef(self, d: int) -> str:
        r = self.r
        ps = []
        for _ in range(int(r.integers(0, 3))):
            k = r.random()
            ps.append(self.name() if k < 0.6 else self.name() + "=" + self.atom(d) if k < 0.85 else
                      "*" + self.name() if k < 0.93 else "**" + self.name())
        return "lambda" + (" " + ", ".join(ps) if ps else "") + ": " + self.expr(d)

    def atom(self, d: int) -> str:
        r = self.r
        k = r.random()
        if k < 0.30 or d <= 0:
            return self.name() if r.random() < 0.7 else str(int(r.integers(0, 1000)))
        if k < 0.37:
            return self.string()
        if k < 0.46:
            return "(" + self.expr(d - 1) + ")"
        if k < 0.53:
            items = [self.expr(d - 1) if r.random() < 0.9 else "*" + self.atom(d - 1)
                     for _ in range(int(r.integers(0, 4)))]
            return "[" + ", ".join(items) + "]"
        if k < 0.58:
            items = [self.expr(d - 1) + ": " + self.expr(d - 1) if r.random() < 0.9 else "**" + self.atom(d - 1)
                     for _ in range(int(r.integers(0, 3)))]
            return "{" + ", ".join(items) + "}"
        if k < 0.61:
            return "{" + ", ".join(self.expr(d - 1) for _ in range(int(r.integers(1, 4)))) + "}"
        if k < 0.67:
            e = self.expr(d - 1)
            kind = int(r.integers(4))
            if kind == 0:
                return "[" + e + self.comp(d - 1) + "]"
            if kind == 1:
                return "{" + e + self.comp(d - 1) + "}"
            if kind == 2:
                return "{" + e + ": " + self.expr(d - 1) + self.comp(d - 1) + "}"
            return "(" + e + self.comp(d - 1) + ")"
        if k < 0.80:
            return self.name() + "(" + self.call_args(d - 1) + ")"
        if k < 0.85:
            sub = self.expr(d - 1)
            if r.random() < 0.3:
                sub = self.pick([sub + ":", ":" + sub, sub + ":" + self.atom(d - 1), "::" + self.atom(d - 1)])
            return self.name() + "[" + sub + "]"
        if k < 0.88:
            return self.name() + "." + self.name() + ("()" if r.random() < 0.4 else "")
        if k < 0.91:
            return "(" + self.lambdef(d - 1) + ")"
        if k < 0.94:
            return "await " + self.name() + "(" + self.call_args(d - 1) + ")"
        if k < 0.96:
            return "..."
        return "(" + self.name() + " := " + self.expr(d - 1) + ")"

    def expr(self, d: int | None = None) -> str:
        r = self.r
        d = self.expr_depth if d is None else d
        s = self.atom(d)
        for _ in range(int(r.integers(0, 3)) if d > 0 else 0):
            op = self.pick(_BIN_OPS)
            s = s + " " + op + " " + self.atom(d - 1)
        if d > 0 and r.random() < 0.05:
            s = s + " if " + self.atom(d - 1) + " else " + self.atom(d - 1)
        if d > 0 and r.random() < 0.05:
            s = "not " + s
        if d > 0 and r.random() < 0.03:
            s = self.lambdef(d - 1)
        return s

    def cond(self) -> str:
        """The condition of if/elif/while: sometimes an assignment expression."""
        if self.r.random() < 0.15:
            return self.name() + " := " + self.expr()
        return self.expr()

    def dotted(self) -> str:
        return ".".join(self.name() for _ in range(int(self.r.integers(1, 3))))

    def simple(self) -> str:
        r = self.r
        k = r.random()
        if k < 0.36:
            return self.name() + " = " + self.expr()
        if k < 0.44:
            return self.name() + " " + self.pick(AUGASSIGN) + " " + self.expr()
        if k < 0.54:
            return self.expr()
        if k < 0.62:
            return "return " + self.expr()
        if k < 0.67:
            return self.name() + ": " + self.annotation() + (" = " + self.expr() if r.random() < 0.7 else "")
        if k < 0.70:
            return self.targets() + " = " + self.expr()
        if k < 0.73:
            return self.name() + ", *" + self.name() + " = " + self.expr()
        if k < 0.76:
            return "yield " + self.expr() if r.random() < 0.6 else "yield from " + self.expr()
        if k < 0.79:
            rel = self.pick([".", "..", "...", ".", ""])
            src = rel + (self.dotted() if not rel or r.random() < 0.6 else "")
            tg = self.pick(["*", self.name(), self.name() + " as " + self.name(),
                            "(" + self.name() + ", " + self.name() + ")"])
            return "from " + src + " import " + tg
        if k < 0.81:
            return "type " + self.pick(["T", "K", "Alias"]) + ("[" + self.pick(["U", "V"]) + "]" if r.random() < 0.4
                                                                else "") + " = " + self.annotation()
        if k < 0.83:
            return "nonlocal " + self.name()
        if k < 0.85:
            return "raise " + self.name() + "(" + self.call_args(1) + ")" + (" from " + self.name() if r.random() < 0.5
                                                                             else "")
        if k < 0.87:
            return "assert " + self.expr() + (", " + self.string() if r.random() < 0.5 else "")
        return self.pick(["pass", "break", "continue", "global " + self.name(), "import os",
                          "import " + self.dotted() + " as " + self.name(), "del " + self.name(),
                          "del " + self.name() + ", " + self.name(), "raise"])

    def block(self, level: int):
        r = self.r
        if level + 1 < self.block_depth and r.random() < 0.08:
            self.out.append(": " + self.simple() + "\n")      # a one-line suite
            return
        self.out.append(":\n" + INDENT)
        for _ in range(int(r.integers(1, 4))):
            self.stmt(level + 1)
        self.out.append(DEDENT)

    def params(self) -> str:
        r = self.r
        ps = []
        for _ in range(int(r.integers(0, 4))):
            p = self.name()
            if r.random() < 0.3:
                p += ": " + self.annotation()
            if r.random() < 0.25:
                p += " = " + self.atom(1)
            ps.append(p)
        k = r.random()
        if k < 0.1:
            ps.append("*" + self.name())
        elif k < 0.15:
            ps.append("*")
            ps.append(self.name() + "=" + self.atom(1))
        if r.random() < 0.08:
            ps.append("**" + self.name())
        if ps and r.random() < 0.05:
            ps.insert(1, "/")
        return ", ".join(ps)

    def type_params(self) -> str:
        if self.r.random() < 0.15:
            return "[" + ", ".join(self.pick(["T", "K", "U: int", "*Ts", "**P"]) for _ in range(int(self.r.integers(1, 3)))) + "]"
        return ""

    def decorators(self):
        for _ in range(int(self.r.integers(1, 3))):
            d = "@" + self.dotted()
            if self.r.random() < 0.4:
                d += "(" + self.call_args(1) + ")"
            self.out.append(d + "\n")

    def funcdef(self, level: int, prefix: str = ""):
        s = prefix + "def " + self.name() + self.type_params() + "(" + self.params() + ")"
        if self.r.random() < 0.3:
            s += " -> " + self.annotation()
        self.out.append(s)
        self.block(level)

    def classdef(self, level: int):
        s = "class " + self.name().capitalize() + self.type_params()
        if self.r.random() < 0.5:
            s += "(" + self.call_args(1) + ")"
        self.out.append(s)
        self.block(level)

    def pattern(self, d: int = 2) -> str:
        """An as-pattern: closed patterns joined by "|", sometimes bound by "as"."""
        r = self.r
        s = " | ".join(self.closed_pattern(d) for _ in range(1 if r.random() < 0.85 else int(r.integers(2, 4))))
        return s + " as " + self.name() if r.random() < 0.1 else s

    def closed_pattern(self, d: int) -> str:
        r = self.r
        k = r.random() * 0.82
        if k < 0.25 or d <= 0:
            return self.pick([str(int(r.integers(0, 100))), "-" + str(int(r.integers(1, 9))), self.string(),
                              "None", "True", "False"])
        if k < 0.45:
            return self.pick(["_", self.name(), self.name() + "." + self.name().upper()])
        if k < 0.6:
            args = [self.pattern(d - 1) if r.random() < 0.6 else self.name() + "=" + self.pattern(d - 1)
                    for _ in range(int(r.integers(0, 3)))]
            return self.name().capitalize() + "(" + ", ".join(args) + ")"
        if k < 0.72:
            items = [self.pattern(d - 1) for _ in range(int(r.integers(0, 3)))]
            if r.random() < 0.3:
                items.append("*" + self.name())
            return self.pick(["[" + ", ".join(items) + "]", "(" + ", ".join(items) + ")" if len(items) != 1
                              else "[" + items[0] + "]"])
        items = [self.pick([str(int(r.integers(0, 9))), self.string()]) + ": " + self.pattern(d - 1)
                 for _ in range(int(r.integers(0, 3)))]
        if r.random() < 0.2:
            items.append("**" + self.name())
        return "{" + ", ".join(items) + "}"

    def match(self, level: int):
        r = self.r
        self.out.append("match " + self.expr() + ":\n" + INDENT)
        for _ in range(int(r.integers(1, 4))):
            s = "case " + self.pattern()
            if r.random() < 0.2:
                s += ", " + self.pattern(1)
            if r.random() < 0.2:
                s += " if " + self.cond()
            self.out.append(s)
            self.block(level + 1)
        self.out.append(DEDENT)

    def stmt(self, level: int):
        r = self.r
        k = r.random()
        if level >= self.block_depth or k < 0.5:
            self.out.append(self.simple() + "\n")
            return
        if k < 0.6:
            self.out.append("if " + self.cond())
            self.block(level)
            for _ in range(int(r.integers(0, 3)) if r.random() < 0.3 else 0):
                self.out.append("elif " + self.cond())
                self.block(level)
            if r.random() < 0.3:
                self.out.append("else")
                self.block(level)
        elif k < 0.65:
            self.out.append("while " + self.cond())
            self.block(level)
        elif k < 0.71:
            self.out.append(("async " if r.random() < 0.1 else "") + "for " + self.targets() + " in " + self.expr())
            self.block(level)
        elif k < 0.79:
            if r.random() < 0.2:
                self.decorators()
            self.funcdef(level, "async " if r.random() < 0.15 else "")
        elif k < 0.83:
            if r.random() < 0.2:
                self.decorators()
            self.classdef(level)
        elif k < 0.88:
            self.out.append("try")
            self.block(level)
            for _ in range(int(r.integers(1, 3))):
                self.out.append(self.pick(["except " + self.name(), "except " + self.name() + " as e", "except",
                                           "except* " + self.name()]))
                self.block(level)
            if r.random() < 0.2:
                self.out.append("else")
                self.block(level)
            if r.random() < 0.3:
                self.out.append("finally")
                self.block(level)
        elif k < 0.93:
            items = [self.expr() + (" as " + self.name() if r.random() < 0.5 else "")
                     for _ in range(int(r.integers(1, 3)))]
            self.out.append(("async " if r.random() < 0.15 else "") + "with " + ", ".join(items))
            self.block(level)
        else:
            self.match(level)

    def program(self, n_stmts: int) -> bytes:
        self.out = []
        for _ in range(n_stmts):
            self.stmt(0)
        return "".join(self.out).encode()


def program(rng: np.random.Generator) -> bytes:
    """A moderate random program (C4 prefixes; stack depth well under 200)."""
    return ProgramGen(rng, expr_depth=int(rng.integers(2, 6)), block_depth=int(rng.integers(2, 6))).program(
        int(rng.integers(3, 12)))


# expression openers that a deep prefix nests without closing
_OPENERS = ["(", "[", "f(", "g(x, ", "a[", "{k: ", "x + (", "y * (", "-(", "not (", "z if (",
            "[i for i in (", "h(a=", "q ** (", "{", "[*(", "await g(", "(n := (", "lambda a=(",
            "{**(", "{v for v in (", "f(*", "x[1:"]
_BLOCK_OPENERS = ["if x:\n" + INDENT, "while y:\n" + INDENT, "for i in z:\n" + INDENT,
                  "def f(a):\n" + INDENT, "class K:\n" + INDENT, "try:\n" + INDENT,
                  "async def g(a, *b) -> int:\n" + INDENT, "with a as b:\n" + INDENT,
                  "match x:\n" + INDENT + "case [1, *r]:\n" + INDENT, "@d\nclass K(B):\n" + INDENT,
                  "if (n := f()):\n" + INDENT, "async for i in z:\n" + INDENT]


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
            s += _OPENERS[int(rng.integers(len(_OPENERS)))]
            if rng.random() < 0.3:
                s += gen.expr(1) + ", "
        out.append(s)
        size += len(s)
    return "".join(out).encode()


def pylike_vocab(rng: np.random.Generator, V: int) -> Vocab:
    """Bytes + Zipf-length strings over identifiers, keywords, operators and
    whitespace runs."""
    idents = [n.encode() for n in _NAMES] + [f"{n}_{k}".encode() for n in _NAMES[:10] for k in range(10)]
    idents += [t.encode() for t in _TYPES]
    kws = [k.encode() for k in KEYWORDS] + [b" " + k.encode() for k in KEYWORDS]
    ops = [op.encode() for lvl in BINARY_LEVELS for op in lvl] + [op.encode() for op in AUGASSIGN]
    ops += [b"(", b")", b"[", b"]", b"{", b"}", b",", b":", b".", b";", b"=", b"->", b"):", b"()", b"],",
            b"\n", INDENT.encode(), DEDENT.encode(), b'"', b"'", b"#", b":=", b"...", b'f"', b"*", b"**"]
    ws = [b" ", b"  ", b"    ", b"        ", b"\t", b"\n    "]
    digits = [bytes([c]) for c in b"0123456789"]
    pieces = idents + kws + ops + ws + digits
    weights = ([0.6] * len(idents) + [0.5] * len(kws) + [1.2] * len(ops) + [3.0] * len(ws)
               + [0.8] * len(digits))
    return piece_vocab(rng, V, pieces, weights, zipf_s=1.2, lo=2, hi=16)


@functools.lru_cache(maxsize=None)
def grammar() -> GrammarTables:
    return pylike_grammar()
