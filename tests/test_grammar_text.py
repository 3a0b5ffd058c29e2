"""The C library's grammar front end (psc_grammar_compile,
psc_build_from_text): grammar text -> the lexer and LALR(1) tables that
Algorithm 1 takes (Sec. 4.1 obtains the parser from an LALR(1) generator).

It is pinned to the input side's own front end (inputs/lexgen.py,
inputs/grammar.py), written independently in Python: on every workload
grammar and on 1,000 seeded random grammars both must produce the same
tables, entry for entry, and reject the same grammars as not LALR(1).  The
Python side writes its grammar in the text form (Grammar.to_text).
"""
import numpy as np
import pytest

from inputs import configs
from inputs.grammar import ConflictError, Grammar, GrammarError
from paper_2608_03065_amd import psc
from paper_2608_03065_amd.psc import Classifier, CompiledGrammar, PscError

from test_random_grammars import _random_grammar, _random_vocab


def _same_tables(c, g):
    assert np.array_equal(c.lex_next, g.lexer.next)
    assert np.array_equal(c.lex_accept, g.lexer.accept)
    assert np.array_equal(c.terminal_ignored, g.terminal_ignored)
    assert c.end_terminal == g.end_terminal
    assert np.array_equal(c.action, g.action)
    assert np.array_equal(c.goto, g.goto)
    assert np.array_equal(c.prod_lhs, g.prod_lhs) and np.array_equal(c.prod_len, g.prod_len)
    assert c.terminal_names == g.terminal_names and c.nonterminal_names == g.nonterminal_names


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema", "pylike", "gosql"])
def test_workload_grammars_compile_to_the_same_tables(name):
    g = configs.get(name).grammar
    _same_tables(CompiledGrammar(g.text), g)


def test_random_grammars_same_tables_and_same_verdicts():
    n_ok = n_conflict = 0
    for seed in range(1000):
        rng = np.random.default_rng(5000 + seed)
        builder = _random_grammar(rng, compiled=False)
        text = builder.to_text()
        try:
            g = builder.compile()
        except ConflictError:
            with pytest.raises(PscError) as e:
                CompiledGrammar(text)
            assert e.value.status == -3 and "LALR(1) conflicts" in str(e.value), seed
            n_conflict += 1
            continue
        _same_tables(CompiledGrammar(text), g)
        n_ok += 1
    assert n_ok >= 50 and n_conflict >= 20, (n_ok, n_conflict)


def test_text_features():
    """Alternatives on one line and on continuation lines, the empty
    production, priorities, comments, escapes; the same grammar written with
    the Python builder gives the same tables, and the keyword wins over the
    identifier on the same lexeme by its priority."""
    text = r'''
# statements separated by ';'
%start prog
%ignore WS /[ \t]+/         # blanks
%ignore COMMENT /\/\/[^\n]*/
ID: /[a-z]+/
NUM.2: /[0-9]+(\.[0-9]*)?/
%literal "if" 1
prog: prog stmt |
stmt: "if" ID ";"
    | ID "=" expr ";"       # assignment
    | "\x7b" prog "}"
expr: expr "+" NUM | NUM | ID | "\"s\""
'''
    b = Grammar("prog")
    b.ignore("WS", r"[ \t]+")
    b.ignore("COMMENT", r"//[^\n]*")
    b.regex("ID", "[a-z]+")
    b.regex("NUM", r"[0-9]+(\.[0-9]*)?", priority=2)
    b.literal("if", 1)
    b.rule("prog", "prog stmt", "")
    b.rule("stmt", '"if" ID ";"', 'ID "=" expr ";"', '"{" prog "}"')
    b.rule("expr", 'expr "+" NUM', "NUM", "ID", '""s""')
    g = b.compile()
    c = CompiledGrammar(text)
    _same_tables(c, g)
    # the lexeme "if" is the keyword, "iff" an identifier
    kw, ident = c.terminal_names.index('"if"'), c.terminal_names.index("ID")
    q = 0
    for ch in b"if":
        q = c.lex_next[q, ch]
    assert c.lex_accept[q] == kw
    assert c.lex_accept[c.lex_next[q, ord("f")]] == ident
    # and the C front end's text round trip is stable
    _same_tables(CompiledGrammar(g.text), g)


@pytest.mark.parametrize("text,status,needle", [
    ('%start e\nN: /[0-9]/\ne: e "+" e | N\n', -3, "LALR(1) conflicts"),
    ('%start s\nX: /x/\ns: "if" s | "if" s "else" s | X\n', -3, "on \"else\""),
    ('%start s\nA: /a/\ns: A t\n', -2, "line 3: undefined symbol t"),
    ('%start s\ns: t\n', -2, "no terminals"),
    ('%start s\nA: /a*/\ns: A\n', -2, "matches the empty string"),
    ('%start s\n%ignore WS / +/\ns: WS\n', -2, "ignored terminal WS"),
    ('s: "a"\n', -2, "no %start"),
    ('%start s\nA: /a/\nA: /b/\ns: A\n', -2, "line 3: terminal A declared twice"),
    ('%start s\ns "a"\n', -2, "line 2: expected ':'"),
    ('%start s\ns: "a\n', -2, "line 2: unterminated literal"),
    ('%start s\nA: /[a-/\ns: A\n', -2, "unterminated class"),
    ('%start s\nA: /(a/\ns: A\n', -2, "missing )"),
    ('%start s\nA: /*a/\ns: A\n', -2, "nothing to repeat"),
    ('%start s\n%bogus\ns: "a"\n', -2, "unknown directive"),
    ('%start t\ns: "a"\n', -2, "start symbol t has no rules"),
    ('', -2, "no %start"),
    ('%start s\nA: /' + '(' * 600 + 'a' + ')' * 600 + '/\ns: A\n', -2, "nested deeper than 500"),
    ('%start s\nA: /a' + '*' * 600 + '/\ns: A\n', -2, "repetition operators in a row"),
    ('%start s\nA: /((((a{100}){100}){100}){100})/\ns: A\n', -7, "NFA exceeds"),
    ('%start s\nA: /[ab]*a[ab]{21}/\ns: A\n', -7, "lexer DFA exceeds"),
])
def test_errors_are_reported(text, status, needle):
    with pytest.raises(PscError) as e:
        CompiledGrammar(text)
    assert e.value.status == status and needle in str(e.value), str(e.value)


def test_bounded_repetition_compiles_in_time_and_exactly():
    """A move of the subset construction is one closure search over all its
    targets: /[ab]{0,2000}c/ (2,000 nested optional copies, whose closures
    overlap) compiles in seconds, and its DFA counts the repetition exactly."""
    import time
    t0 = time.time()
    c = CompiledGrammar('%start s\nA: /[ab]{0,2000}c/\ns: A\n')
    assert time.time() - t0 < 60

    def run(text):
        q = 0
        for ch in text.encode():
            q = int(c.lex_next[q, ch])
            if q < 0:
                return None
        return q

    q = run("ab" * 1000 + "c")
    assert q is not None and c.lex_accept[q] == 0
    assert run("a" * 2001) is None and run("c") is not None and run("cc") is None


def test_build_from_text_equals_build_from_tables():
    """psc_build_from_text gives the classifier psc_build gives on the
    Python front end's tables: same sizes and the same class rows for the
    same prefix states."""
    for name in ("arithmetic", "json"):
        wl = configs.get(name)
        a = Classifier(wl.grammar, wl.vocab)
        b = Classifier.from_text(wl.grammar.text, wl.vocab)
        ia, ib = a.info(), b.info()
        for k in ("n_classes", "dfa_states", "dfa_rows", "table_bytes", "mask_table_bytes", "n_lr_states"):
            assert ia[k] == ib[k], (name, k)
        states = [st for s in range(3) for st in wl.states(s)]
        assert np.array_equal(a.masks_host(states), b.masks_host(states)), name
    rng = np.random.default_rng(77)
    vocab = _random_vocab(rng)
    with pytest.raises(PscError) as e:
        Classifier.from_text('%start e\nN: /[0-9]/\ne: e "+" e | N\n', vocab)
    assert e.value.status == -3


def test_symbol_names_out_of_range_are_null():
    lib = psc.lib()
    import ctypes as C
    h = C.c_void_p()
    text = b'%start s\ns: "a"\n'
    assert lib.psc_grammar_compile(text, len(text), C.byref(h)) == 0
    try:
        assert lib.psc_grammar_symbol_name(h, 1, 0) == b'"a"'
        assert lib.psc_grammar_symbol_name(h, 1, 1) == b"$END"
        assert lib.psc_grammar_symbol_name(h, 1, 2) is None
        assert lib.psc_grammar_symbol_name(h, 0, -1) is None
        assert lib.psc_grammar_symbol_name(h, 0, 1) == b"$start"
    finally:
        lib.psc_grammar_free(h)
