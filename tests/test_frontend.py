"""Pins for the input side: lexer generator, LALR(1) generator, host parser."""
import itertools

import numpy as np
import pytest

from conftest import grammar, host
from inputs import documents, vocab
from inputs.grammar import ACT_ACCEPT, ACT_REDUCE, ACT_SHIFT, ConflictError, Grammar
from inputs.lexgen import TerminalDef, build_lexer, lex_step, literal_ast, parse_regex
from inputs.seeds import rng_for
from recognizers import arith_accepts, json_accepts


def _lex_all(lex, text: bytes, ignored=frozenset()):
    cur, out = 0, []
    for c in text:
        cur, t = lex_step(lex, cur, c, set(ignored))
        if t is not None:
            out.append(lex.terminal_names[t])
        if cur < 0:
            return None
    if cur != 0:
        t = int(lex.accept[cur])
        if t < 0:
            return None
        if t not in ignored:
            out.append(lex.terminal_names[t])
    return out


def test_textbook_expression_grammar_has_12_lalr_states(arith):
    # E -> E+T | T, T -> T*F | F, F -> (E) | id augmented with S' -> E has the
    # twelve LR(0) item sets I0..I11 of the classic textbook construction, and
    # LALR(1) merges nothing further; it is conflict-free.
    assert arith.n_lr_states == 12
    acc = (arith.action & 3) == ACT_ACCEPT
    assert acc.sum() == 1 and acc[:, arith.end_terminal].sum() == 1
    # every state has at least one non-error action (no useless states)
    assert ((arith.action & 3) != 0).any(axis=1).all()


def test_ambiguous_grammar_reports_conflict():
    g = Grammar("e")
    g.regex("N", "[0-9]")
    g.rule("e", 'e "+" e', "N")
    with pytest.raises(ConflictError):
        g.compile()


def test_dangling_else_reports_conflict():
    g = Grammar("s")
    g.regex("X", "x")
    g.rule("s", '"if" s', '"if" s "else" s', "X")
    with pytest.raises(ConflictError):
        g.compile()


def test_json_grammar_is_lalr1(json_g):
    assert json_g.n_lr_states > 10
    kinds = json_g.action & 3
    assert (kinds == ACT_SHIFT).any() and (kinds == ACT_REDUCE).any()


def test_lexer_longest_match_and_priorities():
    terms = [
        TerminalDef("NAME", parse_regex("[a-z]+")),
        TerminalDef('"if"', literal_ast("if"), is_literal=True),
        TerminalDef("NUM", parse_regex("[0-9]+")),
        TerminalDef('"="', literal_ast("="), is_literal=True),
        TerminalDef('"=="', literal_ast("=="), is_literal=True),
        TerminalDef("WS", parse_regex(" +"), ignored=True),
    ]
    lex = build_lexer(terms)
    ign = {5}
    assert _lex_all(lex, b"if", ign) == ['"if"']            # literal beats regex on a tie
    assert _lex_all(lex, b"iffy", ign) == ["NAME"]          # longest match
    assert _lex_all(lex, b"if x==12", ign) == ['"if"', "NAME", '"=="', "NUM"]
    assert _lex_all(lex, b"a = =b", ign) == ["NAME", '"="', '"="', "NAME"]
    assert _lex_all(lex, b"a+b", ign) is None               # no terminal for '+'
    assert lex.accept[0] == -1                              # q0 never accepts
    assert not (lex.next == 0).any()                        # nothing returns to q0


def test_lexer_no_backtracking():
    # "a" and "abc" but not "ab": longest match from "ab" + "x" fails instead
    # of backing up to "a" (one byte of lookahead only).
    terms = [TerminalDef('"a"', literal_ast("a"), is_literal=True),
             TerminalDef('"abc"', literal_ast("abc"), is_literal=True),
             TerminalDef('"x"', literal_ast("x"), is_literal=True)]
    lex = build_lexer(terms)
    assert _lex_all(lex, b"abc", set()) == ['"abc"']
    assert _lex_all(lex, b"ax", set()) == ['"a"', '"x"']
    assert _lex_all(lex, b"abx", set()) is None


def test_regex_features():
    lex = build_lexer([TerminalDef("H", parse_regex(r"0x[0-9a-fA-F]{2,3}")),
                       TerminalDef("S", parse_regex(r'"([^"\\]|\\.)*"')),
                       TerminalDef("D", parse_regex(r"\d+(\.\d+)?"))])
    assert _lex_all(lex, b"0x1f") == ["H"]
    assert _lex_all(lex, b"0x1fA") == ["H"]
    assert _lex_all(lex, b"0x1") is None
    assert _lex_all(lex, b'"a\\"b"') == ["S"]
    assert _lex_all(lex, b"3.25") == ["D"]


@pytest.mark.slow
def test_arithmetic_front_end_matches_recursive_descent_exhaustively():
    # every string over {0,1,+,*,(,),space} up to length 6
    hp = host("arithmetic")
    alphabet = b"01+*() "
    texts = [bytes(t) for n in range(7) for t in itertools.product(alphabet, repeat=n)]
    got = hp.accepts_many(texts)
    want = np.array([arith_accepts(t) for t in texts])
    bad = [texts[i] for i in np.nonzero(got != want)[0][:10]]
    assert not bad, bad


def _mutate(rng, doc: bytes) -> bytes:
    b = bytearray(doc)
    for _ in range(int(rng.integers(1, 4))):
        op = int(rng.integers(3))
        i = int(rng.integers(0, len(b) + 1))
        ch = bytes([int(rng.choice(list(b'{}[],:"\\ 0123456789.eE-+tfnaulrsx\x01\x80')))])
        if op == 0 and len(b):
            del b[min(i, len(b) - 1)]
        elif op == 1:
            b[i:i] = ch
        elif len(b):
            b[min(i, len(b) - 1)] = ch[0]
    return bytes(b)


def test_json_front_end_matches_independent_validator():
    hp = host("json")
    rng = rng_for(2, salt=7)
    words = vocab.synthetic_words(rng, 50)
    docs = [documents.json_document(rng, words, budget=30) for _ in range(400)]
    texts = list(docs)
    texts += [_mutate(rng, d) for d in docs for _ in range(3)]
    alphabet = b'{}[],:"\\ 01-.eEtrunl'
    texts += [bytes(rng.choice(list(alphabet), size=int(rng.integers(0, 8))).tolist()) for _ in range(3000)]
    texts += [b"", b"0", b"-0", b"01", b"1.", b"1.5e", b"1e+2", b'"\\u00e9"', b'"\\x"', b'"\x01"',
              b"[1,]", b"{,}", b'{"a":1,}', b"true false", b" null ", b'"\xff"', b"[[[]]]"]
    got = hp.accepts_many(texts)
    want = np.array([json_accepts(t) for t in texts])
    bad = [texts[i] for i in np.nonzero(got != want)[0][:10]]
    assert not bad, bad
    assert want.sum() > 400  # the generated documents are all valid


def test_generated_documents_are_in_the_language():
    hp = host("arithmetic")
    rng = rng_for(1, salt=3)
    docs = [documents.arithmetic_document(rng) for _ in range(500)]
    assert hp.accepts_many(docs).all()
    assert all(arith_accepts(d) for d in docs)


def test_prefix_states_are_consistent_along_a_document():
    hp = host("json")
    rng = rng_for(2, salt=11)
    words = vocab.synthetic_words(rng, 50)
    doc = documents.json_document(rng, words)
    cuts = sorted(set(rng.integers(0, len(doc) + 1, size=20).tolist()))
    many = hp.states_at(doc, cuts)
    for c, (q, st) in zip(cuts, many):
        q1, st1 = hp.state(doc[:c])
        assert q == q1 and np.array_equal(st, st1)
        assert st[0] == 0                      # the LR start state is the bottom
