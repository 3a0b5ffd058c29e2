"""Pins of the oracle's one-token advance of a prefix state (Sec. 3.2; the
lexing and parsing steps of Algorithm 2).

The independent reference is the input generator's host parser, which lexes
and parses a whole text from scratch: advancing token by token through a
document must reproduce its (lexer state, stack) at every token boundary.
The advance is also tied to the masks: a token the mask allows always
advances, a rejected token is never allowed, and a token that advances
although the mask forbids it leaves a state from which nothing is allowed.
"""
import numpy as np
import pytest

from inputs import configs, pylike
from inputs.seeds import rng_for
from oracle import Oracle


def _walk_document(wl, orc, text):
    toks = wl.vocab.tokenize(text)
    cuts = np.cumsum([len(wl.vocab.tokens[t]) for t in toks])
    want = wl.host.states_at(text, cuts)
    state = wl.host.state(b"")
    for k, t in enumerate(toks):
        st, new = orc.advance(state, t)
        assert st == Oracle.ADVANCED, (k, t)
        assert new[0] == want[k][0] and np.array_equal(new[1], want[k][1]), k
        state = new
    return state


@pytest.mark.parametrize("name,n_docs", [("arithmetic", 12), ("json", 6), ("schema", 3), ("pylike", 2)])
def test_advance_matches_host_parser_on_documents(name, n_docs):
    wl = configs.get(name)
    orc = Oracle(wl.grammar, wl.vocab)
    for i in range(n_docs):
        rng = rng_for(wl.index, 77, i, salt=0xADF)
        # complete documents only (a quarter of the Python-like workload's
        # documents are prefixes that never close)
        text = pylike.program(rng) if name == "pylike" else wl.make_document(rng, wl)
        state = _walk_document(wl, orc, text)
        # the whole document is a sentence: EOS is accepted and changes nothing
        assert wl.host.accepts(text)
        st, new = orc.advance(state, wl.vocab.eos_id)
        assert st == Oracle.EOS_ACCEPTED and new is None


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema"])
def test_advance_agrees_with_masks(name):
    wl = configs.get(name)
    orc = Oracle(wl.grammar, wl.vocab)
    rng = np.random.default_rng(5)
    states = wl.states(3, B=6)
    masks = orc.masks(states)
    for state, m in zip(states, masks):
        bits = np.unpackbits(m.astype("<u4").view(np.uint8), bitorder="little")[:wl.V].astype(bool)
        allowed = np.nonzero(bits)[0]
        cand = np.concatenate([rng.choice(allowed, min(20, allowed.size), replace=False) if allowed.size else [],
                               rng.integers(0, wl.V, 40), [wl.vocab.eos_id]]).astype(int)
        for t in cand:
            st, new = orc.advance(state, int(t))
            if bits[t]:
                assert st == (Oracle.EOS_ACCEPTED if t == wl.vocab.eos_id else Oracle.ADVANCED), t
            if st == Oracle.REJECTED:
                assert not bits[t]
            if st == Oracle.ADVANCED and not bits[t]:
                # a pending lexeme nothing completes: no token is allowed next
                assert not orc.masks([new]).any(), t


def test_advance_capacity_and_rejection_leave_state():
    wl = configs.get("arithmetic")
    orc = Oracle(wl.grammar, wl.vocab)
    toks = wl.vocab.tokens
    lp = toks.index(b"(")
    state = wl.host.state(b"")
    # each "(" pushes onto the stack; a tight cap overflows
    st, new = orc.advance(state, lp)
    assert st == Oracle.ADVANCED
    st2, _ = orc.advance(new, lp, cap=len(new[1]))
    assert st2 == Oracle.OVERFLOW
    # "()" is not a sentence prefix, but with one byte of lookahead the ")"
    # only becomes a terminal on the next token: ")" advances (its lexeme is
    # pending), nothing is allowed after it, and the next token is rejected
    rp, plus = toks.index(b")"), toks.index(b"+")
    st3, new3 = orc.advance(new, rp)
    assert st3 == Oracle.ADVANCED and not orc.masks([new3]).any()
    assert orc.advance(new3, plus) == (Oracle.REJECTED, None)
