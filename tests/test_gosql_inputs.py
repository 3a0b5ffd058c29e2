"""The programming-language-scale workload's input side: a Go-like grammar
with embedded SQL at the size of the paper's Java/Go grammars (Tab.
preprocess), its document generator and its vocabulary.

The generator derives sentences from the grammar's productions (a random
derivation, written without the LALR(1) tables), so every generated program
being accepted by the table-driven host parser pins the LALR(1) construction
on a grammar of this size; the deep prefixes pin the workload's stack depths.
"""
import numpy as np

from inputs import configs, gosql
from inputs.native import HostParser
from inputs.seeds import rng_for


def test_grammar_has_programming_language_size():
    g = gosql.grammar()                       # raises ConflictError on any LALR(1) conflict
    assert g.n_terminals >= 150 and g.n_nonterminals >= 250 and g.n_lr_states >= 1500
    assert len(g.productions) >= 700


def test_generated_programs_are_in_the_language():
    g = gosql.grammar()
    hp = HostParser(g)
    rng = rng_for(5, salt=0x7E57)
    docs = [gosql.program(rng) for _ in range(200)]
    assert hp.accepts_many(docs).all()
    # and they use much of the grammar: most keywords occur
    text = b"".join(docs)
    kws = [k.encode() for k in gosql.SQL_KEYWORDS + gosql.GO_KEYWORDS]
    seen = {k for k in kws if k in text}
    assert len(seen) >= 0.6 * len(kws)


def test_deep_prefixes_are_viable_and_deep():
    hp = HostParser(gosql.grammar())
    rng = rng_for(5, salt=0xDEE9)
    docs = [gosql.deep_program(rng, approx_chars=3000) for _ in range(20)]
    assert hp.viable_many(docs).all()
    assert not hp.accepts_many(docs).any()       # never closed
    depth = [len(hp.state(d)[1]) for d in docs]
    assert min(depth) > 200, depth


def test_workload_prefixes_and_vocabulary():
    wl = configs.get("gosql")
    assert wl.V == 4096
    tokens = [t for i, t in enumerate(wl.vocab.tokens) if i != wl.vocab.eos_id]
    assert len(set(tokens)) == len(tokens)
    assert {bytes([c]) for c in range(256)} <= set(tokens)
    states = wl.states(0)
    assert len(states) == wl.B
    depths = np.array([len(st) for _, st in wl.states(1)])
    assert depths.max() > 100
    assert all(st[0] == 0 for _, st in states)
