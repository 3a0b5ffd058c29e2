"""The Python-like workloads' input side: the full grammar at the size its
configuration names (~90 terminals, ~150 nonterminals, 14 binary precedence
levels), its program generator and the stack depths of its prefixes; and the
core grammar that the deep-nesting workload keeps.

The generator writes programs from its own templates, not from the LALR(1)
tables, so every generated program being accepted by the table-driven host
parser pins the LALR(1) construction on this grammar (and the generator's
use of every construct pins that the grammar has them).
"""
import numpy as np

from inputs import configs, pylike, pylike_core
from inputs.native import HostParser
from inputs.seeds import rng_for


def test_full_grammar_has_the_configured_size():
    g = pylike.grammar()                      # raises ConflictError on any LALR(1) conflict
    assert 90 <= g.n_terminals <= 100 and 140 <= g.n_nonterminals <= 160
    levels = [f"lvl{i}" for i in range(len(pylike.BINARY_LEVELS) - 1)] + ["power"]
    assert len(pylike.BINARY_LEVELS) == 14 and all(n in g.nonterminal_names for n in levels)


def test_generated_programs_are_in_the_language_and_use_it():
    hp = HostParser(pylike.grammar())
    rng = rng_for(3, salt=0x7E57)
    docs = [pylike.program(rng) for _ in range(300)]
    assert hp.accepts_many(docs).all()
    text = b"".join(docs)
    assert all(k.encode() in text for k in pylike.KEYWORDS)
    for construct in (b"match ", b"case ", b"async def", b"await ", b":=", b"except*", b"yield from",
                      b"nonlocal ", b"type ", b"lambda ", b" for ", b"**", b"[::", b"...", b"@", b"f\""):
        assert construct in text, construct


def test_deep_prefixes_are_viable_and_deep():
    hp = HostParser(pylike.grammar())
    rng = rng_for(3, salt=0xDEE9)
    docs = [pylike.deep_program(rng, approx_chars=2500) for _ in range(20)]
    assert hp.viable_many(docs).all()
    assert not hp.accepts_many(docs).any()       # never closed
    assert min(len(hp.state(d)[1]) for d in docs) > 300


def test_c4_prefixes_reach_the_configured_depth():
    wl = configs.get("pylike")
    assert wl.V == 128256 and wl.grammar is pylike.grammar()
    depths = np.array([len(st) for s in range(12) for _, st in wl.states(s)])
    assert 150 <= depths.max() <= 260 and np.median(depths) < 60


def test_the_deep_workload_keeps_the_core_grammar():
    g = pylike_core.grammar()
    assert (g.n_terminals, g.n_nonterminals, g.n_lr_states) == (88, 80, 382)
    wl = configs.get("stress")
    assert wl.grammar is g and wl.V == 262144
    # the core language is contained in the full one: its programs parse there too
    rng = rng_for(4, salt=0x7E57)
    docs = [pylike_core.program(rng) for _ in range(100)]
    assert HostParser(pylike.grammar()).accepts_many(docs).all()
