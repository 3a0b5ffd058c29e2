"""The six synthetic workloads (grammar, vocabulary, prefixes, logits).

Each prefix is drawn independently per (step, b) from a seeded random
document of the workload's language, truncated at a uniform byte position
(0..len inclusive), so prefixes end mid-lexeme as often as the documents'
lexeme lengths dictate.  Everything is a pure function of the seeds.
"""
from __future__ import annotations

import functools
from dataclasses import dataclass
from typing import Callable

import numpy as np

from . import documents, grammars, gosql, pylike, pylike_core, schema, vocab
from .grammar import GrammarTables
from .native import HostParser
from .seeds import rng_for


@dataclass
class Workload:
    index: int                   # 0..5
    name: str
    B: int
    steps: int
    logits_dtype: str            # "f32" | "bf16"
    logits_std: float
    make_grammar: Callable[[], GrammarTables]
    make_vocab: Callable[[GrammarTables], vocab.Vocab]
    make_document: Callable[[np.random.Generator, "Workload"], bytes]
    description: str = ""
    doc_pool: int = 0            # > 0: prefixes cut from a seeded pool of this many documents

    # ---- cached pieces ----
    @functools.cached_property
    def grammar(self) -> GrammarTables:
        return self.make_grammar()

    @functools.cached_property
    def vocab(self) -> vocab.Vocab:
        return self.make_vocab(self.grammar)

    @functools.cached_property
    def host(self) -> HostParser:
        return HostParser(self.grammar)

    @property
    def V(self) -> int:
        return self.vocab.size

    @functools.cached_property
    def documents(self) -> list[bytes]:
        """The seeded document pool (only when doc_pool > 0)."""
        return [self.make_document(rng_for(self.index, 0, i, salt=0xD0C5), self)
                for i in range(self.doc_pool)]

    def prefix(self, step: int, b: int) -> bytes:
        rng = rng_for(self.index, step, b)
        if self.doc_pool:
            doc = self.documents[int(rng.integers(0, self.doc_pool))]
        else:
            doc = self.make_document(rng, self)
        cut = int(rng.integers(0, len(doc) + 1))
        return doc[:cut]

    def states(self, step: int, B: int | None = None) -> list[tuple[int, np.ndarray]]:
        """(q, stack) for every sequence of one decoding step."""
        B = self.B if B is None else B
        return [self.host.state(self.prefix(step, b)) for b in range(B)]

    def logits(self, step: int, B: int | None = None):
        """Seeded logits as a CPU torch tensor [B, V]."""
        import torch
        B = self.B if B is None else B
        gen = torch.Generator().manual_seed(0x50534300 + self.index * 1_000_003 + step)
        x = torch.randn(B, self.V, generator=gen, dtype=torch.float32) * self.logits_std
        return x.to(torch.bfloat16) if self.logits_dtype == "bf16" else x


def _arith_doc(rng, wl):
    return documents.arithmetic_document(rng, max_depth=12)


@functools.lru_cache(maxsize=None)
def _json_words():
    return vocab.synthetic_words(rng_for(1, salt=0xD0C), 400)


def _json_doc(rng, wl):
    return documents.json_document(rng, _json_words(), max_depth=20)


def _c1_vocab(g):
    return vocab.arithmetic_vocab(rng_for(0, salt=0x70C), 513)


def _c2_vocab(g):
    return vocab.json_vocab(rng_for(1, salt=0x70C), 32000)


WORKLOADS: dict[str, Workload] = {}


def _register(w: Workload):
    WORKLOADS[w.name] = w
    return w


ARITHMETIC = _register(Workload(
    0, "arithmetic", B=1, steps=200, logits_dtype="f32", logits_std=1.0,
    make_grammar=grammars.arithmetic, make_vocab=_c1_vocab, make_document=_arith_doc,
    description="E->E+T|T, T->T*F|F, F->(E)|NUM, spaces; V=513; B=1; fp32 N(0,1)"))

JSON = _register(Workload(
    1, "json", B=16, steps=500, logits_dtype="f32", logits_std=1.0,
    make_grammar=grammars.json_grammar, make_vocab=_c2_vocab, make_document=_json_doc,
    description="JSON; byte-level V=32,000; B=16; fp32 N(0,1)"))


def _c3_grammar():
    return schema.schema_grammar(schema.c3_schema())


def _c3_vocab(g):
    return schema.schema_vocab(rng_for(2, salt=0x70C), schema.c3_schema(), 151936)


def _c3_doc(rng, wl):
    return schema.document(rng, schema.c3_schema())


SCHEMA = _register(Workload(
    2, "schema", B=64, steps=1000, logits_dtype="bf16", logits_std=2.0,
    make_grammar=_c3_grammar, make_vocab=_c3_vocab, make_document=_c3_doc, doc_pool=4096,
    description="schema-conformant JSON (seeded schema: 10 object types, 5 levels); "
                "V=151,936; B=64; bf16 N(0,2)"))


def _c4_vocab(g):
    return pylike.pylike_vocab(rng_for(3, salt=0x70C), 128256)


def _c4_doc(rng, wl):
    # one document in four nests without closing, so that prefixes reach
    # stack depths up to about 200
    if rng.random() < 0.25:
        return pylike.deep_program(rng, approx_chars=int(rng.integers(150, 520)))
    return pylike.program(rng)


PYLIKE = _register(Workload(
    3, "pylike", B=128, steps=500, logits_dtype="bf16", logits_std=2.0,
    make_grammar=pylike.grammar, make_vocab=_c4_vocab, make_document=_c4_doc, doc_pool=2048,
    description="Python-like CFG (96 terminals, 144 nonterminals, 14 binary precedence levels, INDENT/DEDENT); "
                "a quarter of the documents nest without closing (stack depth up to ~200); "
                "V=128,256; B=128; bf16 N(0,2)"))


class _DeepWorkload(Workload):
    """Prefixes that reach a target stack depth d ~ U{1..1000}: the first
    position of a deeply nesting program where the stack has d symbols, then
    a cut a few bytes further (inside the next lexeme more often than not)."""

    @functools.cached_property
    def depth_profiles(self) -> list:
        return [self.host.depths(d) for d in self.documents]

    def prefix(self, step: int, b: int) -> bytes:
        rng = rng_for(self.index, step, b)
        i = int(rng.integers(0, self.doc_pool))
        doc, prof = self.documents[i], self.depth_profiles[i]
        d = int(rng.integers(1, 1001))
        p = int(np.argmax(prof >= d)) if (prof >= d).any() else len(doc)
        cut = min(len(doc), p + int(rng.integers(0, 5)))
        return doc[:cut]


def _c5_vocab(g):
    return pylike_core.pylike_vocab(rng_for(4, salt=0x70C), 262144)


def _c5_doc(rng, wl):
    return pylike_core.deep_program(rng, approx_chars=4500)


STRESS = _register(_DeepWorkload(
    4, "stress", B=256, steps=1000, logits_dtype="bf16", logits_std=2.0,
    make_grammar=pylike_core.grammar, make_vocab=_c5_vocab, make_document=_c5_doc, doc_pool=256,
    description="the core of the Python-like CFG (88 terminals, 80 nonterminals), deep nesting (stack depth "
                "~ U{1..1000}); V=262,144; B=256; bf16 N(0,2)"))


def _c6_vocab(g):
    return gosql.gosql_vocab(rng_for(5, salt=0x70C), 4096)


def _c6_doc(rng, wl):
    return gosql.document(rng)


GOSQL = _register(Workload(
    5, "gosql", B=128, steps=500, logits_dtype="bf16", logits_std=2.0,
    make_grammar=gosql.grammar, make_vocab=_c6_vocab, make_document=_c6_doc, doc_pool=1024,
    description="Go-like language with embedded SQL (296 terminals, 255 nonterminals, 1504 LALR(1) states); "
                "a quarter of the documents nest without closing (stack depth p90 ~200, max ~640); "
                "V=4,096; B=128; bf16 N(0,2)"))


def get(name: str) -> Workload:
    return WORKLOADS[name]
