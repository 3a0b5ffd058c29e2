"""Schema-conformant JSON: a seeded random schema, its grammar, documents and
vocabulary (stand-in for JSON-schema grammars of the paper's evaluation,
whose schemas are not available here).

Schema: nested objects (3-5 levels), 4-12 required keys per object drawn
from a 2,000-word synthetic lexicon, field types integer / number / boolean
/ string / enum (3-10 values) / nested object / array of objects.

Grammar: each object type T with keys k1..kn (in schema order) is
  obj_T -> "{" mem_T_n "}",  mem_T_1 -> K1 ":" v1,
  mem_T_j -> mem_T_{j-1} "," Kj ":" vj
(left-nested so stacks stay shallow).  Keys and enum values are quoted
literal terminals; a literal beats STRING on the same lexeme, so free
string values never spell a literal (they always carry an upper-case
letter or a digit).
"""
from __future__ import annotations

import functools
from dataclasses import dataclass, field

import numpy as np

from .grammar import Grammar, GrammarTables
from .grammars import JSON_STRING, JSON_WS
from .seeds import rng_for
from .vocab import Vocab, piece_vocab, synthetic_words

INT = r"-?(0|[1-9][0-9]*)"
FLOAT = r"-?(0|[1-9][0-9]*)(\.[0-9]+([eE][+-]?[0-9]+)?|[eE][+-]?[0-9]+)"


@dataclass
class ObjType:
    name: str
    fields: list = field(default_factory=list)   # [(key, kind, arg)]


@dataclass
class Schema:
    root: str
    objects: dict
    lexicon: list

    def literal_words(self) -> set:
        out = set()
        for o in self.objects.values():
            for k, kind, arg in o.fields:
                out.add(k)
                if kind == "enum":
                    out.update(arg)
        return out


def random_schema(rng: np.random.Generator, lexicon: list[bytes]) -> Schema:
    """Nested objects: the deepest branch has 5 levels, every other nested
    branch draws its depth from 3..5; objects above their branch's depth
    nest 1-2 of their fields."""
    objects: dict[str, ObjType] = {}
    words = [w.decode() for w in lexicon]

    def make(level: int, depth: int) -> str:
        name = f"o{len(objects)}"
        obj = ObjType(name)
        objects[name] = obj
        n = int(rng.integers(4, 13))
        keys = [words[i] for i in rng.choice(len(words), size=n, replace=False)]
        n_nest = int(rng.integers(1, 3)) if level < depth else 0
        nest_at = sorted(rng.choice(n, size=min(n_nest, n), replace=False).tolist())
        for i, k in enumerate(keys):
            if i in nest_at:
                # the first nested field continues this branch's depth
                d = depth if i == nest_at[0] else max(level + 1, int(rng.integers(3, 6)))
                child = make(level + 1, min(d, depth))
                kind = "object" if rng.random() < 0.5 else "array"
                obj.fields.append((k, kind, child))
            else:
                r = rng.random()
                if r < 0.22:
                    obj.fields.append((k, "integer", None))
                elif r < 0.36:
                    obj.fields.append((k, "number", None))
                elif r < 0.50:
                    obj.fields.append((k, "boolean", None))
                elif r < 0.78:
                    obj.fields.append((k, "string", None))
                else:
                    m = int(rng.integers(3, 11))
                    vals = [words[j] for j in rng.choice(len(words), size=m, replace=False)]
                    obj.fields.append((k, "enum", vals))
        return name

    root = make(1, 5)
    return Schema(root, objects, words)


def schema_grammar(s: Schema) -> GrammarTables:
    g = Grammar(s.root)
    g.regex("STRING", JSON_STRING)
    g.regex("INT", INT)
    g.regex("FLOAT", FLOAT)
    g.ignore("WS", JSON_WS)
    q = lambda w: g.literal('"' + w + '"')   # a quoted literal terminal
    used_enum: dict[tuple, str] = {}
    for name, o in s.objects.items():
        for j, (k, kind, arg) in enumerate(o.fields):
            if kind == "integer":
                v = "INT"
            elif kind == "number":
                v = "number"
            elif kind == "boolean":
                v = "boolean"
            elif kind == "string":
                v = "STRING"
            elif kind == "enum":
                key = tuple(arg)
                if key not in used_enum:
                    en = f"enum{len(used_enum)}"
                    used_enum[key] = en
                    g.rule(en, *[[q(x)] for x in arg])
                v = used_enum[key]
            elif kind == "object":
                v = arg
            else:
                v = f"arr_{arg}"
            mem = f"{name}_m{j}"
            if j == 0:
                g.rule(mem, [q(k), '":"', v])
            else:
                g.rule(mem, [f"{name}_m{j - 1}", '","', q(k), '":"', v])
        g.rule(name, ['"{"', f"{name}_m{len(o.fields) - 1}", '"}"'])
    for name, o in s.objects.items():
        used_as_array = any(kind == "array" and arg == name
                            for oo in s.objects.values() for (_, kind, arg) in oo.fields)
        if used_as_array:
            g.rule(f"items_{name}", [name], [f"items_{name}", '","', name])
            g.rule(f"arr_{name}", ['"["', '"]"'], ['"["', f"items_{name}", '"]"'])
    g.rule("number", ["INT"], ["FLOAT"])
    g.rule("boolean", ['"true"'], ['"false"'])
    return g.compile()


_WS_CHOICES = [b"", b"", b"", b" ", b"\n  ", b"\n    ", b"  "]


def free_string(rng) -> bytes:
    """A string value that never spells a literal (has upper case / digits)."""
    parts = []
    n = int(rng.integers(1, 4))
    for i in range(n):
        L = int(rng.integers(2, 8))
        letters = rng.integers(0, 26, size=L)
        w = bytes((65 if j == 0 else 97) + int(c) for j, c in enumerate(letters))
        parts.append(w)
        if rng.random() < 0.3:
            parts.append(str(int(rng.integers(0, 1000))).encode())
    body = b" ".join(parts)
    if rng.random() < 0.15:
        body += [b"\\n", b"\\\"", b"\\u00e9", b"\\t"][int(rng.integers(4))]
    return b'"' + body + b'"'


def document(rng: np.random.Generator, s: Schema, max_items: int = 3) -> bytes:
    out: list[bytes] = []
    ws = lambda: out.append(_WS_CHOICES[int(rng.integers(len(_WS_CHOICES)))])

    def obj(name):
        o = s.objects[name]
        out.append(b"{"); ws()
        for j, (k, kind, arg) in enumerate(o.fields):
            if j:
                out.append(b","); ws()
            out.append(b'"' + k.encode() + b'"'); ws(); out.append(b":"); ws()
            if kind == "integer":
                out.append(str(int(rng.integers(-5000, 100000))).encode())
            elif kind == "number":
                if rng.random() < 0.3:
                    out.append(str(int(rng.integers(-100, 1000))).encode())
                else:
                    out.append(f"{rng.normal(0, 100):.{int(rng.integers(1, 5))}f}".encode())
            elif kind == "boolean":
                out.append(b"true" if rng.random() < 0.5 else b"false")
            elif kind == "string":
                out.append(free_string(rng))
            elif kind == "enum":
                out.append(b'"' + arg[int(rng.integers(len(arg)))].encode() + b'"')
            elif kind == "object":
                obj(arg)
            else:
                out.append(b"["); ws()
                n = int(rng.integers(0, max_items + 1))
                for i in range(n):
                    if i:
                        out.append(b","); ws()
                    obj(arg)
                ws(); out.append(b"]")
            ws()
        out.append(b"}")

    obj(s.root)
    return b"".join(out)


def schema_vocab(rng: np.random.Generator, s: Schema, V: int) -> Vocab:
    """Bytes + Zipf-length merged strings over the lexicon, digits, punctuation."""
    lex = [w.encode() for w in s.lexicon]
    quoted = [b'"' + w + b'"' for w in lex[:600]]
    punct = [b"{", b"}", b"[", b"]", b",", b":", b'"', b'":', b'": ', b'","', b'",', b"},", b"}]", b"[{",
             b"{\"", b", \"", b"\\", b".", b"-"]
    digits = [bytes([c]) for c in b"0123456789"]
    spaces = [b" ", b"\n", b"\n  ", b"    ", b"  "]
    caps = [bytes([c]) for c in range(65, 91)]
    lits = [b"true", b"false"]
    pieces = lex + quoted + punct + digits + spaces + caps + lits
    weights = ([0.01] * len(lex) + [0.01] * len(quoted) + [4.0] * len(punct) + [1.5] * len(digits)
               + [2.0] * len(spaces) + [0.15] * len(caps) + [0.5] * len(lits))
    return piece_vocab(rng, V, pieces, weights, zipf_s=1.2, lo=2, hi=16)


@functools.lru_cache(maxsize=None)
def c3_schema(seed_salt: int = 0x5C4E) -> Schema:
    rng = rng_for(2, salt=seed_salt)
    lexicon = synthetic_words(rng, 2000, lo=3, hi=10)
    return random_schema(rng, lexicon)
