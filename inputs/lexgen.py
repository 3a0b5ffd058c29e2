"""Lexer generator: terminal patterns -> one deterministic lexing automaton.

This builds the problem input T of the paper (the lexing transducer of Sec. 2.1,
defined in Sec. 2.2) from a list of terminal definitions.  It is part of the
seeded-input side of the project: it produces the tables that both the
classifier construction and the brute-force checker take as their given
grammar, and it contains none of the parser-stack-classification arithmetic.

Pipeline: regex text -> AST -> Thompson NFA (one fragment per terminal) ->
subset construction over byte equivalence classes -> Moore minimisation.

Lexing policy (the paper leaves it to the lexer it reuses): bytes are the
input alphabet; the automaton is run with longest match and one byte of
lookahead and never backtracks.  When two terminals match the same longest
lexeme the winner has the higher explicit priority, then a literal beats a
regex, then the earlier declaration wins.  State 0 is q0, the state in which
nothing is pending; minimisation keeps it in a block of its own so that
"state == 0" always means "no pending lexeme".
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

ALL_BYTES = (1 << 256) - 1


# --------------------------------------------------------------------------
# Regex parsing (bytes; a pattern is a Python str whose code points are 0..255)
# --------------------------------------------------------------------------

def _cls(*chars: int) -> int:
    m = 0
    for c in chars:
        m |= 1 << c
    return m


def _range(lo: int, hi: int) -> int:
    return ((1 << (hi + 1)) - 1) ^ ((1 << lo) - 1)


_DIGIT = _range(0x30, 0x39)
_WORD = _DIGIT | _range(0x41, 0x5A) | _range(0x61, 0x7A) | _cls(0x5F)
_SPACE = _cls(0x20, 0x09, 0x0A, 0x0D, 0x0B, 0x0C)
_SIMPLE_ESC = {"n": 0x0A, "t": 0x09, "r": 0x0D, "f": 0x0C, "v": 0x0B, "0": 0x00}


class RegexError(ValueError):
    pass


class _Parser:
    def __init__(self, pat: str):
        self.p = pat
        self.i = 0

    def peek(self):
        return self.p[self.i] if self.i < len(self.p) else None

    def take(self):
        c = self.p[self.i]
        self.i += 1
        return c

    def parse(self):
        node = self.alt()
        if self.i != len(self.p):
            raise RegexError(f"unexpected {self.p[self.i]!r} at {self.i} in {self.p!r}")
        return node

    def alt(self):
        parts = [self.cat()]
        while self.peek() == "|":
            self.take()
            parts.append(self.cat())
        return parts[0] if len(parts) == 1 else ("alt", parts)

    def cat(self):
        parts = []
        while self.peek() is not None and self.peek() not in "|)":
            parts.append(self.repeat())
        if not parts:
            return ("cat", [])
        return parts[0] if len(parts) == 1 else ("cat", parts)

    def repeat(self):
        node = self.atom()
        while True:
            c = self.peek()
            if c == "*":
                self.take(); node = ("star", node)
            elif c == "+":
                self.take(); node = ("plus", node)
            elif c == "?":
                self.take(); node = ("opt", node)
            elif c == "{":
                j = self.p.index("}", self.i)
                body = self.p[self.i + 1:j]
                self.i = j + 1
                if "," in body:
                    a, b = body.split(",", 1)
                    lo = int(a)
                    hi = int(b) if b.strip() else None
                else:
                    lo = hi = int(body)
                node = ("rep", node, lo, hi)
            else:
                return node

    def escape(self, in_class: bool) -> int:
        c = self.take()
        if c in _SIMPLE_ESC:
            return _cls(_SIMPLE_ESC[c])
        if c == "x":
            h = self.p[self.i:self.i + 2]
            self.i += 2
            return _cls(int(h, 16))
        if c == "d":
            return _DIGIT
        if c == "w":
            return _WORD
        if c == "s":
            return _SPACE
        return _cls(ord(c))

    def atom(self):
        c = self.take()
        if c == "(":
            if self.p.startswith("?:", self.i):
                self.i += 2
            node = self.alt()
            if self.peek() != ")":
                raise RegexError(f"missing ) in {self.p!r}")
            self.take()
            return node
        if c == "[":
            return ("set", self.char_class())
        if c == ".":
            return ("set", ALL_BYTES & ~_cls(0x0A))
        if c == "\\":
            return ("set", self.escape(False))
        if c in "*+?{":
            raise RegexError(f"nothing to repeat at {self.i - 1} in {self.p!r}")
        return ("set", _cls(ord(c)))

    def char_class(self) -> int:
        neg = False
        if self.peek() == "^":
            self.take(); neg = True
        m = 0
        first = True
        while True:
            c = self.peek()
            if c is None:
                raise RegexError(f"unterminated class in {self.p!r}")
            if c == "]" and not first:
                self.take()
                break
            first = False
            if c == "\\":
                self.take()
                lo_m = self.escape(True)
            else:
                self.take()
                lo_m = _cls(ord(c))
            if self.peek() == "-" and self.i + 1 < len(self.p) and self.p[self.i + 1] != "]":
                self.take()
                hc = self.take()
                if hc == "\\":
                    hi_m = self.escape(True)
                else:
                    hi_m = _cls(ord(hc))
                lo = lo_m.bit_length() - 1
                hi = hi_m.bit_length() - 1
                if lo_m != 1 << lo or hi_m != 1 << hi or hi < lo:
                    raise RegexError(f"bad range in {self.p!r}")
                m |= _range(lo, hi)
            else:
                m |= lo_m
        return (ALL_BYTES & ~m) if neg else m


def parse_regex(pattern: str):
    return _Parser(pattern).parse()


def literal_ast(text: str):
    return ("cat", [("set", _cls(ord(ch))) for ch in text])


# --------------------------------------------------------------------------
# Thompson NFA
# --------------------------------------------------------------------------

class _NFA:
    def __init__(self):
        self.eps: list[list[int]] = []
        self.edges: list[list[tuple[int, int]]] = []
        self.accept: dict[int, int] = {}

    def new(self) -> int:
        self.eps.append([])
        self.edges.append([])
        return len(self.eps) - 1

    def frag(self, node):
        kind = node[0]
        if kind == "set":
            s, e = self.new(), self.new()
            self.edges[s].append((node[1], e))
            return s, e
        if kind == "cat":
            s = self.new()
            cur = s
            for part in node[1]:
                a, b = self.frag(part)
                self.eps[cur].append(a)
                cur = b
            return s, cur
        if kind == "alt":
            s, e = self.new(), self.new()
            for part in node[1]:
                a, b = self.frag(part)
                self.eps[s].append(a)
                self.eps[b].append(e)
            return s, e
        if kind in ("star", "plus", "opt"):
            s, e = self.new(), self.new()
            a, b = self.frag(node[1])
            self.eps[s].append(a)
            self.eps[b].append(e)
            if kind in ("star", "opt"):
                self.eps[s].append(e)
            if kind in ("star", "plus"):
                self.eps[b].append(a)
            return s, e
        if kind == "rep":
            _, sub, lo, hi = node
            parts = [sub] * lo
            if hi is None:
                parts.append(("star", sub))
            else:
                parts += [("opt", sub)] * (hi - lo)
            return self.frag(("cat", parts))
        raise RegexError(f"bad node {kind}")


# --------------------------------------------------------------------------
# Public data types
# --------------------------------------------------------------------------

@dataclass
class TerminalDef:
    name: str
    ast: object
    priority: int = 0
    is_literal: bool = False
    ignored: bool = False
    pattern: str = ""          # the regex text (regex terminals)


@dataclass
class LexerTables:
    """Deterministic lexer over bytes.

    next: int32 [n_states, 256], -1 where no transition exists.
    accept: int32 [n_states], winning terminal id of an accepting state or -1.
    State 0 is q0 (nothing pending) and is never accepting.
    """
    next: np.ndarray
    accept: np.ndarray
    terminal_names: list[str] = field(default_factory=list)

    @property
    def n_states(self) -> int:
        return int(self.next.shape[0])


def _byte_classes(masks: list[int]) -> tuple[np.ndarray, list[int]]:
    """Partition 0..255 into classes of bytes that no mask distinguishes."""
    sig: dict[tuple, int] = {}
    cls_of = np.zeros(256, dtype=np.int64)
    reps: list[int] = []
    uniq = sorted(set(masks))
    for b in range(256):
        key = tuple((m >> b) & 1 for m in uniq)
        if key not in sig:
            sig[key] = len(reps)
            reps.append(b)
        cls_of[b] = sig[key]
    return cls_of, reps


def build_lexer(terms: list[TerminalDef]) -> LexerTables:
    """Compile terminal definitions into a minimised byte DFA.

    Terminal ids are the indices into ``terms``.
    """
    nfa = _NFA()
    master = nfa.new()
    rank = {}
    for tid, t in enumerate(terms):
        s, e = nfa.frag(t.ast)
        nfa.eps[master].append(s)
        nfa.accept[e] = tid
        # larger rank wins a tie on the same lexeme
        rank[tid] = (t.priority, 1 if t.is_literal else 0, -tid)

    n_nfa = len(nfa.eps)
    masks = [m for row in nfa.edges for (m, _) in row]
    cls_of, reps = _byte_classes(masks)
    n_cls = len(reps)

    # epsilon closures, memoised per NFA state
    closure_cache: dict[int, frozenset] = {}

    def closure_of(state: int) -> frozenset:
        got = closure_cache.get(state)
        if got is not None:
            return got
        seen = {state}
        stack = [state]
        while stack:
            u = stack.pop()
            for v in nfa.eps[u]:
                if v not in seen:
                    seen.add(v)
                    stack.append(v)
        fs = frozenset(seen)
        closure_cache[state] = fs
        return fs

    start = closure_of(master)
    dstates: dict[frozenset, int] = {start: 0}
    order = [start]
    trans: list[list[int]] = []
    accept: list[int] = []
    i = 0
    while i < len(order):
        cur = order[i]
        i += 1
        best = -1
        for s in cur:
            tid = nfa.accept.get(s)
            if tid is not None and (best < 0 or rank[tid] > rank[best]):
                best = tid
        accept.append(best)
        row = [-1] * n_cls
        # gather edges once, then split per byte class
        edges = [(m, v) for u in cur for (m, v) in nfa.edges[u]]
        for c, b in enumerate(reps):
            bit = 1 << b
            tgt = set()
            for m, v in edges:
                if m & bit:
                    tgt |= closure_of(v)
            if not tgt:
                continue
            fs = frozenset(tgt)
            j = dstates.get(fs)
            if j is None:
                j = len(order)
                dstates[fs] = j
                order.append(fs)
            row[c] = j
        trans.append(row)

    T = np.array(trans, dtype=np.int64).reshape(len(order), n_cls)
    A = np.array(accept, dtype=np.int64)
    if A[0] >= 0:
        raise RegexError("a terminal matches the empty string")
    T, A = _prune_dead(T, A)
    T, A = _minimise(T, A)
    nxt = np.where(T[:, cls_of] >= 0, T[:, cls_of], -1).astype(np.int32)
    return LexerTables(next=np.ascontiguousarray(nxt), accept=A.astype(np.int32),
                       terminal_names=[t.name for t in terms])


def _prune_dead(T: np.ndarray, A: np.ndarray):
    """Drop states from which no accepting state is reachable (q0 kept)."""
    n = T.shape[0]
    live = A >= 0
    changed = True
    while changed:
        tgt_live = np.zeros_like(T, dtype=bool)
        ok = T >= 0
        tgt_live[ok] = live[T[ok]]
        new_live = live | tgt_live.any(axis=1)
        changed = bool((new_live != live).any())
        live = new_live
    live[0] = True
    keep = np.nonzero(live)[0]
    remap = -np.ones(n, dtype=np.int64)
    remap[keep] = np.arange(len(keep))
    T2 = T[keep]
    T2 = np.where(T2 >= 0, remap[np.maximum(T2, 0)], -1)
    return T2, A[keep]


def _minimise(T: np.ndarray, A: np.ndarray):
    """Moore refinement; q0 starts in a block of its own and stays state 0."""
    n, k = T.shape
    block = A.copy() + 2          # accepting label blocks (>= 1), -1 -> 1
    block[0] = 0                  # q0 alone
    _, block = np.unique(block, return_inverse=True)
    n_blocks = int(block.max()) + 1
    while True:
        tb = np.where(T >= 0, block[np.maximum(T, 0)], -1)
        sig = np.concatenate([block[:, None], tb], axis=1)
        _, new_block = np.unique(sig, axis=0, return_inverse=True)
        new_block = new_block.reshape(-1)
        nb = int(new_block.max()) + 1
        if nb == n_blocks:
            block = new_block
            break
        block, n_blocks = new_block, nb
    # renumber so q0's block is 0 and the order follows first occurrence
    order = -np.ones(n_blocks, dtype=np.int64)
    nxt_id = 0
    for s in range(n):
        b = block[s]
        if order[b] < 0:
            order[b] = nxt_id
            nxt_id += 1
    block = order[block]
    rep = np.zeros(n_blocks, dtype=np.int64)
    rep[block[::-1]] = np.arange(n)[::-1]
    T2 = T[rep]
    T2 = np.where(T2 >= 0, block[np.maximum(T2, 0)], -1)
    return T2, A[rep]


# --------------------------------------------------------------------------
# Reference lexing helpers (pure Python; small inputs only)
# --------------------------------------------------------------------------

def lex_step(lex: LexerTables, cur: int, byte: int, ignored: set[int]):
    """One byte of the longest-match, one-byte-lookahead rule.

    Returns (new_state, emitted_terminal_or_None); new_state is -1 on a
    lexical error.
    """
    nxt = int(lex.next[cur, byte])
    if nxt >= 0:
        return nxt, None
    if cur != 0 and lex.accept[cur] >= 0:
        t = int(lex.accept[cur])
        nxt = int(lex.next[0, byte])
        return nxt, (None if t in ignored else t)
    return -1, None
