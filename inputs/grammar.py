"""Grammar front end: a small builder API -> lexer DFA + LALR(1) tables.

The classifier construction (Algorithm 1) takes the lexer T, the parser P and
the vocabulary as given; this module produces T and P from a grammar written
with the builder below.  The paper uses an off-the-shelf LALR(1) generator and
relies on the correspondence between LR parsers and deterministic PDAs
(Sec. 4.1, "Implementation"); this is our own generator.  It reports every
conflict instead of resolving it, because the method only covers
deterministic grammars (Sec. 5.3, threats to validity).

Symbols in rule bodies:
  * ``'"text"'``  a literal terminal (declared on first use),
  * ``NAME``      a terminal declared with :meth:`Grammar.regex` (upper case),
  * ``name``      a nonterminal (lower case).

LR table conventions (the encoding of the int32 action table):
  action & 3 == 0: error;  1: shift to state (action >> 2);
  2: reduce by production (action >> 2);  3: accept (only on ``$END``).
Production 0 is the augmented start production ``$start -> start``.
Reductions are never defaulted: an error entry stays an error.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field

import numpy as np

from .lexgen import LexerTables, TerminalDef, build_lexer, literal_ast, parse_regex

ACT_ERROR, ACT_SHIFT, ACT_REDUCE, ACT_ACCEPT = 0, 1, 2, 3
END = "$END"


class GrammarError(ValueError):
    pass


class ConflictError(GrammarError):
    def __init__(self, msg, conflicts=()):
        super().__init__(msg)
        self.conflicts = list(conflicts)


@dataclass
class GrammarTables:
    """The problem inputs T (lexer) and P (LALR(1) parser) as flat arrays."""
    lexer: LexerTables
    terminal_names: list[str]
    terminal_ignored: np.ndarray      # uint8 [n_terminals]
    end_terminal: int                 # id of $END
    nonterminal_names: list[str]
    action: np.ndarray                # int32 [n_lr_states, n_terminals]
    goto: np.ndarray                  # int32 [n_lr_states, n_nonterminals], -1 = none
    prod_lhs: np.ndarray              # int32 [n_productions]
    prod_len: np.ndarray              # int32 [n_productions]
    productions: list[tuple[str, tuple[str, ...]]] = field(default_factory=list)
    text: str = ""                    # the grammar in the C library's text form (Grammar.to_text)

    @property
    def n_terminals(self) -> int:
        return len(self.terminal_names)

    @property
    def n_lr_states(self) -> int:
        return int(self.action.shape[0])

    @property
    def n_nonterminals(self) -> int:
        return len(self.nonterminal_names)

    def terminal_id(self, name: str) -> int:
        return self.terminal_names.index(name)


class Grammar:
    """Builder for a context-free grammar with a regular lexical layer."""

    def __init__(self, start: str):
        self.start = start
        self._terms: list[TerminalDef] = []
        self._term_index: dict[str, int] = {}
        self._rules: list[tuple[str, tuple[str, ...]]] = []
        self._fresh = itertools.count()

    # ----- terminals -------------------------------------------------------
    def literal(self, text: str, priority: int = 0) -> str:
        name = '"' + text + '"'
        if name not in self._term_index:
            self._add_term(TerminalDef(name, literal_ast(text), priority, True, False))
        return name

    def regex(self, name: str, pattern: str, priority: int = 0) -> str:
        if name in self._term_index:
            raise GrammarError(f"terminal {name} declared twice")
        self._add_term(TerminalDef(name, parse_regex(pattern), priority, False, False, pattern))
        return name

    def ignore(self, name: str, pattern: str) -> str:
        self._add_term(TerminalDef(name, parse_regex(pattern), 0, False, True, pattern))
        return name

    def _add_term(self, t: TerminalDef):
        self._term_index[t.name] = len(self._terms)
        self._terms.append(t)

    # ----- rules -----------------------------------------------------------
    def rule(self, lhs: str, *alternatives):
        """Add ``lhs -> alt`` for every alternative (a list/tuple or a str)."""
        for alt in alternatives:
            if isinstance(alt, str):
                alt = alt.split() if alt.strip() else []
            body = tuple(self._sym(s) for s in alt)
            self._rules.append((lhs, body))
        return lhs

    def _sym(self, s: str) -> str:
        if s.startswith('"') and s.endswith('"') and len(s) >= 2:
            return self.literal(s[1:-1])
        return s

    def fresh(self, stem: str) -> str:
        return f"_{stem}_{next(self._fresh)}"

    # EBNF helpers, expanded left-recursively so stacks stay shallow
    def star(self, sym: str) -> str:
        n = self.fresh("star")
        self.rule(n, [], [n, sym])
        return n

    def plus(self, sym: str) -> str:
        n = self.fresh("plus")
        self.rule(n, [sym], [n, sym])
        return n

    def opt(self, sym: str) -> str:
        n = self.fresh("opt")
        self.rule(n, [], [sym])
        return n

    def sep_by(self, sym: str, sep: str, allow_empty: bool = True) -> str:
        """``sym (sep sym)*``, or empty when allowed."""
        n = self.fresh("sep")
        self.rule(n, [sym], [n, sep, sym])
        if not allow_empty:
            return n
        m = self.fresh("sepopt")
        self.rule(m, [], [n])
        return m

    # ----- text form ---------------------------------------------------------
    def to_text(self) -> str:
        """The grammar in the text form that the C library compiles
        (psc_grammar_compile): every terminal declared in this builder's
        order, so that both front ends number terminals, nonterminals and
        productions alike."""
        out = [f"%start {self.start}"]
        for t in self._terms:
            if t.is_literal:
                lit = _escape_literal(t.name[1:-1])
                out.append(f"%literal {lit} {t.priority}" if t.priority else f"%literal {lit}")
            else:
                _check_name(t.name)
                pat = "/" + _escape_regex(t.pattern) + "/"
                if t.ignored:
                    out.append(f"%ignore {t.name} {pat}")
                else:
                    out.append(f"{t.name}.{t.priority}: {pat}" if t.priority else f"{t.name}: {pat}")
        for lhs, body in self._rules:
            _check_name(lhs)
            items = []
            for sym in body:
                t = self._term_index.get(sym)
                if t is not None and self._terms[t].is_literal:
                    items.append(_escape_literal(sym[1:-1]))
                else:
                    _check_name(sym)
                    items.append(sym)
            out.append(f"{lhs}: " + " ".join(items) if items else f"{lhs}:")
        return "\n".join(out) + "\n"

    # ----- compile ---------------------------------------------------------
    def compile(self) -> GrammarTables:
        terms = self._terms
        lexer = build_lexer(terms)
        term_names = [t.name for t in terms] + [END]
        end_id = len(terms)
        ignored = np.array([1 if t.ignored else 0 for t in terms] + [0], dtype=np.uint8)
        nts: list[str] = []
        nt_index: dict[str, int] = {}
        for lhs, _ in self._rules:
            if lhs not in nt_index:
                nt_index[lhs] = len(nts)
                nts.append(lhs)
        if self.start not in nt_index:
            raise GrammarError(f"start symbol {self.start} has no rules")
        aug = "$start"
        nt_index[aug] = len(nts)
        nts.append(aug)

        def enc(s: str):
            if s in self._term_index:
                t = self._term_index[s]
                if terms[t].ignored:
                    raise GrammarError(f"ignored terminal {s} used in a rule")
                return (True, t)
            if s in nt_index:
                return (False, nt_index[s])
            raise GrammarError(f"undefined symbol {s!r}")

        prods = [(nt_index[aug], ((False, nt_index[self.start]),))]
        prods += [(nt_index[lhs], tuple(enc(s) for s in body)) for lhs, body in self._rules]
        names = [(aug, (self.start,))] + list(self._rules)
        try:
            action, goto = lalr1(prods, len(term_names), len(nts), end_id, nt_index[aug])
        except ConflictError as e:
            det = []
            for s, t, a, b in e.conflicts[:5]:
                rs = [names[x >> 2] for x in (a, b) if (x & 3) == 2]
                det.append(f"state {s} on {term_names[t]}: reductions {rs}")
            raise ConflictError(str(e) + "; " + " | ".join(det), e.conflicts) from None
        return GrammarTables(
            lexer=lexer,
            terminal_names=term_names,
            terminal_ignored=ignored,
            end_terminal=end_id,
            nonterminal_names=nts,
            action=action,
            goto=goto,
            prod_lhs=np.array([p[0] for p in prods], dtype=np.int32),
            prod_len=np.array([len(p[1]) for p in prods], dtype=np.int32),
            productions=names,
            text=self.to_text(),
        )


def _check_name(name: str):
    if not name or not all(c.isascii() and (c.isalnum() or c in "_$") for c in name):
        raise GrammarError(f"{name!r} cannot be written in the text form")


def _escape_literal(text: str) -> str:
    out = []
    for ch in text:
        o = ord(ch)
        if ch in '"\\':
            out.append("\\" + ch)
        elif 0x20 <= o < 0x7F:
            out.append(ch)
        else:
            out.append(f"\\x{o:02x}")
    return '"' + "".join(out) + '"'


def _escape_regex(pattern: str) -> str:
    """Bytes outside printable ASCII as \\xHH and a bare '/' as '\\/'; an
    escape sequence of the pattern is kept as it is."""
    out = []
    i = 0
    while i < len(pattern):
        ch = pattern[i]
        if ch == "\\" and i + 1 < len(pattern):
            nxt = pattern[i + 1]
            out.append("\\" + nxt if 0x20 <= ord(nxt) < 0x7F else f"\\x{ord(nxt):02x}")
            i += 2
            continue
        o = ord(ch)
        if ch == "/":
            out.append("\\/")
        elif 0x20 <= o < 0x7F:
            out.append(ch)
        else:
            out.append(f"\\x{o:02x}")
        i += 1
    return "".join(out)


# --------------------------------------------------------------------------
# LALR(1): LR(0) automaton + DeRemer/Pennello lookahead sets
# --------------------------------------------------------------------------

def lalr1(prods, n_terms: int, n_nts: int, end_id: int, aug_nt: int):
    """Return (action, goto) int32 tables; raise ConflictError on conflicts.

    prods[i] = (lhs_nt, ((is_terminal, id), ...)); prods[0] is the augmented
    start production.
    """
    by_lhs: list[list[int]] = [[] for _ in range(n_nts)]
    for i, (lhs, _) in enumerate(prods):
        by_lhs[lhs].append(i)

    # nullable nonterminals
    nullable = [False] * n_nts
    changed = True
    while changed:
        changed = False
        for lhs, body in prods:
            if not nullable[lhs] and all((not t) and nullable[x] for t, x in body):
                nullable[lhs] = True
                changed = True

    # closure of LR(0) items, memoised per nonterminal
    nt_closure: dict[int, frozenset] = {}

    def closure_nts(nt: int) -> frozenset:
        got = nt_closure.get(nt)
        if got is not None:
            return got
        seen = {nt}
        stack = [nt]
        while stack:
            a = stack.pop()
            for p in by_lhs[a]:
                body = prods[p][1]
                if body and not body[0][0] and body[0][1] not in seen:
                    seen.add(body[0][1])
                    stack.append(body[0][1])
        fs = frozenset(seen)
        nt_closure[nt] = fs
        return fs

    def closure(kernel) -> list[tuple[int, int]]:
        items = list(kernel)
        nts_needed = set()
        for p, d in kernel:
            body = prods[p][1]
            if d < len(body) and not body[d][0]:
                nts_needed |= closure_nts(body[d][1])
        for a in sorted(nts_needed):
            for p in by_lhs[a]:
                items.append((p, 0))
        return items

    start_kernel = frozenset([(0, 0)])
    states = {start_kernel: 0}
    kernels = [start_kernel]
    trans: list[dict] = []      # per state: {(is_term, id): state}
    i = 0
    while i < len(kernels):
        items = closure(kernels[i])
        moves: dict = {}
        for p, d in items:
            body = prods[p][1]
            if d < len(body):
                moves.setdefault(body[d], set()).add((p, d + 1))
        row = {}
        for sym in sorted(moves):
            k = frozenset(moves[sym])
            j = states.get(k)
            if j is None:
                j = len(kernels)
                states[k] = j
                kernels.append(k)
            row[sym] = j
        trans.append(row)
        i += 1
    n_states = len(kernels)

    # nonterminal transitions
    nt_trans = []
    nt_trans_id = {}
    for s in range(n_states):
        for (is_t, x), tgt in trans[s].items():
            if not is_t:
                nt_trans_id[(s, x)] = len(nt_trans)
                nt_trans.append((s, x))

    def run(s: int, body) -> int:
        for sym in body:
            s = trans[s].get(sym, -1)
            if s < 0:
                return -1
        return s

    # DR sets as int bitsets
    DR = [0] * len(nt_trans)
    reads: list[list[int]] = [[] for _ in nt_trans]
    for idx, (p, A) in enumerate(nt_trans):
        r = trans[p][(False, A)]
        bits = 0
        for (is_t, x), _ in trans[r].items():
            if is_t:
                bits |= 1 << x
            elif nullable[x]:
                reads[idx].append(nt_trans_id[(r, x)])
        if p == 0 and A == prods[0][1][0][1]:
            bits |= 1 << end_id
        DR[idx] = bits
    Read = _digraph(reads, DR)

    includes: list[list[int]] = [[] for _ in nt_trans]
    lookback: dict[tuple[int, int], list[int]] = {}
    for idx, (p_prime, B) in enumerate(nt_trans):
        for prod in by_lhs[B]:
            body = prods[prod][1]
            s = p_prime
            for pos, sym in enumerate(body):
                if not sym[0]:
                    rest = body[pos + 1:]
                    if all((not t) and nullable[x] for t, x in rest):
                        includes[nt_trans_id[(s, sym[1])]].append(idx)
                s = trans[s][sym]
            lookback.setdefault((s, prod), []).append(idx)
    Follow = _digraph(includes, Read)

    LA: dict[tuple[int, int], int] = {}
    for key, idxs in lookback.items():
        bits = 0
        for idx in idxs:
            bits |= Follow[idx]
        LA[key] = bits

    action = np.zeros((n_states, n_terms), dtype=np.int64)
    goto = -np.ones((n_states, n_nts), dtype=np.int64)
    conflicts = []
    for s in range(n_states):
        for (is_t, x), tgt in trans[s].items():
            if is_t:
                action[s, x] = (tgt << 2) | ACT_SHIFT
            else:
                goto[s, x] = tgt
        for p, d in closure(kernels[s]):
            if d != len(prods[p][1]):
                continue
            if p == 0:
                want = ACT_ACCEPT
                la = 1 << end_id
            else:
                want = (p << 2) | ACT_REDUCE
                la = LA.get((s, p), 0)
            t = 0
            while la:
                if la & 1:
                    if action[s, t] != ACT_ERROR and action[s, t] != want:
                        conflicts.append((s, t, int(action[s, t]), want))
                    else:
                        action[s, t] = want
                la >>= 1
                t += 1
    if conflicts:
        def show(a):
            k = a & 3
            return ("shift" if k == 1 else "reduce" if k == 2 else "accept") + f" {a >> 2}"
        first = [(s, t, show(a), show(b)) for s, t, a, b in conflicts[:5]]
        raise ConflictError(f"{len(conflicts)} LALR(1) conflicts (state, terminal, action, action): {first}",
                            conflicts)
    return action.astype(np.int32), goto.astype(np.int32)


def _digraph(rel: list[list[int]], init: list[int]) -> list[int]:
    """DeRemer/Pennello digraph: F(x) = init(x) | U{F(y) : x rel y}.

    Iterative Tarjan traversal; every member of a strongly connected
    component gets the union over the component.
    """
    n = len(init)
    F = list(init)
    N = [0] * n                 # 0 = unvisited, INF = finished
    depth = [0] * n
    stack: list[int] = []
    INF = 1 << 60
    for root in range(n):
        if N[root]:
            continue
        work = [(root, 0)]
        while work:
            x, it = work.pop()
            if it == 0:
                stack.append(x)
                depth[x] = len(stack)
                N[x] = depth[x]
            else:
                # returning from the child rel[x][it - 1]
                y = rel[x][it - 1]
                N[x] = min(N[x], N[y])
                F[x] |= F[y]
            succ = rel[x]
            descended = False
            while it < len(succ):
                y = succ[it]
                it += 1
                if N[y] == 0:
                    work.append((x, it))
                    work.append((y, 0))
                    descended = True
                    break
                N[x] = min(N[x], N[y])
                F[x] |= F[y]
            if descended:
                continue
            if N[x] == depth[x]:
                while True:
                    top = stack.pop()
                    N[top] = INF
                    F[top] = F[x]
                    if top == x:
                        break
    return F
