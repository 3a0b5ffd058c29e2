"""Independent recognisers used to pin the front end and the oracle.

They are written directly from the language definitions (the arithmetic
expression grammar with spaces, and JSON over bytes), with no lexer DFA and
no LR tables, so a mistake in either of those shows up as a disagreement.
"""
from __future__ import annotations


# ---------------------------------------------------------------- arithmetic

def arith_tokens(s: bytes):
    """Split into NUM runs and single-character operators; spaces separate.
    Returns None on a character outside the language's alphabet."""
    out = []
    i = 0
    n = len(s)
    while i < n:
        c = s[i]
        if c == 0x20:
            i += 1
        elif 0x30 <= c <= 0x39:
            j = i
            while j < n and 0x30 <= s[j] <= 0x39:
                j += 1
            out.append("N")
            i = j
        elif c in b"+*()":
            out.append(chr(c))
            i += 1
        else:
            return None
    return out


def arith_accepts(s: bytes) -> bool:
    """Recursive descent for E -> T ('+' T)*, T -> F ('*' F)*, F -> '(' E ')' | N."""
    toks = arith_tokens(s)
    if toks is None:
        return False
    pos = 0

    def peek():
        return toks[pos] if pos < len(toks) else None

    def E():
        nonlocal pos
        if not T():
            return False
        while peek() == "+":
            pos += 1
            if not T():
                return False
        return True

    def T():
        nonlocal pos
        if not F():
            return False
        while peek() == "*":
            pos += 1
            if not F():
                return False
        return True

    def F():
        nonlocal pos
        t = peek()
        if t == "N":
            pos += 1
            return True
        if t == "(":
            pos += 1
            if not E() or peek() != ")":
                return False
            pos += 1
            return True
        return False

    return E() and pos == len(toks)


# ---------------------------------------------------------------------- JSON

_WS = b" \t\n\r"
_ESC = b'"\\/bfnrt'
_HEX = b"0123456789abcdefABCDEF"


class _JP:
    def __init__(self, s: bytes):
        self.s = s
        self.i = 0

    def ws(self):
        while self.i < len(self.s) and self.s[self.i] in _WS:
            self.i += 1

    def lit(self, word: bytes) -> bool:
        if self.s.startswith(word, self.i):
            self.i += len(word)
            return True
        return False

    def string(self) -> bool:
        s = self.s
        if self.i >= len(s) or s[self.i] != 0x22:
            return False
        self.i += 1
        while self.i < len(s):
            c = s[self.i]
            if c == 0x22:
                self.i += 1
                return True
            if c < 0x20:
                return False
            if c == 0x5C:
                if self.i + 1 >= len(s):
                    return False
                e = s[self.i + 1]
                if e in _ESC:
                    self.i += 2
                elif e == 0x75:
                    h = s[self.i + 2:self.i + 6]
                    if len(h) != 4 or any(ch not in _HEX for ch in h):
                        return False
                    self.i += 6
                else:
                    return False
            else:
                self.i += 1
        return False

    def digits(self) -> int:
        j = self.i
        while self.i < len(self.s) and 0x30 <= self.s[self.i] <= 0x39:
            self.i += 1
        return self.i - j

    def number(self) -> bool:
        s = self.s
        if self.i < len(s) and s[self.i] == 0x2D:
            self.i += 1
        if self.i < len(s) and s[self.i] == 0x30:
            self.i += 1
        elif self.i < len(s) and 0x31 <= s[self.i] <= 0x39:
            self.digits()
        else:
            return False
        if self.i < len(s) and s[self.i] == 0x2E:
            self.i += 1
            if self.digits() == 0:
                return False
        if self.i < len(s) and s[self.i] in b"eE":
            self.i += 1
            if self.i < len(s) and s[self.i] in b"+-":
                self.i += 1
            if self.digits() == 0:
                return False
        return True

    def value(self) -> bool:
        self.ws()
        if self.i >= len(self.s):
            return False
        c = self.s[self.i]
        if c == 0x7B:
            self.i += 1
            self.ws()
            if self.lit(b"}"):
                return True
            while True:
                self.ws()
                if not self.string():
                    return False
                self.ws()
                if not self.lit(b":"):
                    return False
                if not self.value():
                    return False
                self.ws()
                if self.lit(b"}"):
                    return True
                if not self.lit(b","):
                    return False
        if c == 0x5B:
            self.i += 1
            self.ws()
            if self.lit(b"]"):
                return True
            while True:
                if not self.value():
                    return False
                self.ws()
                if self.lit(b"]"):
                    return True
                if not self.lit(b","):
                    return False
        if c == 0x22:
            return self.string()
        if c == 0x2D or 0x30 <= c <= 0x39:
            return self.number()
        return self.lit(b"true") or self.lit(b"false") or self.lit(b"null")


def json_accepts(s: bytes) -> bool:
    p = _JP(s)
    if not p.value():
        return False
    p.ws()
    return p.i == len(s)


class _End(Exception):
    """The text ended where the document could still go on."""


class _JPrefix:
    """JSON read in prefix mode: running out of text anywhere a document
    could continue means the text is a viable prefix."""

    def __init__(self, s: bytes):
        self.s = s
        self.i = 0

    def peek(self) -> int:
        if self.i >= len(self.s):
            raise _End
        return self.s[self.i]

    def ws(self):
        while self.i < len(self.s) and self.s[self.i] in _WS:
            self.i += 1

    def lit(self, word: bytes) -> bool:
        rest = self.s[self.i:self.i + len(word)]
        if rest == word:
            self.i += len(word)
            return True
        if len(rest) < len(word) and word.startswith(rest):
            raise _End
        return False

    def string(self) -> bool:
        if self.peek() != 0x22:
            return False
        self.i += 1
        while True:
            c = self.peek()
            if c == 0x22:
                self.i += 1
                return True
            if c < 0x20:
                return False
            self.i += 1
            if c != 0x5C:
                continue
            e = self.peek()
            self.i += 1
            if e == 0x75:
                for _ in range(4):
                    if self.peek() not in _HEX:
                        return False
                    self.i += 1
            elif e not in _ESC:
                return False

    def digits(self) -> int:
        n = 0
        while self.i < len(self.s) and 0x30 <= self.s[self.i] <= 0x39:
            self.i += 1
            n += 1
        return n

    def number(self) -> bool:
        if self.peek() == 0x2D:
            self.i += 1
        c = self.peek()
        if c == 0x30:
            self.i += 1
        elif 0x31 <= c <= 0x39:
            self.digits()
        else:
            return False
        if self.i < len(self.s) and self.s[self.i] == 0x2E:
            self.i += 1
            if self.digits() == 0:
                self.peek()            # text ends after the point: more digits may come
                return False
        if self.i < len(self.s) and self.s[self.i] in b"eE":
            self.i += 1
            if self.peek() in b"+-":
                self.i += 1
            if self.digits() == 0:
                self.peek()
                return False
        return True

    def value(self) -> bool:
        self.ws()
        c = self.peek()
        if c == 0x7B or c == 0x5B:
            close = b"}" if c == 0x7B else b"]"
            self.i += 1
            self.ws()
            if self.lit(close):
                return True
            while True:
                if c == 0x7B:
                    self.ws()
                    if not self.string():
                        return False
                    self.ws()
                    if not self.lit(b":"):
                        return False
                if not self.value():
                    return False
                self.ws()
                if self.lit(close):
                    return True
                if not self.lit(b","):
                    return False
        if c == 0x22:
            return self.string()
        if c == 0x2D or 0x30 <= c <= 0x39:
            return self.number()
        return self.lit(b"true") or self.lit(b"false") or self.lit(b"null")


def json_viable_prefix(s: bytes) -> bool:
    """Is s the beginning of some JSON document (s itself included)?"""
    p = _JPrefix(s)
    try:
        if not p.value():
            return False
        p.ws()
        return p.i == len(s)
    except _End:
        return True


def greedy_tokenize(text: bytes, tokens: list[bytes], eos_id: int) -> list[int]:
    """Longest-match tokenisation over a vocabulary (teacher forcing)."""
    from inputs.vocab import Vocab
    return Vocab(list(tokens), eos_id).tokenize(text)
