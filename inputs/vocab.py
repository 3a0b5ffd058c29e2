"""Synthetic token vocabularies (byte strings; EOS is the last id, empty spelling).

Real tokenizers are not available, so each vocabulary is built the way BPE
vocabularies look from the outside: every single byte (or every single
character of a small alphabet) is a token, plus many unique longer strings
made by concatenating pieces of the workload's surface syntax, with a Zipf
length distribution.  Spellings are unique; a collision is resampled.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Vocab:
    tokens: list[bytes]          # spellings; tokens[eos_id] == b""
    eos_id: int

    @property
    def size(self) -> int:
        return len(self.tokens)

    def packed(self) -> tuple[np.ndarray, np.ndarray]:
        """(bytes uint8 [sum len], offsets int64 [V+1])."""
        offs = np.zeros(len(self.tokens) + 1, dtype=np.int64)
        np.cumsum([len(t) for t in self.tokens], out=offs[1:])
        blob = np.frombuffer(b"".join(self.tokens), dtype=np.uint8).copy()
        if blob.size == 0:
            blob = np.zeros(1, np.uint8)
        return blob, offs

    def tokenize(self, text: bytes) -> list[int]:
        """Longest-match tokenisation of text over the spellings (teacher
        forcing); raises ValueError if the text cannot be covered."""
        index = self.__dict__.get("_index")
        if index is None:
            index = {t: i for i, t in enumerate(self.tokens) if i != self.eos_id and t}
            self.__dict__["_index"] = index
            self.__dict__["_maxlen"] = max(len(t) for t in index)
        maxlen = self.__dict__["_maxlen"]
        out, i = [], 0
        while i < len(text):
            for L in range(min(maxlen, len(text) - i), 0, -1):
                j = index.get(text[i:i + L])
                if j is not None:
                    out.append(j)
                    i += L
                    break
            else:
                raise ValueError("text not coverable by the vocabulary")
        return out

    def length_histogram(self) -> dict[int, int]:
        h: dict[int, int] = {}
        for t in self.tokens:
            h[len(t)] = h.get(len(t), 0) + 1
        return dict(sorted(h.items()))


def zipf_lengths(rng: np.random.Generator, n: int, s: float, lo: int, hi: int) -> np.ndarray:
    ks = np.arange(lo, hi + 1)
    w = ks.astype(np.float64) ** (-s)
    return rng.choice(ks, size=n, p=w / w.sum())


def synthetic_words(rng: np.random.Generator, n: int, lo: int = 2, hi: int = 9,
                    alphabet: bytes = b"abcdefghijklmnopqrstuvwxyz") -> list[bytes]:
    """n distinct lowercase pseudo-words."""
    out: list[bytes] = []
    seen = set()
    alpha = np.frombuffer(alphabet, dtype=np.uint8)
    while len(out) < n:
        L = int(rng.integers(lo, hi + 1))
        w = bytes(alpha[rng.integers(0, len(alpha), size=L)])
        if w not in seen:
            seen.add(w)
            out.append(w)
    return out


def _fill_unique(rng, base: list[bytes], n_extra: int, make_one) -> list[bytes]:
    seen = set(base)
    out = list(base)
    tries = 0
    while len(out) < len(base) + n_extra:
        t = make_one(rng)
        tries += 1
        if t and t not in seen:
            seen.add(t)
            out.append(t)
        if tries > 50 * (n_extra + 10):
            raise RuntimeError("vocabulary generator cannot find enough unique strings")
    return out


def arithmetic_vocab(rng: np.random.Generator, V: int = 513) -> Vocab:
    """All 15 single characters of the alphabet, unique random strings over
    it with length uniform in 2..8, and EOS."""
    alphabet = b"0123456789+*() "
    singles = [bytes([c]) for c in alphabet]
    alpha = np.frombuffer(alphabet, dtype=np.uint8)

    def one(r):
        L = int(r.integers(2, 9))
        return bytes(alpha[r.integers(0, len(alpha), size=L)])

    toks = _fill_unique(rng, singles, V - 1 - len(singles), one)
    return Vocab(toks + [b""], V - 1)


def piece_vocab(rng: np.random.Generator, V: int, pieces: list[bytes], weights,
                zipf_s: float = 1.2, lo: int = 2, hi: int = 16) -> Vocab:
    """256 single bytes + unique Zipf-length strings cut from concatenated
    random pieces + EOS."""
    singles = [bytes([b]) for b in range(256)]
    w = np.asarray(weights, dtype=np.float64)
    w = w / w.sum()
    n_extra = V - 1 - 256
    lengths = iter(zipf_lengths(rng, 4 * n_extra + 1000, zipf_s, lo, hi).tolist())
    stream: list[int] = []

    def draw() -> int:
        if not stream:
            stream.extend(rng.choice(len(pieces), size=1 << 16, p=w).tolist()[::-1])
        return stream.pop()

    def one(r):
        L = next(lengths)
        buf = bytearray()
        while len(buf) < L:
            buf += pieces[draw()]
        return bytes(buf[:L])

    toks = _fill_unique(rng, singles, n_extra, one)
    return Vocab(toks + [b""], V - 1)


def json_vocab(rng: np.random.Generator, V: int = 32000) -> Vocab:
    """Byte-level JSON vocabulary: punctuation, digits, lowercase words, spaces."""
    words = synthetic_words(rng, 400)
    punct = [b"{", b"}", b"[", b"]", b",", b":", b'"', b'\\', b'\\"', b'\\n', b"-", b".", b"e"]
    digits = [bytes([c]) for c in b"0123456789"]
    spaces = [b" ", b"  ", b"\n", b"\t", b"    "]
    lits = [b"true", b"false", b"null"]
    pieces = punct + digits + words + spaces + lits
    weights = ([6.0] * len(punct) + [2.0] * len(digits) + [0.1] * len(words)
               + [3.0] * len(spaces) + [1.0] * len(lits))
    return piece_vocab(rng, V, pieces, weights)
