"""ctypes wrapper for the input-side host lexer/parser (``hoststate.c``)."""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

from .grammar import GrammarTables

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hoststate.c")
_LIB = os.path.join(_HERE, "_hoststate.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the helper with gcc (always when ``force``)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _HsGrammar(C.Structure):
    _fields_ = [
        ("n_lex", C.c_int32), ("lex_next", C.c_void_p), ("lex_accept", C.c_void_p),
        ("n_term", C.c_int32), ("ignored", C.c_void_p), ("end_term", C.c_int32),
        ("n_lr", C.c_int32), ("n_nt", C.c_int32), ("action", C.c_void_p), ("go", C.c_void_p),
        ("prod_lhs", C.c_void_p), ("prod_len", C.c_void_p),
    ]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = C.CDLL(_LIB)
        P = C.c_void_p
        _lib.hs_prefix_states_at.argtypes = [P, P, C.c_int64, P, C.c_int32, P, P, C.c_int64, P, P]
        _lib.hs_prefix_states_at.restype = C.c_int
        _lib.hs_accepts.argtypes = [P, P, C.c_int64]
        _lib.hs_accepts.restype = C.c_int
        _lib.hs_accepts_batch.argtypes = [P, P, P, C.c_int64, P]
        _lib.hs_viable_batch.argtypes = [P, P, P, C.c_int64, P]
        _lib.hs_depths.argtypes = [P, P, C.c_int64, P]
        _lib.hs_depths.restype = C.c_int
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class HostParser:
    """Prefix -> (lexer state q, parser stack alpha) for one grammar."""

    def __init__(self, g: GrammarTables):
        self.g = g
        self._keep = [
            np.ascontiguousarray(g.lexer.next, dtype=np.int32),
            np.ascontiguousarray(g.lexer.accept, dtype=np.int32),
            np.ascontiguousarray(g.terminal_ignored, dtype=np.uint8),
            np.ascontiguousarray(g.action, dtype=np.int32),
            np.ascontiguousarray(g.goto, dtype=np.int32),
            np.ascontiguousarray(g.prod_lhs, dtype=np.int32),
            np.ascontiguousarray(g.prod_len, dtype=np.int32),
        ]
        k = self._keep
        self._s = _HsGrammar(
            g.lexer.n_states, _ptr(k[0]), _ptr(k[1]), g.n_terminals, _ptr(k[2]), g.end_terminal,
            g.n_lr_states, g.n_nonterminals, _ptr(k[3]), _ptr(k[4]), _ptr(k[5]), _ptr(k[6]))
        self._sp = C.addressof(self._s)

    def states_at(self, text: bytes, cuts) -> list[tuple[int, np.ndarray]]:
        """(q, stack bottom->top) for each prefix text[:cut]; cuts ascending."""
        cuts = np.ascontiguousarray(cuts, dtype=np.int64)
        n = len(cuts)
        cap = 1 << 16
        buf = np.frombuffer(text, dtype=np.uint8) if text else np.zeros(1, np.uint8)
        while True:
            q = np.zeros(n, np.int32)
            lens = np.zeros(n, np.int32)
            offs = np.zeros(n, np.int64)
            st = np.zeros(cap, np.int32)
            rc = lib().hs_prefix_states_at(self._sp, _ptr(buf), len(text), _ptr(cuts), n,
                                           _ptr(q), _ptr(st), cap, _ptr(offs), _ptr(lens))
            if rc == 3 and cap < (1 << 30):
                cap *= 8
                continue
            if rc != 0:
                raise ValueError(f"prefix does not lex/parse (code {rc})")
            return [(int(q[i]), st[offs[i]:offs[i] + lens[i]].copy()) for i in range(n)]

    def state(self, text: bytes) -> tuple[int, np.ndarray]:
        return self.states_at(text, [len(text)])[0]

    def depths(self, text: bytes) -> np.ndarray:
        """Parser stack length after every prefix text[:i], i = 0..len."""
        buf = np.frombuffer(text, dtype=np.uint8) if text else np.zeros(1, np.uint8)
        out = np.zeros(len(text) + 1, np.int32)
        rc = lib().hs_depths(self._sp, _ptr(buf), len(text), _ptr(out))
        if rc != 0:
            raise ValueError(f"text does not lex/parse (code {rc})")
        return out

    def accepts(self, text: bytes) -> bool:
        buf = np.frombuffer(text, dtype=np.uint8) if text else np.zeros(1, np.uint8)
        return bool(lib().hs_accepts(self._sp, _ptr(buf), len(text)))

    def accepts_many(self, texts: list[bytes]) -> np.ndarray:
        return self._batch(lib().hs_accepts_batch, texts)

    def viable_many(self, texts: list[bytes]) -> np.ndarray:
        return self._batch(lib().hs_viable_batch, texts)

    def _batch(self, fn, texts):
        offs = np.zeros(len(texts) + 1, np.int64)
        np.cumsum([len(t) for t in texts], out=offs[1:])
        blob = np.frombuffer(b"".join(texts) or b"\0", dtype=np.uint8)
        out = np.zeros(len(texts), np.uint8)
        fn(self._sp, _ptr(blob), _ptr(offs), len(texts), _ptr(out))
        return out.astype(bool)
