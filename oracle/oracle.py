"""ctypes wrapper of oracle.c (test infrastructure; see the package docstring)."""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = C.CDLL(_LIB)
        P = C.c_void_p
        lib.oracle_new.argtypes = [P, P, P, C.c_int32, C.c_int32]
        lib.oracle_new.restype = P
        lib.oracle_free.argtypes = [P]
        lib.oracle_masks.argtypes = [P, P, P, P, P, C.c_int32, P, C.c_int32]
        lib.oracle_masks.restype = C.c_int
        lib.oracle_token_bits.argtypes = [P, P, C.c_int32, C.c_int32, P, C.c_int64, P]
        lib.oracle_advance.argtypes = [P, C.c_int32, P, C.c_int32, C.c_int32, C.c_int32, P, P, P]
        lib.oracle_advance.restype = C.c_int
        _lib = lib
    return _lib


class _OrGrammar(C.Structure):
    _fields_ = [
        ("n_lex", C.c_int32), ("lex_next", C.c_void_p), ("lex_accept", C.c_void_p),
        ("n_term", C.c_int32), ("ignored", C.c_void_p), ("end_term", C.c_int32),
        ("n_lr", C.c_int32), ("n_nt", C.c_int32), ("action", C.c_void_p), ("go", C.c_void_p),
        ("prod_lhs", C.c_void_p), ("prod_len", C.c_void_p),
    ]


class Oracle:
    """Masks by brute force for one (grammar tables, vocabulary) instance.

    ``grammar`` needs the attributes lexer.next, lexer.accept,
    terminal_ignored, end_terminal, action, goto, prod_lhs, prod_len;
    ``vocab`` needs tokens (list of bytes) and eos_id.
    """

    def __init__(self, grammar, vocab):
        g = grammar
        arrs = [
            np.ascontiguousarray(g.lexer.next, dtype=np.int32),
            np.ascontiguousarray(g.lexer.accept, dtype=np.int32),
            np.ascontiguousarray(g.terminal_ignored, dtype=np.uint8),
            np.ascontiguousarray(g.action, dtype=np.int32),
            np.ascontiguousarray(g.goto, dtype=np.int32),
            np.ascontiguousarray(g.prod_lhs, dtype=np.int32),
            np.ascontiguousarray(g.prod_len, dtype=np.int32),
        ]
        toks = vocab.tokens
        offs = np.zeros(len(toks) + 1, dtype=np.int64)
        np.cumsum([len(t) for t in toks], out=offs[1:])
        blob = np.frombuffer(b"".join(toks) + b"\0", dtype=np.uint8).copy()
        self._keep = arrs + [offs, blob]
        p = [a.ctypes.data for a in arrs]
        self._g = _OrGrammar(arrs[0].shape[0], p[0], p[1], arrs[3].shape[1], p[2],
                             int(g.end_terminal), arrs[3].shape[0], arrs[4].shape[1],
                             p[3], p[4], p[5], p[6])
        self.V = len(toks)
        self.W = (self.V + 31) // 32
        self.eos = int(vocab.eos_id)
        self._ctx = _load().oracle_new(C.addressof(self._g), blob.ctypes.data, offs.ctypes.data,
                                       self.V, self.eos)
        self.threads_used = 0

    def __del__(self):
        if getattr(self, "_ctx", None) and _lib is not None:
            _lib.oracle_free(self._ctx)
            self._ctx = None

    def masks(self, states, n_threads: int = 0) -> np.ndarray:
        """states: list of (q, stack bottom->top) -> uint32 [B, W]."""
        B = len(states)
        qs = np.array([s[0] for s in states], dtype=np.int32)
        lens = np.array([len(s[1]) for s in states], dtype=np.int32)
        offs = np.zeros(B + 1, dtype=np.int64)
        np.cumsum(lens, out=offs[1:])
        stacks = (np.concatenate([np.asarray(s[1], np.int32) for s in states])
                  if B else np.zeros(1, np.int32))
        if stacks.size == 0:
            stacks = np.zeros(1, np.int32)
        out = np.zeros((max(B, 1), self.W), dtype=np.uint32)
        self.threads_used = _load().oracle_masks(
            self._ctx, stacks.ctypes.data, offs.ctypes.data, lens.ctypes.data, qs.ctypes.data,
            B, out.ctypes.data, int(n_threads))
        return out[:B]

    def token_bits(self, state, tokens) -> np.ndarray:
        q, stack = state
        stack = np.ascontiguousarray(stack, dtype=np.int32)
        if stack.size == 0:
            stack = np.zeros(1, np.int32)
            n = 0
        else:
            n = len(state[1])
        toks = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.zeros(len(toks), dtype=np.uint8)
        _load().oracle_token_bits(self._ctx, stack.ctypes.data, n, int(q), toks.ctypes.data,
                                  len(toks), out.ctypes.data)
        return out.astype(bool)

    ADVANCED, REJECTED, EOS_ACCEPTED, OVERFLOW = 0, 1, 2, 3

    def advance(self, state, tok: int, cap: int | None = None):
        """One token on a prefix state: (status, new state or None).  Status
        0 advanced, 1 rejected, 2 EOS accepted (state unchanged), 3 the new
        stack would be longer than cap (default: no practical limit)."""
        q, stack = state
        stack = np.ascontiguousarray(stack, dtype=np.int32)
        n = stack.size
        if cap is None:
            cap = n + 8192
        buf = np.zeros(max(cap, 1), np.int32)
        qo, lo = C.c_int32(0), C.c_int32(0)
        st = _load().oracle_advance(self._ctx, int(q), (stack if n else np.zeros(1, np.int32)).ctypes.data, n,
                                    int(tok), int(cap), C.byref(qo), buf.ctypes.data, C.byref(lo))
        if st != 0:
            return st, None
        return 0, (int(qo.value), buf[:lo.value].copy())


def unpack(mask_row: np.ndarray, V: int) -> np.ndarray:
    """uint32 [W] LSB-first -> bool [V]."""
    bits = np.unpackbits(mask_row.astype("<u4").view(np.uint8), bitorder="little")
    return bits[:V].astype(bool)
