"""Seeded random documents of each workload's language (prefix sources)."""
from __future__ import annotations

import numpy as np


def arithmetic_document(rng: np.random.Generator, max_depth: int = 12) -> bytes:
    """A random derivation of E/T/F with depth <= max_depth, optional spaces."""
    out: list[str] = []

    def sp():
        if rng.random() < 0.25:
            out.append(" " * int(rng.integers(1, 3)))

    def num():
        out.append("".join(str(int(d)) for d in rng.integers(0, 10, size=int(rng.integers(1, 4)))))

    def expr(d):
        if d < max_depth and rng.random() < 0.4:
            expr(d + 1); sp(); out.append("+"); sp(); term(d + 1)
        else:
            term(d + 1)

    def term(d):
        if d < max_depth and rng.random() < 0.4:
            term(d + 1); sp(); out.append("*"); sp(); factor(d + 1)
        else:
            factor(d + 1)

    def factor(d):
        if d < max_depth and rng.random() < 0.3:
            out.append("("); sp(); expr(d + 1); sp(); out.append(")")
        else:
            num()

    sp()
    expr(1)
    sp()
    return "".join(out).encode()


_JSON_ESC = ['\\"', "\\\\", "\\/", "\\b", "\\f", "\\n", "\\r", "\\t"]


def _json_string(rng, words) -> bytes:
    parts = [b'"']
    for _ in range(int(rng.integers(0, 6))):
        r = rng.random()
        if r < 0.6:
            parts.append(words[int(rng.integers(len(words)))])
        elif r < 0.75:
            parts.append(b" ")
        elif r < 0.85:
            parts.append(_JSON_ESC[int(rng.integers(len(_JSON_ESC)))].encode())
        elif r < 0.92:
            parts.append(("\\u%04x" % int(rng.integers(0, 0x10000))).encode())
        else:
            # raw high bytes (not validated as UTF-8)
            parts.append(bytes(rng.integers(0x80, 0x100, size=int(rng.integers(1, 4))).tolist()))
    parts.append(b'"')
    return b"".join(parts)


def _json_number(rng) -> bytes:
    s = "-" if rng.random() < 0.3 else ""
    if rng.random() < 0.2:
        s += "0"
    else:
        s += str(int(rng.integers(1, 10))) + "".join(
            str(int(d)) for d in rng.integers(0, 10, size=int(rng.integers(0, 5))))
    if rng.random() < 0.3:
        s += "." + "".join(str(int(d)) for d in rng.integers(0, 10, size=int(rng.integers(1, 4))))
    if rng.random() < 0.15:
        s += "eE"[int(rng.integers(2))] + ["", "+", "-"][int(rng.integers(3))] + str(int(rng.integers(0, 100)))
    return s.encode()


def json_document(rng: np.random.Generator, words: list[bytes], max_depth: int = 20,
                  budget: int = 160) -> bytes:
    """A random JSON value with nesting depth <= max_depth."""
    out: list[bytes] = []
    left = [budget]

    def ws():
        if rng.random() < 0.3:
            out.append([b" ", b"  ", b"\n", b"\n  ", b"\t", b"\r\n"][int(rng.integers(6))])

    def value(d):
        left[0] -= 1
        r = rng.random()
        deep_ok = d < max_depth and left[0] > 0
        if deep_ok and r < 0.3:
            obj(d + 1)
        elif deep_ok and r < 0.55:
            arr(d + 1)
        elif r < 0.75:
            out.append(_json_string(rng, words))
        elif r < 0.9:
            out.append(_json_number(rng))
        else:
            out.append([b"true", b"false", b"null"][int(rng.integers(3))])

    def obj(d):
        out.append(b"{"); ws()
        n = int(rng.integers(0, 5))
        for i in range(n):
            if i:
                out.append(b","); ws()
            out.append(_json_string(rng, words)); ws(); out.append(b":"); ws()
            value(d); ws()
        out.append(b"}")

    def arr(d):
        out.append(b"["); ws()
        n = int(rng.integers(0, 5))
        for i in range(n):
            if i:
                out.append(b","); ws()
            value(d); ws()
        out.append(b"]")

    ws()
    # documents start with a container most of the time, as JSON outputs do
    if rng.random() < 0.5:
        obj(1)
    elif rng.random() < 0.6:
        arr(1)
    else:
        value(1)
    ws()
    return b"".join(out)
