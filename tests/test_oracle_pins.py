"""Pins for the brute-force oracle, against what the definitions fix.

* exhaustive enumeration of the arithmetic language (independent
  recursive-descent recogniser): mask[v] == [x v is a prefix of a member];
* hand-derived worked examples (tests/golden);
* EOS <=> x is in the language (independent recognisers);
* teacher forcing: the true next token of a valid document is always allowed
  (the paper's correctness methodology, Sec. 4.1 / 4.2);
* every viable prefix has a non-empty mask, and a proper prefix (not in the
  language) has a non-EOS token allowed;
* prefix closure: a token's vocabulary prefixes are allowed when it is
  (Sec. 2.5, vocabulary preprocessing).
"""
import ast
import itertools
import os

import numpy as np
import pytest

from conftest import grammar, host
from inputs import configs, documents
from inputs.seeds import rng_for
from inputs.vocab import Vocab
from oracle import Oracle
from oracle.oracle import unpack
from recognizers import arith_accepts, greedy_tokenize, json_accepts

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "arithmetic_worked_examples.txt")


def _golden_rows():
    rows = []
    for line in open(GOLDEN):
        line = line.rstrip("\n")
        if not line or line.startswith("#"):
            continue
        p, t, e = line.split("\t")
        rows.append((ast.literal_eval(p).encode(), None if t == "EOS" else ast.literal_eval(t).encode(),
                     e == "1"))
    return rows


def test_golden_worked_examples():
    rows = _golden_rows()
    toks = sorted({t for _, t, _ in rows if t is not None})
    v = Vocab(toks + [b""], len(toks))
    o = Oracle(grammar("arithmetic"), v)
    hp = host("arithmetic")
    for prefix, tok, want in rows:
        m = unpack(o.masks([hp.state(prefix)])[0], v.size)
        i = v.eos_id if tok is None else toks.index(tok)
        assert m[i] == want, (prefix, tok, want)


def _open_parens(s: bytes) -> int:
    depth = 0
    for c in s:
        depth += (c == 0x28) - (c == 0x29)
    return max(depth, 0)


@pytest.mark.slow
def test_exhaustive_arithmetic_prefix_language():
    """mask(x)[v] == [x v in Pref(L_<=N)] whenever every viable x v is known to
    complete within N bytes (one digit, then one ')' per open parenthesis)."""
    N = 7
    alphabet = b"01+*() "
    members = [bytes(t) for n in range(N + 1) for t in itertools.product(alphabet, repeat=n)
               if arith_accepts(bytes(t))]
    pref = {m[:i] for m in members for i in range(len(m) + 1)}
    toks = [bytes(t) for n in (1, 2) for t in itertools.product(alphabet, repeat=n)]
    v = Vocab(toks + [b""], len(toks))
    o = Oracle(grammar("arithmetic"), v)
    hp = host("arithmetic")
    xs = [bytes(t) for n in range(5) for t in itertools.product(alphabet, repeat=n)]
    parsed = []
    for x in xs:
        try:
            parsed.append((x, hp.state(x)))
        except ValueError:
            assert x not in pref     # the host parser rejects only non-viable prefixes
    masks = o.masks([s for _, s in parsed])
    checked = 0
    for (x, _), row in zip(parsed, masks):
        m = unpack(row, v.size)
        assert m[v.eos_id] == arith_accepts(x), x
        for i, t in enumerate(toks):
            y = x + t
            if len(y) + 1 + _open_parens(y) <= N:
                assert m[i] == (y in pref), (x, t)
                checked += 1
    assert checked > 20000


def _c1_c2_cases(name, n_steps):
    wl = configs.get(name)
    out = []
    for step in range(n_steps):
        for b in range(wl.B):
            out.append(wl.prefix(step, b))
    return wl, out


@pytest.mark.parametrize("name,n_steps", [("arithmetic", 200), ("json", 8)])
def test_eos_iff_member_and_nonempty(name, n_steps):
    wl, prefixes = _c1_c2_cases(name, n_steps)
    accepts = arith_accepts if name == "arithmetic" else json_accepts
    o = Oracle(wl.grammar, wl.vocab)
    states = [wl.host.state(p) for p in prefixes]
    masks = o.masks(states)
    for p, row in zip(prefixes, masks):
        m = unpack(row, wl.V)
        assert m[wl.vocab.eos_id] == accepts(p), p
        assert m.any(), p
        if not accepts(p):
            assert m[:wl.vocab.eos_id].any(), p


@pytest.mark.parametrize("name,n_docs", [("arithmetic", 60), ("json", 6)])
def test_teacher_forcing_never_rejects_the_true_token(name, n_docs):
    wl = configs.get(name)
    o = Oracle(wl.grammar, wl.vocab)
    rng = rng_for(wl.index, salt=0x7EAC)
    for _ in range(n_docs):
        doc = wl.make_document(rng, wl)
        ids = greedy_tokenize(doc, wl.vocab.tokens, wl.vocab.eos_id)
        cuts = np.cumsum([0] + [len(wl.vocab.tokens[i]) for i in ids])
        states = wl.host.states_at(doc, cuts)
        masks = o.masks(states)
        for k, tok in enumerate(ids + [wl.vocab.eos_id]):
            assert unpack(masks[k], wl.V)[tok], (doc[:cuts[k]], wl.vocab.tokens[tok])


@pytest.mark.parametrize("name,n_steps", [("arithmetic", 100), ("json", 4)])
def test_prefix_closure(name, n_steps):
    wl, prefixes = _c1_c2_cases(name, n_steps)
    toks = wl.vocab.tokens
    index = {t: i for i, t in enumerate(toks) if t}
    # for every token, its longest proper prefix that is also a token
    parent = np.full(len(toks), -1)
    for i, t in enumerate(toks):
        for L in range(len(t) - 1, 0, -1):
            j = index.get(t[:L])
            if j is not None:
                parent[i] = j
                break
    o = Oracle(wl.grammar, wl.vocab)
    masks = o.masks([wl.host.state(p) for p in prefixes])
    has = parent >= 0
    for row in masks:
        m = unpack(row, wl.V)
        assert not (m[has] & ~m[parent[has]]).any()


def test_equal_states_give_equal_rows():
    hp = host("arithmetic")
    a, b = hp.state(b"1+2"), hp.state(b"(3)+4")
    assert a[0] == b[0] and np.array_equal(a[1], b[1])
    wl = configs.get("arithmetic")
    o = Oracle(wl.grammar, wl.vocab)
    m = o.masks([a, b])
    assert np.array_equal(m[0], m[1])


def test_token_bits_agree_with_full_masks():
    wl = configs.get("json")
    o = Oracle(wl.grammar, wl.vocab)
    st = wl.host.state(wl.prefix(0, 3))
    full = unpack(o.masks([st])[0], wl.V)
    rng = np.random.default_rng(5)
    toks = rng.integers(0, wl.V, size=2000)
    assert np.array_equal(o.token_bits(st, toks), full[toks])


def _mutated(rng, doc: bytes, alphabet: bytes) -> bytes:
    b = bytearray(doc)
    for _ in range(int(rng.integers(1, 4))):
        op, i = int(rng.integers(3)), int(rng.integers(0, len(b) + 1))
        ch = alphabet[int(rng.integers(len(alphabet)))]
        if op == 0 and len(b):
            del b[min(i, len(b) - 1)]
        elif op == 1:
            b[i:i] = bytes([ch])
        elif len(b):
            b[min(i, len(b) - 1)] = ch
    return bytes(b)


@pytest.mark.parametrize("name,n_docs", [("arithmetic", 150), ("json", 12)])
def test_teacher_forcing_rejects_negative_samples(name, n_docs):
    """The RQ1 method's other half (Sec. 4.2): an invalid document, fed token
    by token (greedy tokenisation) and then EOS, is rejected at some step.
    Documents are mutated copies of valid ones, kept when the independent
    recogniser says they are not in the language.  The oracle's masks and
    the classifier's host walk decide every step identically."""
    from paper_2608_03065_amd.psc import Classifier
    wl = configs.get(name)
    accepts = arith_accepts if name == "arithmetic" else json_accepts
    alphabet = b"0123456789+*() " if name == "arithmetic" else b'{}[],:"\\ 0123456789.eE-+tfnaulrsx\x01'
    o = Oracle(wl.grammar, wl.vocab)
    clf = Classifier(wl.grammar, wl.vocab)
    rng = rng_for(wl.index, salt=0xBAD)
    negatives = 0
    while negatives < n_docs:
        doc = _mutated(rng, wl.make_document(rng, wl), alphabet)
        if accepts(doc):
            continue
        negatives += 1
        st, rejected = (0, np.array([0], np.int32)), False
        for tok in greedy_tokenize(doc, wl.vocab.tokens, wl.vocab.eos_id) + [wl.vocab.eos_id]:
            row = o.masks([st])[0]
            assert np.array_equal(clf.masks_host([st])[0], row), doc
            if not unpack(row, wl.V)[tok]:
                rejected = True
                break
            code, st = o.advance(st, tok)
            assert code == Oracle.ADVANCED, doc
        assert rejected, doc


def test_json_masks_equal_prefix_language():
    """On the JSON workload, token v is allowed after x exactly when x v is
    the beginning of some JSON document, decided by an independent
    prefix-mode recogniser written from the JSON grammar; EOS exactly when
    x is a document.  Every single-byte token and 1,500 random multi-byte
    ones, after 48 prefixes of the workload (cut to at most 120 bytes)."""
    from recognizers import json_viable_prefix
    wl = configs.get("json")
    o = Oracle(wl.grammar, wl.vocab)
    toks = wl.vocab.tokens
    rng = np.random.default_rng(0x150)
    pick = np.unique(np.concatenate([[i for i, t in enumerate(toks) if len(t) == 1],
                                     rng.integers(0, wl.V - 1, 1500)]))
    prefixes = [wl.prefix(s, b)[:120] for s in range(3) for b in range(wl.B)]
    masks = o.masks([wl.host.state(x) for x in prefixes])
    for x, row in zip(prefixes, masks):
        m = unpack(row, wl.V)
        assert m[wl.vocab.eos_id] == json_accepts(x), x
        want = np.array([json_viable_prefix(x + toks[i]) for i in pick])
        bad = pick[m[pick] != want]
        assert bad.size == 0, (x, [toks[i] for i in bad[:5]])
