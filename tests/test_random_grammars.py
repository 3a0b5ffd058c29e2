"""Differential test of the construction on random small LALR(1) grammars.

For each seeded random grammar (conflicted ones are skipped) and a random
vocabulary over its characters, prefix states are reached by random walks
of the oracle itself (a random allowed token, then the oracle's one-token
advance), so every state is a viable prefix.  The classifier's masks, from
the host walk (CPU) and from the device (GPU), must equal the oracle's
masks bit for bit.  This exercises the construction (lock-step simulation,
minimisation, early exit, chains and their extension) on grammar shapes
the five workloads do not have: empty productions, right recursion,
nonterminals that derive each other, and tokens spanning several lexemes.
"""
import numpy as np
import pytest

from inputs.grammar import ConflictError, Grammar, GrammarError
from inputs.vocab import Vocab
from oracle import Oracle

CHARS = ["a", "b", "c", "(", ")", ","]


def _random_grammar(rng, compiled=True):
    n_nt = int(rng.integers(2, 6))
    nts = [f"n{i}" for i in range(n_nt)]
    g = Grammar("n0")
    g.ignore("WS", " +")
    g.regex("NUM", "[0-9]+")
    terms = ['"%s"' % c for c in CHARS] + ["NUM"]
    for i, nt in enumerate(nts):
        alts = set()
        for _ in range(int(rng.integers(1, 4))):
            body = [str(rng.choice(nts)) if rng.random() < 0.45 else str(rng.choice(terms))
                    for _ in range(int(rng.integers(0, 5)))]
            alts.add(" ".join(body))
        alts.add(str(rng.choice(terms)))          # every nonterminal derives a terminal
        if i + 1 < n_nt:                          # the next nonterminal is reachable, nested
            alts.add('"(" %s ")"' % nts[i + 1] if rng.random() < 0.5 else "%s %s" % (nts[i + 1], rng.choice(terms)))
        g.rule(nt, *sorted(alts))
    return g.compile() if compiled else g


def _random_vocab(rng):
    toks = [c.encode() for c in CHARS] + [b" ", b"0", b"7", b"42"]
    alphabet = list("abc(),0123 ")
    while len(toks) < 60:
        t = "".join(rng.choice(alphabet) for _ in range(int(rng.integers(2, 5)))).encode()
        if t not in toks:
            toks.append(t)
    return Vocab(tokens=toks + [b""], eos_id=len(toks))


def _walk_states(orc, vocab, rng, n_walks=10, n_tokens=24):
    states = []
    for _ in range(n_walks):
        st = (0, np.array([0], np.int32))
        for _ in range(n_tokens):
            states.append(st)
            m = orc.masks([st])[0]
            allowed = np.nonzero(np.unpackbits(m.astype("<u4").view(np.uint8), bitorder="little")
                                 [:len(vocab.tokens)])[0]
            allowed = allowed[allowed != vocab.eos_id]
            if allowed.size == 0:
                break
            solid = np.array([t for t in allowed if vocab.tokens[t].strip()], np.int64)
            pick = solid if solid.size and rng.random() < 0.85 else allowed
            code, new = orc.advance(st, int(rng.choice(pick)))
            assert code == Oracle.ADVANCED
            st = new
    return states


def _cases(n_grammars):
    out, seed = [], 0
    while len(out) < n_grammars:
        rng = np.random.default_rng(1000 + seed)
        seed += 1
        try:
            g = _random_grammar(rng)
        except (ConflictError, GrammarError):
            continue
        out.append((seed, g, _random_vocab(rng), rng))
    return out


@pytest.fixture(scope="module")
def cases():
    from paper_2608_03065_amd.psc import Classifier
    res = []
    for seed, g, vocab, rng in _cases(48):
        orc = Oracle(g, vocab)
        states = _walk_states(orc, vocab, rng)
        res.append((seed, g, vocab, Classifier(g, vocab), orc, states))
    return res


def test_host_walk_matches_oracle_on_random_grammars(cases):
    n_states = 0
    for seed, g, vocab, clf, orc, states in cases:
        want = orc.masks(states)
        got = clf.masks_host(states)
        bad = np.nonzero((got != want).any(axis=1))[0]
        assert bad.size == 0, (seed, bad[:5])
        n_states += len(states)
    assert n_states > 5000


@pytest.mark.gpu
def test_device_masks_match_oracle_on_random_grammars(cases):
    torch = pytest.importorskip("torch")
    from paper_2608_03065_amd.psc import pack_states
    for seed, g, vocab, clf, orc, states in cases:
        clf.bind("cuda:0")
        stacks, lens, qs = pack_states(states, "cuda:0")
        got = clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32)
        assert np.array_equal(got, orc.masks(states)), seed
        assert clf.error_count() == 0
        del torch
        torch = pytest.importorskip("torch")


@pytest.mark.gpu
def test_device_advance_matches_oracle_on_random_grammars(cases):
    """psc_advance and psc_decode_step on the same states with random
    tokens (allowed or not, EOS included) against the oracle's advance."""
    torch = pytest.importorskip("torch")
    from paper_2608_03065_amd import psc
    from paper_2608_03065_amd.psc import DecodeStates
    cap = 64
    for seed, g, vocab, clf, orc, states in cases:
        clf.bind("cuda:0")
        sel = [states[i] for i in range(0, len(states), max(1, len(states) // 64))][:64]
        rng = np.random.default_rng(seed)
        toks = rng.integers(0, len(vocab.tokens), len(sel)).astype(np.int32)
        ds = DecodeStates(clf, len(sel), cap, "cuda:0").load(sel)
        st = ds.advance(torch.from_numpy(toks).to("cuda:0")).cpu().numpy()
        dd = DecodeStates(clf, len(sel), cap, "cuda:0").load(sel)
        logits = torch.zeros((len(sel), len(vocab.tokens)), dtype=torch.float32, device="cuda:0")
        st2 = dd.decode_step(torch.from_numpy(toks).to("cuda:0"), logits).cpu().numpy()
        got, got2 = ds.host_states(), dd.host_states()
        for b, (s0, t) in enumerate(zip(sel, toks)):
            code, new = orc.advance(s0, int(t), cap)
            want = new if code == Oracle.ADVANCED else s0
            assert st[b] == code and st2[b] == code, (seed, b)
            for q, a in (got[b], got2[b]):
                assert q == want[0] and np.array_equal(a, want[1]), (seed, b)
