"""The device walk against the host walk on stacks no prefix produces.

Both walks read the same automaton (eq. final_c: the class of a (lexer
state, stack) pair, read top-first), so they must agree on any input stack,
valid or not: the same class, or -1 for a symbol out of range that the walk
reaches.  The mutated stacks below drive the walk into the paths valid
prefixes rarely take: a stack cut short at its bottom (a skip over a run of
wildcard chain entries that would cross it falls back to the chain), a
planted out-of-range symbol (inside a skipped run it must still be caught),
and segments repeated into stacks hundreds of symbols deep (runs and chains
that cross the 63-symbol window).  Every call goes through the C-ABI; the
error counter must count exactly the rejected sequences.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import Classifier, DecodeStates, pack_states  # noqa: E402

from test_random_grammars import _cases  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _mutants(states, n_lr, rng):
    out = []
    for q, st in states:
        st = np.asarray(st, np.int32)
        kind = int(rng.integers(4))
        if kind == 0 and len(st) > 1:            # drop a bottom part
            out.append((q, st[int(rng.integers(1, len(st))):].copy()))
        elif kind == 1:                          # plant a symbol out of range
            s = st.copy()
            s[int(rng.integers(len(s)))] = n_lr + int(rng.integers(0, 7))
            out.append((q, s))
        elif kind == 2:                          # repeat a top segment many times
            seg = st[max(0, len(st) - int(rng.integers(1, 12))):]
            out.append((q, np.concatenate([st] + [seg] * int(rng.integers(2, 40))).astype(np.int32)))
        else:
            out.append((q, st.copy()))
    return out


def _check(clf, states):
    clf.error_count(reset=True)
    stacks, lens, qs = pack_states(states, DEV)
    got = clf.compute_classes(stacks, lens, qs).cpu().numpy()
    want = clf.classify_host(states)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad[:8].tolist(), got[bad[:8]].tolist(), want[bad[:8]].tolist())
    assert clf.error_count(reset=True) == int((want < 0).sum())
    # the dense layout and the fused step's bitmask agree too
    cap = max(len(a) for _, a in states) + 1
    dense = DecodeStates(clf, len(states), cap, DEV).load(states).compute_classes().cpu().numpy()
    assert np.array_equal(dense, want)
    bits = clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32)
    for b in range(0, len(states), max(1, len(states) // 16)):
        row = clf.class_mask(int(want[b])) if want[b] >= 0 else np.zeros(clf.W, np.uint32)
        assert np.array_equal(bits[b], row), b
    clf.error_count(reset=True)
    return int((want < 0).sum())


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema", "pylike", "gosql"])
def test_mutated_stacks_device_equals_host(built, name):
    wl, clf, _ = built(name)
    rng = np.random.default_rng(0x5EED + wl.index)
    states = [st for s in range(4) for st in wl.states(3 + 11 * s)]
    n_rejected = _check(clf, _mutants(states, wl.grammar.n_lr_states, rng))
    assert 0 < n_rejected < len(states)


def test_mutated_stacks_on_random_grammars():
    n_skips = 0
    for seed, g, vocab, rng in _cases(24):
        clf = Classifier(g, vocab).bind(DEV)
        n_skips += clf.info()["skip_edges"]
        from oracle import Oracle
        from test_random_grammars import _walk_states
        states = _walk_states(Oracle(g, vocab), vocab, rng, n_walks=6, n_tokens=16)
        _check(clf, _mutants(states, g.n_lr_states, np.random.default_rng(seed)))
    assert n_skips > 0
