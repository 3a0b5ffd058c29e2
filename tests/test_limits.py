"""Maximum sizes and extreme shapes.

CPU: the oracle and the host walk on stacks hundreds of thousands of
symbols deep, from a right-recursive grammar whose mask depends on the
bottom of the stack, pinned to masks worked out by hand and to a fresh
parse of the equivalent short prefix.

GPU (through the C-ABI, against the oracle): the largest batch (B = 65,535,
one grid row per sequence) in the ragged and dense layouts and through the
decoding step; B = 65,536 rejected before any launch; ragged stacks whose
offsets pass 2^31 symbols; a negative length in the ragged layout; and the
deep stacks above (the walk reads every symbol, the advance reduces through
all of them).
"""
import functools

import numpy as np
import pytest

from inputs.grammar import Grammar
from inputs.native import HostParser
from inputs.vocab import Vocab
from oracle import Oracle

DEV = "cuda:0"
B_MAX = 65535
DEEP = 300_000

# tokens of the bracket grammar below
A, OPEN, CLOSE, AA, SPACE, A_CLOSE, EOS = range(7)


@functools.lru_cache(maxsize=None)
def _bracket():
    """s -> "[" l "]" | l ;  l -> "a" l | "a".  After a prefix of a's,
    whether "]" or the end may come next depends on the first symbol of the
    stack, so the classifier reads the whole stack; a closing bracket
    reduces through every a (right recursion)."""
    g = Grammar("s")
    g.ignore("WS", " +")
    g.rule("s", '"[" l "]"', "l")
    g.rule("l", '"a" l', '"a"')
    G = g.compile()
    voc = Vocab(tokens=[b"a", b"[", b"]", b"aa", b" ", b"a]", b""], eos_id=EOS)
    return G, voc, HostParser(G), Oracle(G, voc)


def _allowed(row, V):
    return set(np.nonzero(np.unpackbits(np.asarray(row, "<u4").view(np.uint8), bitorder="little")[:V])[0])


# ------------------------------------------------------------------ CPU

@pytest.mark.parametrize("n", [1, 63, 64, 65, DEEP])
def test_deep_stack_masks_by_hand(n):
    """Inside "[a...a" the next token may continue the a's, close the
    bracket or add space, never open one or end the text; without the
    bracket the end is allowed and "]" is not."""
    G, voc, hp, orc = _bracket()
    from paper_2608_03065_amd.psc import Classifier
    clf = Classifier(G, voc)
    inside, bare = hp.state(b"[" + b"a" * n), hp.state(b"a" * n)
    assert len(inside[1]) == n + 1 and len(bare[1]) == n     # the pending a is not on the stack yet
    want = [{A, CLOSE, AA, SPACE, A_CLOSE}, {A, AA, SPACE, EOS}]
    got = orc.masks([inside, bare])
    assert [_allowed(r, len(voc.tokens)) for r in got] == want
    assert np.array_equal(clf.masks_host([inside, bare]), got)


def test_deep_reduction_chain_matches_short_parse():
    """Closing "[a^n]" (the space ends the "]" lexeme) reduces l -> a l
    n times; the state left is the one a parse of "[a] " reaches."""
    G, voc, hp, orc = _bracket()
    st = hp.state(b"[" + b"a" * DEEP + b"]")
    code, new = orc.advance(st, SPACE, cap=DEEP + 8)
    short = hp.state(b"[a] ")
    assert code == orc.ADVANCED
    assert new[0] == short[0] and np.array_equal(new[1], short[1]) and len(short[1]) == 4


# ------------------------------------------------------------------ GPU

def _closed_form_apply(x, bits, V):
    m = np.unpackbits(bits.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    return np.where(m, x, np.float32(-np.inf)), m


def _closed_form_argmax(x, bits, V):
    masked, m = _closed_form_apply(x, bits, V)
    tok = np.argmax(masked, axis=1).astype(np.int32)       # the first maximum: the lowest id
    tok[~m.any(axis=1)] = -1
    return tok


def _tiled_states(wl, orc):
    distinct = [s for k in range(wl.steps) for s in wl.states(k)]
    want = orc.masks(distinct)
    idx = (np.arange(B_MAX, dtype=np.int64) * 7919) % len(distinct)
    return [distinct[i] for i in idx], want[idx]


@pytest.mark.gpu
def test_max_batch_ragged(built):
    import torch
    from paper_2608_03065_amd.psc import pack_states
    wl, clf, orc = built("arithmetic")
    clf.error_count(reset=True)
    states, want = _tiled_states(wl, orc)
    stacks, lens, qs = pack_states(states, DEV)
    got = clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32)
    assert np.array_equal(got, want)
    assert np.array_equal(clf.compute_classes(stacks, lens, qs).cpu().numpy(), clf.classify_host(states))
    x = (torch.randn(B_MAX, wl.V, generator=torch.Generator().manual_seed(5)) * 2).numpy()
    dev = torch.from_numpy(x).to(DEV)
    bm = torch.empty((B_MAX, clf.W), dtype=torch.int32, device=DEV)
    clf.compute_and_apply(stacks, lens, qs, dev, out=bm)
    want_x, _ = _closed_form_apply(x, want, wl.V)
    assert np.array_equal(dev.cpu().numpy().view(np.uint32), want_x.view(np.uint32))
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), want)
    toks = clf.compute_and_argmax(stacks, lens, qs, torch.from_numpy(x).to(DEV)).cpu().numpy()
    assert np.array_equal(toks, _closed_form_argmax(x, want, wl.V))
    assert clf.error_count() == 0


@pytest.mark.gpu
def test_max_batch_dense_and_decode_step(built):
    """The dense layout at B = 65,535, and the decoding step there (two
    launches at this size) against the advance followed by the dense step."""
    import torch
    from paper_2608_03065_amd import psc
    from paper_2608_03065_amd.psc import DecodeStates
    wl, clf, orc = built("arithmetic")
    clf.error_count(reset=True)
    states, want = _tiled_states(wl, orc)
    cap = max(len(a) for _, a in states) + 64
    ds = DecodeStates(clf, B_MAX, cap, DEV).load(states)
    assert np.array_equal(ds.compute_masks().cpu().numpy().view(np.uint32), want)
    assert np.array_equal(ds.compute_classes().cpu().numpy(), clf.classify_host(states))
    x = (torch.randn(B_MAX, wl.V, generator=torch.Generator().manual_seed(6)) * 2).numpy()
    toks = ds.argmax(torch.from_numpy(x).to(DEV)).cpu().numpy()
    assert np.array_equal(toks, _closed_form_argmax(x, want, wl.V))

    # one allowed token per row (or a skip where none is allowed)
    rng = np.random.default_rng(11)
    unpacked = np.unpackbits(want.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
    tokens = np.full(B_MAX, -1, np.int32)
    for b in range(B_MAX):
        allowed = np.flatnonzero(unpacked[b])
        if allowed.size:
            tokens[b] = rng.choice(allowed)
    t_dev = torch.from_numpy(tokens).to(DEV)
    ref = DecodeStates(clf, B_MAX, cap, DEV).load(states)
    st_ref = ref.advance(t_dev).clone()
    lg_ref = torch.from_numpy(x).to(DEV)
    bm_ref = torch.empty((B_MAX, clf.W), dtype=torch.int32, device=DEV)
    ref.compute_and_apply(lg_ref, out=bm_ref)
    lg = torch.from_numpy(x).to(DEV)
    bm = torch.empty_like(bm_ref)
    st = ds.decode_step(t_dev, lg, out=bm)
    torch.cuda.synchronize()
    assert torch.equal(st, st_ref)
    assert torch.equal(ds.lens, ref.lens) and torch.equal(ds.qs, ref.qs)
    for b in range(0, B_MAX, 997):
        n = int(ref.lens[b])
        assert torch.equal(ds.stacks[b, :n], ref.stacks[b, :n]), b
    assert torch.equal(bm, bm_ref) and torch.equal(lg.view(torch.int32), lg_ref.view(torch.int32))
    # a sample of rows against the oracle's advance
    got = st.cpu().numpy()
    for b in range(0, B_MAX, 4099):
        if tokens[b] < 0:
            assert got[b] == psc.ADV_SKIPPED
            continue
        code, new = orc.advance(states[b], int(tokens[b]), cap)
        n = int(ds.lens[b])
        assert code == orc.ADVANCED and got[b] == psc.ADV_OK, b
        assert int(ds.qs[b]) == new[0] and np.array_equal(ds.stacks[b, :n].cpu().numpy(), new[1]), b
    assert clf.error_count() == 0


@pytest.mark.gpu
def test_batch_above_limit_rejected(built):
    import torch
    from paper_2608_03065_amd.psc import DecodeStates, PscError
    wl, clf, _ = built("arithmetic")
    B = B_MAX + 1
    stacks = torch.zeros(B, dtype=torch.int32, device=DEV)
    lens = torch.ones(B, dtype=torch.int32, device=DEV)
    qs = torch.zeros(B, dtype=torch.int32, device=DEV)
    logits = torch.zeros((B, wl.V), dtype=torch.float32, device=DEV)
    with pytest.raises(PscError):
        clf.compute_masks(stacks, lens, qs)
    with pytest.raises(PscError):
        clf.compute_and_apply(stacks, lens, qs, logits)
    with pytest.raises(PscError):
        clf.compute_and_argmax(stacks, lens, qs, logits)
    ds = DecodeStates(clf, B, 4, DEV)
    with pytest.raises(PscError):
        ds.compute_masks()
    with pytest.raises(PscError):
        ds.decode_step(torch.full((B,), -1, dtype=torch.int32, device=DEV), logits)
    torch.cuda.synchronize()
    assert (logits == 0).all()


@pytest.mark.gpu
def test_ragged_offsets_past_2_31(built):
    """Stack 0 fills 2^31 - 2 symbols (its lexer state is out of range, so it
    is never read); stacks 1 to 3 follow it, the later ones at offsets past
    2^31.  8.6 GB of device memory."""
    import torch
    wl, clf, orc = built("arithmetic")
    clf.error_count(reset=True)
    good = [s for k in range(7, 60) for s in wl.states(k) if len(s[1]) >= 2][:3]
    assert len(good) == 3
    n0 = 2**31 - 2
    total = n0 + sum(len(a) for _, a in good)
    stacks = torch.zeros(total, dtype=torch.int32, device=DEV)
    off = n0
    for _, a in good:
        stacks[off:off + len(a)] = torch.from_numpy(np.asarray(a, np.int32)).to(DEV)
        off += len(a)
    lens = torch.tensor([n0] + [len(a) for _, a in good], dtype=torch.int32, device=DEV)
    qs = torch.tensor([-1] + [q for q, _ in good], dtype=torch.int32, device=DEV)
    want = np.concatenate([np.zeros((1, clf.W), np.uint32), orc.masks(good)])
    got = clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32)
    assert np.array_equal(got, want)
    classes = clf.compute_classes(stacks, lens, qs).cpu().numpy()
    assert classes[0] == -1 and np.array_equal(classes[1:], clf.classify_host(good))
    x = np.random.default_rng(3).standard_normal((len(good) + 1, wl.V)).astype(np.float32)
    toks = clf.compute_and_argmax(stacks, lens, qs, torch.from_numpy(x).to(DEV)).cpu().numpy()
    assert np.array_equal(toks, _closed_form_argmax(x, want, wl.V))
    assert clf.error_count(reset=True) == 3
    del stacks
    torch.cuda.empty_cache()


@pytest.mark.gpu
def test_negative_length_holds_no_symbols(built):
    import torch
    wl, clf, orc = built("json")
    clf.error_count(reset=True)
    good = wl.states(6)[:3]
    stacks = torch.from_numpy(np.concatenate([np.asarray(a, np.int32) for _, a in good])).to(DEV)
    lens = torch.tensor([-5] + [len(a) for _, a in good], dtype=torch.int32, device=DEV)
    qs = torch.tensor([good[0][0]] + [q for q, _ in good], dtype=torch.int32, device=DEV)
    got = clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32)
    assert not got[0].any() and np.array_equal(got[1:], orc.masks(good))
    host = clf.classify_host([(good[0][0], np.zeros(0, np.int32))] + list(good))
    assert np.array_equal(clf.compute_classes(stacks, lens, qs).cpu().numpy(), host)
    assert clf.error_count(reset=True) == 2


@pytest.mark.gpu
def test_deep_right_recursive_stacks():
    """Stacks of 300,000 symbols whose class depends on the bottom symbol:
    ragged and dense masks against the oracle, and one advance per row,
    one of which reduces through every a."""
    import torch
    from paper_2608_03065_amd import psc
    from paper_2608_03065_amd.psc import Classifier, DecodeStates, pack_states
    G, voc, hp, orc = _bracket()
    clf = Classifier(G, voc).bind(DEV)
    states = [hp.state(b"[" + b"a" * DEEP), hp.state(b"a" * DEEP), hp.state(b"[" + b"a" * DEEP + b"]"),
              hp.state(b"[aaaaaaa"), hp.state(b"a" * 64)]
    want = orc.masks(states)
    stacks, lens, qs = pack_states(states, DEV)
    assert np.array_equal(clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32), want)
    assert np.array_equal(clf.compute_classes(stacks, lens, qs).cpu().numpy(), clf.classify_host(states))
    cap = DEEP + 16
    ds = DecodeStates(clf, len(states), cap, DEV).load(states)
    assert np.array_equal(ds.compute_masks().cpu().numpy().view(np.uint32), want)
    tokens = np.array([A, AA, SPACE, CLOSE, EOS], np.int32)
    status = ds.advance(torch.from_numpy(tokens).to(DEV)).cpu().numpy()
    got = ds.host_states()
    codes = {orc.ADVANCED: psc.ADV_OK, orc.REJECTED: psc.ADV_REJECTED, orc.EOS_ACCEPTED: psc.ADV_EOS}
    for b, st in enumerate(states):
        code, new = orc.advance(st, int(tokens[b]), cap)
        assert status[b] == codes[code], b
        if code == orc.ADVANCED:
            assert got[b][0] == new[0] and np.array_equal(got[b][1], new[1]), b
        else:
            assert got[b][0] == st[0] and np.array_equal(got[b][1], st[1]), b
    assert len(got[2][1]) == 4            # the whole chain of a's reduced
    assert clf.error_count() == 0


# ------------------------------------------------- many lexer states

@functools.lru_cache(maxsize=None)
def _keywords():
    """s -> item | s "," item, item -> one of 600 literal 12-letter keywords:
    a lexer of 6,403 states (a trie of the keywords), more than the first
    4,096 that get a start block on the device, so walks start from lexer
    states on both sides of that limit.  The vocabulary has the letters,
    ',' and ' ', pieces of keywords (which end deep in the trie) and EOS."""
    rng = np.random.default_rng(7)
    kws = set()
    while len(kws) < 600:
        kws.add("".join(rng.choice(list("abcdefghijklmnopqrstuvwxyz"), size=12)))
    kws = sorted(kws)
    g = Grammar("s")
    g.ignore("WS", " +")
    g.rule("s", "item", 's "," item')
    g.rule("item", *['"%s"' % k for k in kws])
    G = g.compile()
    toks = [bytes([c]) for c in b"abcdefghijklmnopqrstuvwxyz, "]
    pieces = {k[i:i + n].encode() for k in kws[:200]
              for i, n in [(int(rng.integers(0, 8)), int(rng.integers(2, 6)))]}
    toks += sorted(pieces - set(toks)) + [b""]
    voc = Vocab(tokens=toks, eos_id=len(toks) - 1)
    hp = HostParser(G)
    docs = [",".join(kws[int(x)] for x in rng.integers(0, len(kws), size=3)).encode() for _ in range(256)]
    states = [hp.state(d[:int(rng.integers(1, len(d) + 1))]) for d in docs]
    return G, voc, docs, states, Oracle(G, voc)


def test_many_lexer_states_host_walk():
    G, voc, _, states, orc = _keywords()
    from paper_2608_03065_amd.psc import Classifier
    clf = Classifier(G, voc)
    assert clf.info()["n_lex_states"] > 4096
    qs = np.array([q for q, _ in states])
    assert (qs >= 4096).sum() > 50 and (qs < 4096).sum() > 50
    assert np.array_equal(clf.masks_host(states), orc.masks(states))


@pytest.mark.gpu
def test_many_lexer_states_on_device():
    """The walk from lexer states with and without a start block: masks
    (two-launch and fused paths, ragged stacks), the masked logits, and
    the decoding step (advance, then a walk that reads the pushed states
    from LDS) along the documents, all against the oracle."""
    import torch
    from paper_2608_03065_amd.psc import Classifier, DecodeStates, pack_states
    G, voc, docs, states, orc = _keywords()
    clf = Classifier(G, voc)
    clf.bind(DEV)
    V, B = len(voc.tokens), len(states)
    want = orc.masks(states)
    stacks, lens, qs = pack_states(states, DEV)
    assert np.array_equal(clf.compute_masks(stacks, lens, qs).cpu().numpy().view(np.uint32), want)
    x = torch.randn(B, V, generator=torch.Generator().manual_seed(9))
    lg = x.to(DEV)
    bm = torch.empty((B, clf.W), dtype=torch.int32, device=DEV)
    clf.compute_and_apply(stacks, lens, qs, lg, out=bm)
    assert np.array_equal(bm.cpu().numpy().view(np.uint32), want)
    bits = np.unpackbits(want.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    ref = np.where(bits, x.numpy(), -np.inf).astype(np.float32)
    assert np.array_equal(lg.cpu().numpy().view(np.int32), ref.view(np.int32))
    # decoding along the documents, one token per step
    ids = [voc.tokenize(d) for d in docs]
    cap = 16
    ds = DecodeStates(clf, B, cap, DEV).load([(0, np.array([0], np.int32))] * B)
    host = [(0, np.array([0], np.int32))] * B
    out = torch.empty((B, clf.W), dtype=torch.int32, device=DEV)
    for k in range(max(len(t) for t in ids)):
        tok = np.array([t[k] if k < len(t) else -1 for t in ids], np.int32)
        lg = torch.zeros((B, V), dtype=torch.float32, device=DEV)
        ds.decode_step(torch.from_numpy(tok).to(DEV), lg, out=out)
        for b in range(B):
            if tok[b] >= 0:
                code, new = orc.advance(host[b], int(tok[b]))
                assert code == Oracle.ADVANCED, (b, k)
                host[b] = new
        got = ds.host_states()
        assert all(g[0] == h[0] and np.array_equal(g[1], h[1]) for g, h in zip(got, host)), k
        assert np.array_equal(out.cpu().numpy().view(np.uint32), orc.masks(host)), k
    assert clf.error_count() == 0
