"""psc_save / psc_load: round trips, and rejection of damaged or crafted files
before they can reach the device kernels."""
import ctypes as C
import struct

import numpy as np
import pytest

from inputs import configs
from paper_2608_03065_amd.psc import Classifier, PscError

E_IO, E_FORMAT = -8, -9


@pytest.fixture(scope="module")
def built_host():
    cache = {}

    def get(name):
        if name not in cache:
            wl = configs.get(name)
            cache[name] = (wl, Classifier(wl.grammar, wl.vocab))
        return cache[name]
    return get


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema"])
def test_round_trip(built_host, name, tmp_path):
    wl, clf = built_host(name)
    p1, p2 = tmp_path / "a.psc", tmp_path / "b.psc"
    clf.save(str(p1))
    back = Classifier.load(str(p1))
    a, b = clf.info(), back.info()
    for k in a:
        assert a[k] == b[k], k
    states = [st for s in range(0, 40, 4) for st in wl.states(s)]
    assert np.array_equal(back.classify_host(states), clf.classify_host(states))
    for c in range(0, a["n_classes"], max(1, a["n_classes"] // 64)):
        assert np.array_equal(back.class_mask(c), clf.class_mask(c)), c
    back.save(str(p2))
    assert p1.read_bytes() == p2.read_bytes()


def _sections(raw):
    """(header bytes, [(tag, codec, raw, stored, checksum, offset of data)])."""
    hb = struct.unpack_from("<I", raw, 8)[0]
    out, pos = [], hb
    for _ in range(4):
        tag, codec, n_raw, n_stored, ck = struct.unpack_from("<IIQQQ", raw, pos)
        out.append((tag, codec, n_raw, n_stored, ck, pos + 32))
        pos += 32 + n_stored
    return hb, out


def _fnv1a(b):
    h = 0xcbf29ce484222325
    for x in b:
        h = ((h ^ x) * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h


def _patch_table(raw, fn):
    """Apply fn to the (raw, uncompressed) classifier table and re-checksum."""
    hb, secs = _sections(raw)
    tag, codec, n_raw, n_stored, ck, at = secs[0]
    assert codec == 0, "use a grammar whose table is stored raw"
    t = np.frombuffer(raw[at:at + n_raw], dtype=np.int32).copy()
    fn(t)
    tb = t.tobytes()
    hdr = struct.pack("<IIQQQ", tag, codec, n_raw, n_stored, _fnv1a(tb))
    return raw[:at - 32] + hdr + tb + raw[at + n_raw:]


def _expect(path, code):
    with pytest.raises(PscError) as e:
        Classifier.load(str(path))
    assert e.value.status == code, str(e.value)


def test_damaged_files(built_host, tmp_path):
    wl, clf = built_host("schema")
    p = tmp_path / "s.psc"
    clf.save(str(p))
    raw = p.read_bytes()
    _expect(tmp_path / "missing.psc", E_IO)
    (tmp_path / "magic.psc").write_bytes(b"XXXX" + raw[4:])
    _expect(tmp_path / "magic.psc", E_FORMAT)
    (tmp_path / "short.psc").write_bytes(raw[:len(raw) // 2])
    _expect(tmp_path / "short.psc", E_FORMAT)
    hb, secs = _sections(raw)
    mask = secs[1]
    assert mask[1] == 1, "the mask table is compressed"
    flip = bytearray(raw)
    flip[mask[5] + mask[3] // 2] ^= 0x40
    (tmp_path / "flip.psc").write_bytes(bytes(flip))
    _expect(tmp_path / "flip.psc", E_FORMAT)


@pytest.mark.parametrize("name", ["arithmetic", "json"])
def test_crafted_tables_are_rejected(built_host, tmp_path, name):
    """Checksums intact, structure wrong: the validator must refuse each."""
    wl, clf = built_host(name)
    p = tmp_path / "a.psc"
    clf.save(str(p))
    raw = p.read_bytes()
    info = clf.info()
    n_lex = info["n_lex_states"]

    def first_chain_ref(t):
        for q in range(n_lex):
            if t[q] >= 0 and (t[q] & 3) == 2:
                return q
        raise AssertionError("no start state in a chain")

    cases = {
        "kind 3 ref": lambda t: t.__setitem__(0, (t[0] & ~3) | 3 if t[0] >= 0 else 3),
        "ref past the end": lambda t: t.__setitem__(0, (len(t) + 64) & ~3),
        "class out of range": lambda t: t.__setitem__(0, -info["n_classes"] - 1),
        "ref into the middle of a row": lambda t: t.__setitem__(
            0, next(int(t[q]) for q in range(n_lex) if t[q] >= 0 and (t[q] & 3) == 0) + 4),
        "ref to a jump entry": lambda t: _point_at_jump(t, first_chain_ref(t)),
        "sparse row symbols out of order": lambda t: _sparse_edges(t, n_lex, lambda e: (e[1], e[0])),
        "sparse row symbol out of range": lambda t: _sparse_edges(
            t, n_lex, lambda e: (info["n_lr_states"] + 5, e[1])),
    }
    for case, fn in cases.items():
        bad = tmp_path / "bad.psc"
        bad.write_bytes(_patch_table(raw, fn))
        _expect(bad, E_FORMAT)


def _sparse_edges(t, n_lex, change):
    """Rewrite the first two edge symbols of the first sparse row that has
    at least two edges (every row of this table is sparse)."""
    pos = (n_lex + 3) & ~3
    while int(t[pos + 1]) < 2:
        pos += (8 + 4 * int(t[pos + 1]) + 3) & ~3
    a, b = change((int(t[pos + 8]), int(t[pos + 12])))
    t[pos + 8], t[pos + 12] = a, b


def _point_at_jump(t, q):
    off = t[q] & ~3
    while (int(t[off]) & 0xFFFF) != 0xFFFD:
        off += 4
    t[q] = off | 2


def test_load_then_walk_matches_oracle(built_host, tmp_path):
    """A loaded classifier's host walk gives the oracle's masks."""
    from oracle import Oracle
    wl, clf = built_host("json")
    p = tmp_path / "j.psc"
    clf.save(str(p))
    back = Classifier.load(str(p))
    states = wl.states(5)
    assert np.array_equal(back.masks_host(states), Oracle(wl.grammar, wl.vocab).masks(states))
