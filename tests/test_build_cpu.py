"""CPU checks of the library: exports, argument errors, and the host walk of
the built classifier against the oracle (bit-exact)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from inputs import configs
from inputs.vocab import Vocab
from oracle import Oracle
from paper_2608_03065_amd import psc
from paper_2608_03065_amd.psc import Classifier, PscError


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "psc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(psc_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 10
    lib = psc.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(psc.EXPORTED) == names


@pytest.mark.parametrize("name,steps", [("arithmetic", 200), ("json", 40), ("schema", 6)])
def test_host_walk_matches_oracle(name, steps):
    wl = configs.get(name)
    clf = Classifier(wl.grammar, wl.vocab)
    states = [st for s in range(steps) for st in wl.states(s)]
    got = clf.masks_host(states)
    want = Oracle(wl.grammar, wl.vocab).masks(states)
    bad = np.nonzero((got != want).any(axis=1))[0]
    assert bad.size == 0, f"{bad.size} rows differ, first at {bad[:5]}"


def test_classes_partition_is_consistent_with_oracle():
    # rows that share a class must have identical oracle rows
    wl = configs.get("json")
    clf = Classifier(wl.grammar, wl.vocab)
    states = [st for s in range(40, 60) for st in wl.states(s)]
    cls = clf.classify_host(states)
    want = Oracle(wl.grammar, wl.vocab).masks(states)
    for c in np.unique(cls):
        rows = want[cls == c]
        assert (rows == rows[0]).all()


def test_info_is_consistent():
    wl = configs.get("json")
    inf = Classifier(wl.grammar, wl.vocab).info()
    assert inf["vocab_size"] == wl.V and inf["mask_words"] == (wl.V + 31) // 32
    assert inf["mask_stride_words"] % 64 == 0 and inf["mask_stride_words"] >= inf["mask_words"]
    assert inf["dfa_states"] <= inf["dfa_states_built"]
    assert inf["device_bytes"] >= inf["table_bytes"] + inf["mask_table_bytes"]
    # the sliced layout: distinct 64-word slices plus one id per (row, slice)
    n_slices = inf["mask_stride_words"] // 64
    assert inf["sliced_mask_bytes"] == 4 * (64 * inf["mask_slices_unique"] + inf["n_classes"] * n_slices)
    assert 1 <= inf["mask_slices_unique"] <= inf["n_classes"] * n_slices
    assert inf["sliced_mask_bytes"] < inf["mask_table_bytes"]
    assert inf["bound_mask_layout"] == 0
    # skip edges exist on this grammar, so the host-walk parity tests take them
    assert inf["skip_edges"] > 0
    clf = Classifier(wl.grammar, wl.vocab)
    lib = psc.lib()
    flat, sliced = (lib.psc_device_bytes_ex(clf._h, f) for f in (psc.BIND_FLAT, psc.BIND_SLICED))
    assert flat == lib.psc_device_bytes(clf._h) == lib.psc_device_bytes_ex(clf._h, 0)
    assert flat - sliced >= inf["mask_table_bytes"] - inf["sliced_mask_bytes"] - 512


def test_host_walk_range_faults():
    wl = configs.get("arithmetic")
    clf = Classifier(wl.grammar, wl.vocab)
    good = wl.states(0)[0]
    n_lex = wl.grammar.lexer.n_states
    bad_q = (n_lex, good[1])
    bad_sym = (good[0], np.array([0, wl.grammar.n_lr_states + 5], np.int32))
    cls = clf.classify_host([good, bad_q, bad_sym])
    assert cls[0] >= 0 and cls[1] == -1 and cls[2] == -1


def _tables(wl):
    return wl.grammar


def test_build_rejects_bad_inputs():
    wl = configs.get("arithmetic")
    g = wl.grammar
    # EOS with a spelling
    v = Vocab([b"1", b"+", b"x"], 2)
    with pytest.raises(PscError) as e:
        Classifier(g, v)
    assert e.value.status == -2
    # a non-EOS token with an empty spelling
    v = Vocab([b"1", b"", b""], 2)
    with pytest.raises(PscError) as e:
        Classifier(g, v)
    assert e.value.status == -2

    class Broken:
        pass
    b = Broken()
    b.lexer = type("L", (), {})()
    b.lexer.next = g.lexer.next.copy()
    b.lexer.accept = g.lexer.accept.copy()
    b.lexer.accept[0] = 1                  # q0 accepting is not allowed
    for k in ("terminal_ignored", "end_terminal", "action", "goto", "prod_lhs", "prod_len"):
        setattr(b, k, getattr(g, k))
    with pytest.raises(PscError) as e:
        Classifier(b, wl.vocab)
    assert e.value.status == -2
    b.lexer.accept = g.lexer.accept
    b.action = g.action.copy()
    b.action[0, 0] = (999 << 2) | 1        # shift target out of range
    with pytest.raises(PscError) as e:
        Classifier(b, wl.vocab)
    assert e.value.status == -2


def test_null_arguments():
    lib = psc.lib()
    h = C.c_void_p()
    assert lib.psc_build(None, None, C.byref(h)) == -1
    assert lib.psc_info(None, None) == -1
    assert lib.psc_compute_masks(None, None, None, None, 1, None, None) == -1
    assert lib.psc_apply_mask(None, 0, None, -1, 5, None) == -1
    assert lib.psc_apply_mask(None, 7, None, 1, 5, None) == -1
    assert lib.psc_apply_mask(None, 0, None, 0, 5, None) == 0      # B == 0: no-op
    assert b"null" in lib.psc_last_error() or lib.psc_last_error()


def test_compute_masks_requires_binding():
    wl = configs.get("arithmetic")
    clf = Classifier(wl.grammar, wl.vocab)
    dummy = C.c_int32(0)
    st = psc.lib().psc_compute_masks(clf._h, C.addressof(dummy), C.addressof(dummy), C.addressof(dummy), 1,
                                     C.addressof(dummy), None)
    assert st == -6


def test_build_is_deterministic():
    # class ids and table layout must not depend on thread scheduling
    wl = configs.get("json")
    states = [st for s in range(20) for st in wl.states(s)]
    outs = []
    for _ in range(3):
        clf = Classifier(wl.grammar, wl.vocab)
        inf = clf.info()
        rows = np.stack([clf.class_mask(c) for c in range(inf["n_classes"])])
        outs.append((clf.classify_host(states).tobytes(), rows.tobytes(), inf["table_bytes"]))
    assert outs[0] == outs[1] == outs[2]


def test_binding_rejects_bad_tensors_before_the_library():
    """The binding's argument checks are explicit (they hold under python -O)
    and fire before any call into the library: wrong dtype, shape, layout or
    device (device indices as torch's get_device(): -1 is host memory)."""
    import torch
    from paper_2608_03065_amd import psc
    ok = torch.zeros(4, dtype=torch.int32)
    assert psc._i32(ok, "x", -1, numel=4) is ok
    with pytest.raises(ValueError):
        psc._i32(torch.zeros(4, dtype=torch.int64), "x", -1)
    with pytest.raises(ValueError):
        psc._i32(ok, "x", -1, numel=5)
    with pytest.raises(ValueError):
        psc._i32(torch.zeros((2, 3), dtype=torch.int32), "x", -1, shape=(3, 2))
    with pytest.raises(ValueError):
        psc._i32(torch.zeros((2, 3), dtype=torch.int32).t(), "x", -1)
    with pytest.raises(ValueError):
        psc._i32(ok, "x", 0)                      # host memory where device 0 is bound
    with pytest.raises(ValueError):
        psc._i32([0, 1], "x", -1)
    with pytest.raises(ValueError):
        psc._logits(torch.zeros((2, 5), dtype=torch.float16), -1, 2, 5)
    with pytest.raises(ValueError):
        psc._logits(torch.zeros((2, 4), dtype=torch.float32), -1, 2, 5)
    assert psc._logits(torch.zeros((2, 5), dtype=torch.bfloat16), -1, 2, 5) == psc.PSC_BF16
    # an unbound classifier reports PSC_E_NOT_BOUND, as the library would
    wl = configs.get("arithmetic")
    clf = Classifier(wl.grammar, wl.vocab)
    with pytest.raises(PscError) as e:
        clf.compute_masks(ok, ok, ok)
    assert e.value.status == -6


_OOM_SCRIPT = r"""
import resource, sys
sys.path.insert(0, sys.argv[1])
from inputs import configs
from paper_2608_03065_amd import psc
psc.lib()
wl = configs.get("schema")
G, voc = wl.grammar, wl.vocab
vm = int([l for l in open("/proc/self/status") if l.startswith("VmSize")][0].split()[1]) * 1024
soft, hard = resource.getrlimit(resource.RLIMIT_AS)
resource.setrlimit(resource.RLIMIT_AS, (vm + (16 << 20), hard))
try:
    psc.Classifier(G, voc)
    print("BUILT", flush=True)
except psc.PscError as e:
    print("STATUS", e.status, flush=True)
resource.setrlimit(resource.RLIMIT_AS, (soft, hard))
a = configs.get("arithmetic")
print("AFTER", psc.Classifier(a.grammar, a.vocab).info()["n_lr_states"], flush=True)
"""


def test_build_reports_out_of_memory():
    """An allocation failure inside psc_build (forced with an address-space
    limit of 16 MB above what the process holds, far below what the schema
    construction needs) is PSC_E_OOM, not a crash; the process then builds
    another classifier normally."""
    import subprocess
    import sys
    env = dict(os.environ, PSC_BUILD_THREADS="1")
    r = subprocess.run([sys.executable, "-c", _OOM_SCRIPT, ROOT], capture_output=True, text=True, timeout=300,
                       env=env, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "STATUS -4" in r.stdout and "AFTER 12" in r.stdout, r.stdout


@pytest.mark.parametrize("name,steps", [("arithmetic", 200), ("json", 40), ("schema", 4)])
def test_host_state_matches_input_side_parser(name, steps):
    """psc_host_state on the workloads' prefixes equals the input side's own
    host parser (inputs/hoststate.c), state for state."""
    wl = configs.get(name)
    clf = Classifier(wl.grammar, wl.vocab)
    for s in range(steps):
        for b in range(wl.B):
            text = wl.prefix(s, b)
            q, st = clf.host_state(text)
            q2, st2 = wl.host.state(text)
            assert q == q2 and np.array_equal(st, st2), (s, b, text[-40:])


def test_host_state_matches_oracle_advance():
    """Along greedily tokenised documents, the oracle's one-token advance
    (Sec. 3.2) from the empty prefix reaches, after every token, the state
    psc_host_state computes for the text so far."""
    from inputs.seeds import rng_for
    from recognizers import greedy_tokenize
    wl = configs.get("json")
    clf = Classifier(wl.grammar, wl.vocab)
    orc = Oracle(wl.grammar, wl.vocab)
    rng = rng_for(wl.index, salt=0x4057)
    for _ in range(4):
        doc = wl.make_document(rng, wl)
        st = (0, np.array([0], np.int32))
        text = b""
        for tok in greedy_tokenize(doc, wl.vocab.tokens, wl.vocab.eos_id):
            code, st = orc.advance(st, tok)
            assert code == Oracle.ADVANCED
            text += wl.vocab.tokens[tok]
            q, stack = clf.host_state(text)
            assert q == st[0] and np.array_equal(stack, st[1]), text[-40:]


def test_host_state_errors():
    wl = configs.get("arithmetic")
    clf = Classifier(wl.grammar, wl.vocab)
    q, st = clf.host_state(b"")
    assert q == 0 and st.tolist() == [0]
    # the last lexeme stays pending and is not fed: "1+)" is a prefix state
    # (whose mask is empty), "1+)1" feeds the ")" and fails
    assert clf.host_state(b"1+)")[1].size == 3
    for bad in (b"1+)1", b"()1", b"1 2 ", b"a", b"1+a"):
        with pytest.raises(PscError) as e:
            clf.host_state(bad)
        assert e.value.status == -10, bad
    with pytest.raises(PscError) as e:
        clf.host_state(b"((((((((((1", cap=4)
    assert e.value.status == -7
    with pytest.raises(ValueError):
        clf.host_state("1+2")


def test_probe_library_exports_and_checks_its_arguments():
    """libpsc_probe.so (the dependent-load latency aid) exports what
    include/psc_probe.h declares and rejects bad arguments before any launch
    (no GPU is touched by these calls)."""
    from paper_2608_03065_amd import probe
    src = open(os.path.join(ROOT, "include", "psc_probe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(psc_[a-z_]+)\s*\(", src)))
    assert names == ["psc_probe_chase"]
    L = probe.lib()
    tab = C.create_string_buffer(1024)
    bad = [(2, None, tab, 1, 1, 0, 1, 1), (0, None, None, 1, 1, 0, 1, 1), (0, None, tab, 0, 1, 0, 1, 1),
           (0, None, tab, 1, -1, 0, 1, 1), (0, None, tab, 1, 1, 0, 1, 70000), (0, None, tab, 1, 1, 1, 1, 1),
           (1, None, tab, 1, 1, 0, 1 << 13, 1 << 12)]
    for mode, out, t, n_rows, k, fill, gx, gy in bad:
        assert L.psc_probe_chase(mode, out, C.cast(t, C.c_void_p) if t is not None else None, n_rows, k, fill,
                                 gx, gy, 0, None) == 1      # hipErrorInvalidValue
