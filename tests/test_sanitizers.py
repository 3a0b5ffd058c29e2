"""The host side of the library under AddressSanitizer + UndefinedBehaviour-
Sanitizer, and the construction's thread pool under ThreadSanitizer.

The construction, persistence and grammar-text sources are built with g++ and a sanitizer
into a temporary shared library (no device code: the calls exercised are
the construction, the host walk, the class rows, saving and loading), which
a child Python process loads with the sanitizer runtime preloaded.  The
child compiles the grammars from their text and some malformed ones, builds
the small workloads, random grammars and a keyword grammar with dense rows
and thousands of lexer states, compares the host walk
with the oracle, round-trips the classifier through a file, and loads
damaged files.  Any sanitizer report ends the child with an error.
"""
import os
import subprocess
import sys

import pytest

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
CSRC = os.path.join(ROOT, "paper_2608_03065_amd", "csrc")

_CHILD = r"""
import ctypes as C, os, sys
sys.path[:0] = [sys.argv[2], sys.argv[3]]
import numpy as np
from paper_2608_03065_amd import psc
L = C.CDLL(sys.argv[1])
P, I32 = C.c_void_p, C.c_int32
for name, args in [("psc_build", [P, P, C.POINTER(P)]), ("psc_info", [P, P]),
                   ("psc_classify_host", [P, P, P, P, I32, P]), ("psc_class_mask_host", [P, I32, P]),
                   ("psc_save", [P, C.c_char_p]), ("psc_load", [C.c_char_p, C.POINTER(P)])]:
    getattr(L, name).argtypes = args
    getattr(L, name).restype = C.c_int
L.psc_device_bytes.argtypes = [P]
L.psc_device_bytes.restype = C.c_size_t
L.psc_free.argtypes = [P]
L.psc_free.restype = None
L.psc_last_error.restype = C.c_char_p
L.psc_grammar_compile.argtypes = [C.c_char_p, C.c_size_t, C.POINTER(P)]
L.psc_grammar_compile.restype = C.c_int
L.psc_grammar_view.argtypes = [P, P]
L.psc_grammar_view.restype = C.c_int
L.psc_grammar_symbol_name.argtypes = [P, I32, I32]
L.psc_grammar_symbol_name.restype = C.c_char_p
L.psc_grammar_free.argtypes = [P]
L.psc_grammar_free.restype = None
psc._lib = L                       # host calls only: nothing here binds a device
from inputs import configs
from oracle import Oracle
import test_random_grammars as RG
tmp = sys.argv[4]
cases = [(n, configs.get(n).grammar, configs.get(n).vocab,
          [configs.get(n).host.state(configs.get(n).prefix(s, b)) for s in range(4) for b in range(configs.get(n).B)])
         for n in sys.argv[5].split(",")]
if sys.argv[7] == "1":                 # dense rows, and more lexer states than have start blocks
    import test_limits as TL
    g, vocab, _, states, _ = TL._keywords()
    cases.append(("keywords", g, vocab, states))
for seed, g, vocab, rng in RG._cases(int(sys.argv[6])):
    orc = Oracle(g, vocab)
    cases.append((f"random{seed}", g, vocab, RG._walk_states(orc, vocab, rng, n_walks=3, n_tokens=12)))
for name, g, vocab, states in cases:          # the grammar text front end
    if getattr(g, "text", ""):
        c = psc.CompiledGrammar(g.text)
        assert np.array_equal(c.action, g.action) and np.array_equal(c.lex_next, g.lexer.next), name
for bad in ['%start e\nN: /[0-9]/\ne: e "+" e | N\n', '%start s\nA: /(a/\ns: A\n', '%start s\ns: "a\n',
            '%start s\nA: /a{3,1}/\ns: A\n', '%start s\nA: /[b-a]/\ns: A\n', '%start s\nA: /a\\x4/\ns: A\n']:
    try:
        psc.CompiledGrammar(bad)
        raise SystemExit("accepted " + bad)
    except psc.PscError:
        pass
for name, g, vocab, states in cases:
    clf = psc.Classifier(g, vocab)
    want = Oracle(g, vocab).masks(states)
    assert np.array_equal(clf.masks_host(states), want), name
    path = os.path.join(tmp, name + ".psc")
    clf.save(path)
    back = psc.Classifier.load(path)
    assert np.array_equal(back.masks_host(states), want), name
    raw = open(path, "rb").read()
    for cut in (0, 7, len(raw) // 2, len(raw) - 1):
        open(path, "wb").write(raw[:cut])
        try:
            psc.Classifier.load(path)
            raise SystemExit(f"{name}: a file cut at {cut} bytes was loaded")
        except psc.PscError:
            pass
print("CHILD OK", len(cases), flush=True)
"""


def _build(tmp_path, flags):
    so = str(tmp_path / "libpsc_host.so")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fPIC", "-shared",
                           *flags, f"-I{os.environ.get('ROCM_PATH', '/opt/rocm')}/include",
                           os.path.join(CSRC, "psc_build.cpp"), os.path.join(CSRC, "psc_store.cpp"),
                           os.path.join(CSRC, "psc_grammar.cpp"), "-lz", "-o", so])
    return so


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(p) or not os.path.exists(p):
        pytest.skip(f"{name} is not installed")
    return p


def _run_child(so, preload, env_extra, tmp_path, workloads, n_random, threads, keywords):
    # the C++ runtime is preloaded too, so that the sanitizer's exception
    # interceptors find it at start-up (python itself does not link it)
    env = dict(os.environ, LD_PRELOAD=f"{preload} {_runtime('libstdc++.so.6')}", PSC_BUILD_THREADS=str(threads),
               **env_extra)
    r = subprocess.run([sys.executable, "-c", _CHILD, so, ROOT, TESTS, str(tmp_path), workloads, str(n_random),
                        "1" if keywords else "0"],
                       capture_output=True, text=True, timeout=900, env=env, cwd=ROOT)
    assert r.returncode == 0 and "CHILD OK" in r.stdout, (r.stdout[-2000:], r.stderr[-6000:])


@pytest.mark.slow
def test_host_code_under_asan_and_ubsan(tmp_path):
    so = _build(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"])
    _run_child(so, _runtime("libasan.so"),
               {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1"},
               tmp_path, "arithmetic,json", 8, threads=4, keywords=True)


@pytest.mark.slow
def test_build_thread_pool_under_tsan(tmp_path):
    so = _build(tmp_path, ["-fsanitize=thread"])
    _run_child(so, _runtime("libtsan.so"), {"TSAN_OPTIONS": "halt_on_error=1:report_signal_unsafe=0"},
               tmp_path, "arithmetic,json", 4, threads=8, keywords=False)
