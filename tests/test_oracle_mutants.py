"""The oracle's pins catch plausible mistakes in the oracle itself.

Each case copies oracle/oracle.c to a temporary directory, plants one
mistake in the copy (a dropped term, a wrong index or operand, an inverted
condition), builds it with gcc and runs the pins of test_oracle_pins.py
against the mutant.  At least one pin must fail for every mutant; the
unmodified source, built the same way, must pass all of them.  Nothing is
changed in oracle/: the mistakes exist only in the temporary copies.

The mistakes follow the definition the oracle writes out (eq. simp over
the realizable terminal sequences R_q(v) of Sec. 3.1, fed to the LR parser
of Sec. 2.4, with EOS read as membership of x in the language).
"""
import os
import subprocess
import sys

import pytest

import oracle.oracle as om
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(om.__file__), "oracle.c")

# (name, text in oracle.c, replacement, which occurrence (0-based))
MUTANTS = [
    # feed (the parser step): a shift that forgets to push its state
    ("shift_without_push", "if (kind == 1) { view_push(v, a >> 2); return 1; }", "if (kind == 1) { return 1; }", 0),
    # a reduction pops one symbol too few
    ("reduce_pops_one_less", "view_pop(v, g->prod_len[p])", "view_pop(v, g->prod_len[p] - 1)", 0),
    # GOTO taken from the state that was on top before the pop
    ("goto_from_popped_state", "g->go[(int64_t)base * g->n_nt", "g->go[(int64_t)top * g->n_nt", 0),
    # an error entry read as success
    ("error_entry_succeeds", "if (kind == 0) return 0;", "if (kind == 0) return 1;", 0),
    # EOS: the pending lexeme is not fed before $end
    ("eos_skips_pending_lexeme", "if (!g->ignored[t] && !feed(g, v, t)) return 0;\n        }\n        return feed",
     "\n        }\n        return feed", 0),
    # EOS: $end is never fed (any completed lexeme allows EOS)
    ("eos_without_end_marker", "return feed(g, v, g->end_term);", "return 1;", 0),
    # EOS: a pending lexeme that is not a terminal yet is accepted
    ("eos_accepts_unfinished_lexeme", "if (t < 0) return 0;\n            if (!g->ignored[t]",
     "if (t < 0) return 1;\n            if (!g->ignored[t]", 0),
    # end of token: the pending lexeme need not complete to anything
    ("no_completion_check", "if (o->reach_eps[cur]) return 1;", "return 1;", 0),
    # end of token: only the current winner counts, not every reachable one
    ("completion_only_current_winner", "if (!(rs[t / 64] >> (t % 64) & 1)) continue;",
     "if (t != g->lex_accept[cur]) continue;", 0),
    # T_p: one sweep over the lexer states instead of iterating to the fixpoint
    ("completion_one_sweep", "while (changed) {", "for (int sweep = 0; sweep < 1; sweep++) {", 0),
    # T_p: ignored terminals do not make a lexeme completable to nothing
    ("ignored_not_epsilon", "if (g->ignored[t] && (o->reach", "if (0 && (o->reach", 0),
    # the lexer feeds ignored terminals (whitespace) to the parser
    ("ignored_fed_to_parser", "if (!g->ignored[t] && !feed(g, v, t)) return 0;\n        cur",
     "if (!feed(g, v, t)) return 0;\n        cur", 0),
    # after emitting a lexeme, the byte is retried from the old state, not q0
    ("retry_from_old_state", "cur = g->lex_next[c];\n        if (cur < 0) return 0;",
     "cur = g->lex_next[(int64_t)cur * 256 + c];\n        if (cur < 0) return 0;", 0),
    # the token's last byte is not lexed
    ("last_byte_dropped", "for (int64_t i = o->voffs[tok]; i < o->voffs[tok + 1]; i++)",
     "for (int64_t i = o->voffs[tok]; i < o->voffs[tok + 1] - 1; i++)", 0),
    # bits packed MSB-first
    ("msb_first_packing", "word |= 1u << j;", "word |= 1u << (31 - j);", 0),
    # the stack is read from its bottom instead of its top
    ("top_is_bottom", "*out = v->alpha[v->depth - 1];", "*out = v->alpha[0];", 0),
]

# the pins, cheapest first; each raises AssertionError when it fails
BATTERY = [
    ("golden", pins.test_golden_worked_examples),
    ("eos_nonempty_arith", lambda: pins.test_eos_iff_member_and_nonempty("arithmetic", 200)),
    ("teacher_arith", lambda: pins.test_teacher_forcing_never_rejects_the_true_token("arithmetic", 60)),
    ("closure_arith", lambda: pins.test_prefix_closure("arithmetic", 100)),
    ("equal_states", pins.test_equal_states_give_equal_rows),
    ("teacher_json", lambda: pins.test_teacher_forcing_never_rejects_the_true_token("json", 6)),
    ("eos_nonempty_json", lambda: pins.test_eos_iff_member_and_nonempty("json", 8)),
    ("closure_json", lambda: pins.test_prefix_closure("json", 4)),
    ("prefix_language_json", pins.test_json_masks_equal_prefix_language),
    ("exhaustive_arith", pins.test_exhaustive_arithmetic_prefix_language),
]


def _mutate(src: str, old: str, new: str, k: int) -> str:
    at = -1
    for _ in range(k + 1):
        at = src.find(old, at + 1)
        assert at >= 0, f"mutation site not found: {old!r}"
    return src[:at] + new + src[at + len(old):]


def _build(src: str, path) -> str:
    c = path / "oracle.c"
    c.write_text(src)
    so = str(path / "liboracle.so")
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fopenmp", "-shared", "-fPIC", "-o", so, str(c)])
    return so


# Runs the battery in a child process with the oracle library at argv[1]:
# a mutant may also crash or loop, which must not take the test run with it.
_RUNNER = r"""
import sys
sys.path[:0] = [sys.argv[3], sys.argv[4]]
import oracle.oracle as om
om._LIB, om._lib = sys.argv[1], None
import test_oracle_mutants as T
failed = []
for name, pin in T.BATTERY:
    try:
        pin()
    except AssertionError:
        failed.append(name)
        if sys.argv[2] == "first":
            break
print("FAILED:" + ",".join(failed), flush=True)
"""

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)


def _failing_pins(so: str, stop_at_first: bool, timeout: float = 300):
    """Names of the pins that fail with this oracle library; ["crashed"] or
    ["hung"] when the oracle does not finish normally."""
    try:
        r = subprocess.run([sys.executable, "-c", _RUNNER, so, "first" if stop_at_first else "all", ROOT, TESTS],
                           capture_output=True, text=True, timeout=timeout, cwd=ROOT)
    except subprocess.TimeoutExpired:
        return ["hung"]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("FAILED:")]
    if r.returncode != 0 or not lines:
        return ["crashed"]
    return [x for x in lines[-1][len("FAILED:"):].split(",") if x]


def test_unmodified_source_passes_every_pin(tmp_path):
    assert _failing_pins(_build(open(SRC).read(), tmp_path), stop_at_first=False) == []


@pytest.mark.parametrize("name,old,new,k", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new, k):
    src = _mutate(open(SRC).read(), old, new, k)
    assert _failing_pins(_build(src, tmp_path), stop_at_first=True), f"mutant {name} passes every pin"
