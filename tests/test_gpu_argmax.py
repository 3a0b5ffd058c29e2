"""GPU parity of the masked argmax (greedy decoding folded into the mask
step) against its closed form on the oracle's masks, and a greedy
constrained decoder run entirely on device states."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd import psc  # noqa: E402
from paper_2608_03065_amd.psc import DecodeStates, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _closed_form(logits_cpu, bits, V):
    """Per row: the allowed token with the largest logit (float32 values;
    the first NaN wins; ties to the lowest id); -1 if nothing is allowed."""
    x = logits_cpu.float().numpy()
    out = []
    for b in range(x.shape[0]):
        allowed = np.nonzero(np.unpackbits(bits[b].astype("<u4").view(np.uint8), bitorder="little")[:V])[0]
        if allowed.size == 0:
            out.append(-1)
            continue
        vals = x[b, allowed]
        nan = np.nonzero(np.isnan(vals))[0]
        out.append(int(allowed[nan[0]] if nan.size else allowed[int(np.argmax(vals))]))
    return np.array(out, np.int32)


@pytest.mark.parametrize("name,steps", [("arithmetic", [1, 2, 3]), ("json", [4, 40]), ("schema", [5, 600]),
                                        ("pylike", [7]), ("stress", [9])])
def test_argmax_matches_closed_form(built, name, steps):
    wl, clf, orc = built(name)
    for step in steps:
        states = wl.states(step)
        logits = wl.logits(step)
        stacks, lens, qs = pack_states(states, DEV)
        dev = logits.to(DEV)
        got = clf.compute_and_argmax(stacks, lens, qs, dev).cpu().numpy()
        want = _closed_form(logits, orc.masks(states), wl.V)
        assert np.array_equal(got, want), (step, np.nonzero(got != want)[0][:5])
        assert torch.equal(dev.cpu().view(torch.int16 if dev.dtype == torch.bfloat16 else torch.int32),
                           logits.view(torch.int16 if logits.dtype == torch.bfloat16 else torch.int32))


@pytest.mark.parametrize("dtype,offset", [(torch.float32, 0), (torch.bfloat16, 0), (torch.float32, 1),
                                          (torch.bfloat16, 3)])
def test_argmax_special_values(built, dtype, offset):
    """NaN, infinities, signed zeros, ties and rows whose allowed logits are
    all -inf, on the fast (aligned) and the general path."""
    wl, clf, orc = built("json")
    states = wl.states(12)
    B, V = len(states), wl.V
    bits = orc.masks(states)
    rng = np.random.default_rng(8)
    x = torch.from_numpy(rng.standard_normal((B, V)).astype(np.float32))
    for b in range(B):
        allowed = np.nonzero(np.unpackbits(bits[b].astype("<u4").view(np.uint8), bitorder="little")[:V])[0]
        if allowed.size < 4:
            continue
        kind = b % 6
        if kind == 0:
            x[b, allowed[2]] = float("nan")
        elif kind == 1:
            x[b, allowed[1]] = float("inf")
            x[b, allowed[3]] = float("inf")           # tie: the lower id wins
        elif kind == 2:
            x[b, allowed] = float("-inf")              # every allowed logit -inf: the lowest allowed id
        elif kind == 3:
            x[b, allowed] = 0.0
            x[b, allowed[0]] = -0.0                    # -0 == +0: the lowest allowed id
        elif kind == 4:
            x[b] = float("nan")
            x[b, allowed] = 1.0                        # NaNs only where masked: ignored
    x = x.to(dtype)
    want = _closed_form(x, bits, V)
    buf = torch.empty(offset + B * V, dtype=dtype, device=DEV)
    dev = buf[offset:].view(B, V)
    dev.copy_(x.to(DEV))
    stacks, lens, qs = pack_states(states, DEV)
    got = clf.compute_and_argmax(stacks, lens, qs, dev).cpu().numpy()
    assert np.array_equal(got, want), np.nonzero(got != want)[0][:5]


def test_argmax_rejected_rows(built):
    wl, clf, orc = built("arithmetic")
    clf.error_count(reset=True)
    good = wl.states(3)[0]
    states = [good, (wl.grammar.lexer.n_states, good[1]), good]
    stacks, lens, qs = pack_states(states, DEV)
    logits = torch.randn(3, wl.V, device=DEV)
    logits[2] = logits[0]                      # same state, same logits: same token
    got = clf.compute_and_argmax(stacks, lens, qs, logits).cpu().numpy()
    assert got[1] == -1 and got[0] == got[2] and got[0] >= 0
    assert clf.error_count(reset=True) == 1


@pytest.mark.parametrize("name,B,steps", [("json", 16, 60), ("schema", 32, 60)])
def test_greedy_decoding_on_device(built, name, B, steps):
    """argmax (dense) -> advance, entirely on device states, against the same
    loop replayed on the host with the oracle's masks and advance."""
    wl, clf, orc = built(name)
    cap = 1024
    ds = DecodeStates(clf, B, cap, DEV)
    host = ds.host_states()
    done = np.zeros(B, bool)
    eos = wl.vocab.eos_id
    for k in range(steps):
        logits = wl.logits(1000 + k, B=B)
        toks = ds.argmax(logits.to(DEV)).cpu().numpy()
        want = _closed_form(logits, orc.masks(host), wl.V)
        assert np.array_equal(toks, want), (k, np.nonzero(toks != want)[0][:5])
        toks = np.where(done | (toks == eos), -1, toks).astype(np.int32)
        st = ds.advance(torch.from_numpy(toks).to(DEV)).cpu().numpy()
        for b in range(B):
            if toks[b] < 0:
                assert st[b] == psc.ADV_SKIPPED
                done[b] |= want[b] == eos
                continue
            code, new = orc.advance(host[b], int(toks[b]), cap)
            assert st[b] == code == psc.ADV_OK, (k, b)
            host[b] = new
        got = ds.host_states()
        for b in range(B):
            assert got[b][0] == host[b][0] and np.array_equal(got[b][1], host[b][1]), (k, b)


def test_argmax_calls_in_a_row_leave_no_state(built):
    """The per-sequence slots and arrival counters are cleared by each call:
    a full batch, a smaller one, the general path and the full batch again,
    back to back on one stream, each against the closed form."""
    wl, clf, orc = built("schema")
    cases = [(wl.states(40), 0), (wl.states(41)[:5], 0), (wl.states(42)[:9], 1), (wl.states(43), 0)]
    launched = []
    for k, (states, offset) in enumerate(cases):
        logits = wl.logits(40 + k)[:len(states)].contiguous()
        buf = torch.empty(offset + logits.numel(), dtype=logits.dtype, device=DEV)
        dev = buf[offset:].view(logits.shape)
        dev.copy_(logits.to(DEV))
        stacks, lens, qs = pack_states(states, DEV)
        launched.append((clf.compute_and_argmax(stacks, lens, qs, dev), logits, states, dev, stacks, lens, qs))
    torch.cuda.synchronize()
    for got, logits, states, *_ in launched:
        assert np.array_equal(got.cpu().numpy(), _closed_form(logits, orc.masks(states), wl.V))


def test_argmax_graph_replays(built):
    """The masked argmax captured in a HIP graph: every replay, with new
    logits written into the captured buffer and eager argmax calls between
    the replays, gives the eager result."""
    wl, clf, orc = built("json")
    states = wl.states(20)
    stacks, lens, qs = pack_states(states, DEV)
    g_logits = wl.logits(0).to(DEV)
    g_out = torch.full((len(states),), -7, dtype=torch.int32, device=DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        clf.compute_and_argmax(stacks, lens, qs, g_logits, out=g_out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        clf.compute_and_argmax(stacks, lens, qs, g_logits, out=g_out)
    want_bits = orc.masks(states)
    for rep in range(4):
        logits = wl.logits(100 + rep)
        g_logits.copy_(logits.to(DEV))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        eager = clf.compute_and_argmax(stacks, lens, qs, logits.to(DEV))
        torch.cuda.synchronize()
        assert torch.equal(g_out, eager), rep
        assert np.array_equal(g_out.cpu().numpy(), _closed_form(logits, want_bits, wl.V)), rep
