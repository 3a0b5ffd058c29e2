"""GPU parity through the C-ABI: device masks vs the oracle (bit-exact), and
the in-place apply vs its closed form (bit-exact, compared as integers)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import apply_mask, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _device_masks(clf, states):
    stacks, lens, qs = pack_states(states, DEV)
    out = clf.compute_masks(stacks, lens, qs)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint32)


def test_arithmetic_all_steps_bit_exact(built):
    wl, clf, orc = built("arithmetic")
    states = [st for s in range(wl.steps) for st in wl.states(s)]
    want = orc.masks(states)
    # one launch over every step, and one launch per step (B = 1)
    got = _device_masks(clf, states)
    assert np.array_equal(got, want)
    for s in range(0, wl.steps, 25):
        assert np.array_equal(_device_masks(clf, states[s:s + 1]), want[s:s + 1])
    assert clf.error_count() == 0


@pytest.mark.parametrize("name,steps", [("json", range(0, 60, 3)), ("schema", range(0, 1000, 50)),
                                        ("pylike", range(0, 500, 100)), ("stress", range(0, 1000, 250))])
def test_full_shape_steps_bit_exact(built, name, steps):
    """Every row of every listed step at the workload's full batch and
    vocabulary (the shape the benchmark times), one launch per step."""
    wl, clf, orc = built(name)
    for step in steps:
        states = wl.states(step)
        got = _device_masks(clf, states)
        want = orc.masks(states)
        bad = np.nonzero((got != want).any(axis=1))[0]
        assert bad.size == 0, (step, bad[:8])
    assert clf.error_count() == 0


def test_schema_many_steps_in_one_launch(built):
    wl, clf, orc = built("schema")
    states = [st for s in range(1000, 1010) for st in wl.states(s)]
    assert np.array_equal(_device_masks(clf, states), orc.masks(states))


def test_device_matches_host_walk_many_steps(built):
    wl, clf, _ = built("json")
    states = [st for s in range(60, 160) for st in wl.states(s)]
    assert np.array_equal(_device_masks(clf, states), clf.masks_host(states))


def test_range_faults_give_zero_rows_and_count(built):
    wl, clf, orc = built("arithmetic")
    clf.error_count(reset=True)
    good = wl.states(3)[0]
    n_lex = wl.grammar.lexer.n_states
    n_lr = wl.grammar.n_lr_states
    states = [good, (n_lex + 1, good[1]), (-1, good[1]),
              (good[0], np.concatenate([good[1][:-1], [n_lr]]).astype(np.int32)), good]
    got = _device_masks(clf, states)
    want = orc.masks([good])[0]
    assert np.array_equal(got[0], want) and np.array_equal(got[4], want)
    assert not got[1].any() and not got[2].any() and not got[3].any()
    assert clf.error_count(reset=True) == 3


def test_zero_length_stack_is_a_fault(built):
    wl, clf, _ = built("arithmetic")
    clf.error_count(reset=True)
    good = wl.states(4)[0]
    stacks, lens, qs = pack_states([good, good], DEV)
    lens[0] = 0
    stacks = stacks[len(good[1]):].contiguous()
    out = clf.compute_masks(stacks, lens, qs)
    torch.cuda.synchronize()
    o = out.cpu().numpy().view(np.uint32)
    assert not o[0].any() and np.array_equal(o[1], clf.masks_host([good])[0])
    assert clf.error_count(reset=True) == 1


def test_empty_batch_is_noop(built):
    wl, clf, _ = built("arithmetic")
    z = torch.zeros(1, dtype=torch.int32, device=DEV)
    e = torch.zeros(0, dtype=torch.int32, device=DEV)
    out = torch.empty((0, clf.W), dtype=torch.int32, device=DEV)
    clf.compute_masks(z, e, e, out=out)
    torch.cuda.synchronize()


# ------------------------------------------------------------------ apply

def _closed_form(logits_cpu, bits_np, V):
    m = np.unpackbits(bits_np.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    neg = torch.full_like(logits_cpu, float("-inf"))
    return torch.where(torch.from_numpy(m), logits_cpu, neg)


def _as_int(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


@pytest.mark.parametrize("B,V,dtype", [
    (1, 513, torch.float32), (3, 513, torch.bfloat16), (16, 32000, torch.float32),
    (5, 151936, torch.bfloat16), (2, 4096, torch.float32), (7, 96, torch.bfloat16),
    (4, 33, torch.float32), (1, 1, torch.bfloat16)])
def test_apply_matches_closed_form(B, V, dtype):
    g = torch.Generator().manual_seed(B * 1000 + V)
    logits = (torch.randn(B, V, generator=g) * 2).to(dtype)
    logits[0, 0] = float("nan")
    W = (V + 31) // 32
    rng = np.random.default_rng(V)
    # mixes all-zero, all-one and random words, tail bits zero
    bits = rng.integers(0, 2**32, size=(B, W), dtype=np.uint64).astype(np.uint32)
    bits[:, ::3] = 0
    bits[:, 1::5] = 0xFFFFFFFF
    if V % 32:
        bits[:, -1] &= np.uint32((1 << (V % 32)) - 1)
    want = _closed_form(logits, bits, V)
    # canaries after the tensor
    buf = torch.empty(B * V + 64, dtype=dtype, device=DEV)
    buf[B * V:] = 7
    dev = buf[:B * V].view(B, V)
    dev.copy_(logits.to(DEV))
    bm = torch.from_numpy(bits.view(np.int32)).to(DEV)
    apply_mask(dev, bm)
    torch.cuda.synchronize()
    assert torch.equal(_as_int(dev.cpu()), _as_int(want))
    assert (buf[B * V:].cpu() == 7).all()


@pytest.mark.parametrize("name,step", [("arithmetic", 5), ("json", 7), ("schema", 3), ("schema", 777),
                                       ("pylike", 11), ("stress", 13)])
def test_apply_after_compute_end_to_end(built, name, step):
    """The whole step (compute_masks then apply_mask on one stream) against
    the oracle's masks applied by the closed form."""
    wl, clf, orc = built(name)
    states = wl.states(step)
    stacks, lens, qs = pack_states(states, DEV)
    logits = wl.logits(step)
    dev = logits.to(DEV)
    bm = clf.compute_masks(stacks, lens, qs)
    apply_mask(dev, bm)
    torch.cuda.synchronize()
    want = _closed_form(logits, orc.masks(states), wl.V)
    assert torch.equal(_as_int(dev.cpu()), _as_int(want))


@pytest.mark.parametrize("name,steps", [("arithmetic", range(0, 200, 7)), ("json", range(0, 40, 5)),
                                        ("schema", [0, 333, 999]), ("pylike", [2, 222]), ("stress", [5, 555])])
def test_classes_match_host_walk_and_masks(built, name, steps):
    """psc_compute_classes (ragged and dense) gives the host walk's class,
    and that class's mask row is the oracle's mask."""
    from paper_2608_03065_amd.psc import DecodeStates
    wl, clf, orc = built(name)
    clf.error_count(reset=True)
    for step in steps:
        states = wl.states(step)
        stacks, lens, qs = pack_states(states, DEV)
        got = clf.compute_classes(stacks, lens, qs).cpu().numpy()
        assert np.array_equal(got, clf.classify_host(states)), step
        cap = max(len(a) for _, a in states) + 3
        dense = DecodeStates(clf, len(states), cap, DEV).load(states).compute_classes().cpu().numpy()
        assert np.array_equal(dense, got), step
        want = orc.masks(states[:4])
        for b in range(len(want)):
            assert np.array_equal(clf.class_mask(int(got[b])), want[b]), (step, b)
    assert clf.error_count() == 0


def test_classes_reject_out_of_range(built):
    wl, clf, _ = built("arithmetic")
    clf.error_count(reset=True)
    good = wl.states(3)[0]
    n_lr = wl.grammar.n_lr_states
    states = [good, (wl.grammar.lexer.n_states, good[1]),
              (good[0], np.concatenate([good[1][:-1], [n_lr]]).astype(np.int32)), good]
    stacks, lens, qs = pack_states(states, DEV)
    got = clf.compute_classes(stacks, lens, qs).cpu().numpy()
    want = clf.classify_host([good])[0]
    assert got.tolist() == [want, -1, -1, want]
    assert clf.error_count(reset=True) == 2
