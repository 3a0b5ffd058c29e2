"""GPU parity of the single-launch step (psc_compute_and_apply) through the
C-ABI: its bitmask against the oracle's masks (bit-exact) and its logits
against the closed form of those masks applied (bit-exact, as integers)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import Classifier, PscError, apply_mask, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _closed_form(logits_cpu, bits_np, V):
    m = np.unpackbits(bits_np.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    return torch.where(torch.from_numpy(m), logits_cpu, torch.full_like(logits_cpu, float("-inf")))


def _as_int(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


def _fused(clf, states, logits_cpu, with_out=True, offset=0):
    """Run the fused step on a device copy of logits_cpu placed `offset`
    elements into a buffer with canaries after it; returns (bits, logits)."""
    B, V = logits_cpu.shape
    stacks, lens, qs = pack_states(states, DEV)
    buf = torch.empty(offset + B * V + 64, dtype=logits_cpu.dtype, device=DEV)
    buf.fill_(7)
    dev = buf[offset:offset + B * V].view(B, V)
    dev.copy_(logits_cpu.to(DEV))
    out = torch.empty((B, clf.W), dtype=torch.int32, device=DEV) if with_out else None
    clf.compute_and_apply(stacks, lens, qs, dev, out=out)
    torch.cuda.synchronize()
    assert (buf[:offset].cpu() == 7).all() and (buf[offset + B * V:].cpu() == 7).all()
    bits = out.cpu().numpy().view(np.uint32) if with_out else None
    return bits, dev.cpu()


@pytest.mark.parametrize("name,steps", [("arithmetic", [0, 5, 77]), ("json", [0, 7, 300]),
                                        ("schema", [3, 500, 777]), ("pylike", [11, 250]),
                                        ("stress", [13, 600])])
def test_fused_step_bit_exact(built, name, steps):
    """Full batch and vocabulary of each workload, in its logits dtype."""
    wl, clf, orc = built(name)
    clf.error_count(reset=True)
    for step in steps:
        states = wl.states(step)
        logits = wl.logits(step)
        want_bits = orc.masks(states)
        bits, got = _fused(clf, states, logits)
        bad = np.nonzero((bits != want_bits).any(axis=1))[0]
        assert bad.size == 0, (step, bad[:8])
        assert torch.equal(_as_int(got), _as_int(_closed_form(logits, want_bits, wl.V))), step
    assert clf.error_count() == 0


@pytest.mark.parametrize("name,dtype,offset", [
    ("arithmetic", torch.bfloat16, 0),   # V = 513: general path
    ("json", torch.bfloat16, 0),         # V = 32000: fast path, the other dtype
    ("json", torch.float32, 1),          # misaligned logits: general path
    ("schema", torch.float32, 0),        # fast path, fp32
    ("schema", torch.bfloat16, 3),       # misaligned bf16: general path
    ("stress", torch.float32, 0),        # fast path, fp32, 16,384 workgroups
    ("stress", torch.bfloat16, 1)])      # general path, 16,384 workgroups
def test_fused_other_dtype_and_alignment(built, name, dtype, offset):
    wl, clf, orc = built(name)
    states = wl.states(9)
    logits = (wl.logits(9).float() * 1.0).to(dtype)
    logits[0, 0] = float("nan")
    want_bits = orc.masks(states)
    bits, got = _fused(clf, states, logits, offset=offset)
    assert np.array_equal(bits, want_bits)
    assert torch.equal(_as_int(got), _as_int(_closed_form(logits, want_bits, wl.V)))


@pytest.mark.parametrize("name", ["schema", "stress"])
def test_fused_equals_two_launches(built, name):
    """Bit-identical to psc_compute_masks + psc_apply_mask, many steps in
    one batch, and the bitmask output is optional."""
    wl, clf, _ = built(name)
    steps = range(100, 104)
    states = [st for s in steps for st in wl.states(s)]
    logits = torch.cat([wl.logits(s) for s in steps])
    stacks, lens, qs = pack_states(states, DEV)
    two = logits.to(DEV)
    apply_mask(two, clf.compute_masks(stacks, lens, qs))
    bits, got = _fused(clf, states, logits)
    _, got_no_out = _fused(clf, states, logits, with_out=False)
    torch.cuda.synchronize()
    assert torch.equal(_as_int(got), _as_int(two.cpu()))
    assert torch.equal(_as_int(got_no_out), _as_int(two.cpu()))
    assert np.array_equal(bits, clf.masks_host(states))


@pytest.mark.parametrize("name", ["arithmetic", "schema"])
def test_fused_rejected_rows(built, name):
    """Out-of-range inputs: an all-zero mask row, an all -inf logits row, one
    count each; the neighbours are unaffected."""
    wl, clf, orc = built(name)
    clf.error_count(reset=True)
    good = wl.states(3)[0]
    n_lex, n_lr = wl.grammar.lexer.n_states, wl.grammar.n_lr_states
    states = [good, (n_lex, good[1]), (good[0], np.concatenate([good[1][:-1], [n_lr]]).astype(np.int32)), good]
    logits = wl.logits(3, B=len(states))
    bits, got = _fused(clf, states, logits)
    want = orc.masks([good])[0]
    assert np.array_equal(bits[0], want) and np.array_equal(bits[3], want)
    assert not bits[1].any() and not bits[2].any()
    assert torch.isneginf(got[1].float()).all() and torch.isneginf(got[2].float()).all()
    ref = _closed_form(logits[[0, 3]], np.stack([want, want]), wl.V)
    assert torch.equal(_as_int(got[[0, 3]]), _as_int(ref))
    assert clf.error_count(reset=True) == 2


def test_fused_argument_errors(built):
    wl, clf, _ = built("arithmetic")
    states = wl.states(1)
    stacks, lens, qs = pack_states(states, DEV)
    bad_v = torch.zeros((1, wl.V + 1), dtype=torch.float32, device=DEV)
    with pytest.raises(PscError) as e:
        from paper_2608_03065_amd import psc
        psc._check(psc.lib().psc_compute_and_apply(clf._h, stacks.data_ptr(), lens.data_ptr(), qs.data_ptr(),
                                                   1, None, bad_v.data_ptr(), psc.PSC_F32, wl.V + 1, None))
    assert e.value.status == -1
    unbound = Classifier(wl.grammar, wl.vocab)
    logits = torch.zeros((1, wl.V), dtype=torch.float32, device=DEV)
    with pytest.raises(PscError) as e:
        unbound.compute_and_apply(stacks, lens, qs, logits)
    assert e.value.status == -6
    # B == 0 is a no-op
    z = torch.zeros(1, dtype=torch.int32, device=DEV)
    e0 = torch.zeros(0, dtype=torch.int32, device=DEV)
    clf.compute_and_apply(z, e0, e0, torch.zeros((0, wl.V), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,offset", [("arithmetic", 0), ("arithmetic", 1), ("json", 0), ("json", 1),
                                         ("schema", 0), ("schema", 3)])
def test_bitmask_rows_stay_in_bounds(built, name, offset):
    """out_bitmask [B, W] placed `offset` words into a buffer filled with
    canaries: compute_masks (16-byte and word-wise row copies) and the fused
    step write exactly the B x W words, equal to the oracle's masks."""
    wl, clf, orc = built(name)
    states = wl.states(4)
    want = orc.masks(states)
    B, W = len(states), clf.W
    stacks, lens, qs = pack_states(states, DEV)
    for fused in (False, True):
        buf = torch.full((offset + B * W + 67,), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
        out = buf[offset:offset + B * W].view(B, W)
        if fused:
            lg = wl.logits(4).to(DEV)
            clf.compute_and_apply(stacks, lens, qs, lg, out=out)
        else:
            clf.compute_masks(stacks, lens, qs, out=out)
        h = buf.cpu().numpy()
        assert (h[:offset] == 0x5A5A5A5A).all() and (h[offset + B * W:] == 0x5A5A5A5A).all(), fused
        assert np.array_equal(h[offset:offset + B * W].view(np.uint32).reshape(B, W), want), fused
