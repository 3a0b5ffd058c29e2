"""Every decoding step of the three smaller workloads through both step forms
at the benchmarked shape, against the oracle; twenty sampled steps of each
programming-language workload.

PSC computes exactly the set of eq. simp (Theorems 1-3), so the bar is bit
equality with the oracle on every row of every step (Algorithm 2: the
classification and mask steps; the masked logits of Sec. 1, Fig. 1a).  Each
step's batch goes through psc_compute_and_apply (one launch, the benchmarked
step: bitmask and masked logits) and through psc_compute_masks then
psc_apply_mask (two launches).  Both bitmasks are compared with the oracle's
masks on every step; the masked logits of both forms are compared with the
closed form of the oracle's masks on every tenth step (bit-exact, as
integers).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import apply_mask, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _closed_form(logits_cpu, bits_np, V):
    m = np.unpackbits(bits_np.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    return torch.where(torch.from_numpy(m), logits_cpu, torch.full_like(logits_cpu, float("-inf")))


def _as_int(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


def _run_steps(built, name, steps, logits_every):
    wl, clf, orc = built(name)
    clf.error_count(reset=True)
    tdt = torch.bfloat16 if wl.logits_dtype == "bf16" else torch.float32
    lg = torch.empty((wl.B, wl.V), dtype=tdt, device=DEV)
    lg2 = torch.empty_like(lg)
    out = torch.empty((wl.B, clf.W), dtype=torch.int32, device=DEV)
    out2 = torch.empty_like(out)
    n = 0
    for k, step in enumerate(steps):
        states = wl.states(step)
        stacks, lens, qs = pack_states(states, DEV)
        check_logits = k % logits_every == 0
        if check_logits:
            logits = wl.logits(step)
            lg.copy_(logits)
            lg2.copy_(logits)
        clf.compute_and_apply(stacks, lens, qs, lg, out=out)
        clf.compute_masks(stacks, lens, qs, out=out2)
        if check_logits:
            apply_mask(lg2, out2)
        torch.cuda.synchronize()
        want = orc.masks(states)
        for form, got in (("fused", out), ("two-launch", out2)):
            bad = np.nonzero((got.cpu().numpy().view(np.uint32) != want).any(axis=1))[0]
            assert bad.size == 0, (name, form, step, bad[:8].tolist())
        if check_logits:
            ref = _as_int(_closed_form(logits, want, wl.V))
            assert torch.equal(_as_int(lg.cpu()), ref), (name, "fused logits", step)
            assert torch.equal(_as_int(lg2.cpu()), ref), (name, "two-launch logits", step)
        n += len(states)
    assert clf.error_count() == 0
    return n


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema"])
def test_every_step_bit_exact(built, name):
    wl = built(name)[0]
    rows = _run_steps(built, name, range(wl.steps), logits_every=10)
    assert rows == wl.steps * wl.B


@pytest.mark.parametrize("name", ["json", "schema"])
def test_every_step_bit_exact_speculative(built, name):
    """The same with PSC_OPT_SPECULATE, the class predictor trained on
    held-out prefixes first (the fused step then loads the predicted class's
    data during the walk)."""
    wl, clf, _ = built(name)
    clf.set_options(speculate=True)
    try:
        train = [st for s in range(wl.steps, wl.steps + 100) for st in wl.states(s)]
        clf.compute_classes(*pack_states(train, DEV))
        rows = _run_steps(built, name, range(wl.steps), logits_every=25)
        assert rows == wl.steps * wl.B
    finally:
        clf.set_options(speculate=False)
        clf.predictor_fill(-1)


@pytest.mark.parametrize("name", ["pylike", "stress", "gosql"])
def test_twenty_sampled_steps_bit_exact(built, name):
    wl = built(name)[0]
    steps = np.linspace(0, wl.steps - 1, 20).astype(int).tolist()
    assert len(set(steps)) == 20
    _run_steps(built, name, steps, logits_every=5)
