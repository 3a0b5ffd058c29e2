"""GPU parity of the sliced mask layout, of the class predictor and of the
bounded ragged calls, through the C-ABI.

The sliced layout (the runtime mask table compressed: each distinct 64-word
slice of the precomputed rows stored once) and the predictor (which decides
only what the speculative kernels load before the walk has ended) must never
change a result: every call is compared bit for bit with the oracle's masks
(eq. simp, Theorems 1-3) and the closed form of the masked logits, under
every predictor state, including one that predicts a wrong class everywhere.
"""
import os
import tempfile

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import Classifier, DecodeStates, apply_mask, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _closed_form(logits_cpu, bits_np, V):
    m = np.unpackbits(bits_np.astype("<u4").view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    return torch.where(torch.from_numpy(m), logits_cpu, torch.full_like(logits_cpu, float("-inf")))


def _as_int(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


_SLICED = {}


def _sliced(built, name):
    """The workload's classifier (saved and loaded again) bound with the
    sliced mask layout."""
    if name not in _SLICED:
        wl, clf, orc = built(name)
        with tempfile.TemporaryDirectory() as d:
            path = os.path.join(d, "c.psc")
            clf.save(path)
            sl = Classifier.load(path)
        sl.bind(DEV, layout="sliced")
        assert sl.info()["bound_mask_layout"] == 2
        _SLICED[name] = sl
    return _SLICED[name]


def _step_outputs(clf, wl, states, step):
    """(bitmask of the fused step, its logits, bitmask of compute_masks,
    logits after apply_mask, classes) for one batch."""
    stacks, lens, qs = pack_states(states, DEV)
    logits = wl.logits(step, B=len(states))
    lg = logits.to(DEV)
    out = torch.empty((len(states), clf.W), dtype=torch.int32, device=DEV)
    clf.compute_and_apply(stacks, lens, qs, lg, out=out)
    bm = clf.compute_masks(stacks, lens, qs)
    lg2 = logits.to(DEV)
    apply_mask(lg2, bm)
    cls = clf.compute_classes(stacks, lens, qs)
    torch.cuda.synchronize()
    return logits, out.cpu().numpy().view(np.uint32), lg.cpu(), bm.cpu().numpy().view(np.uint32), lg2.cpu(), \
        cls.cpu().numpy()


def _check_step(clf, wl, orc, states, step, ref_classes=None):
    logits, bits, lg, bits2, lg2, cls = _step_outputs(clf, wl, states, step)
    want = orc.masks(states)
    for form, got in (("fused", bits), ("two-launch", bits2)):
        bad = np.nonzero((got != want).any(axis=1))[0]
        assert bad.size == 0, (wl.name, form, step, bad[:8].tolist())
    ref = _as_int(_closed_form(logits, want, wl.V))
    assert torch.equal(_as_int(lg), ref), (wl.name, "fused logits", step)
    assert torch.equal(_as_int(lg2), ref), (wl.name, "two-launch logits", step)
    if ref_classes is not None:
        assert np.array_equal(cls, ref_classes), (wl.name, step)


@pytest.mark.parametrize("name,steps", [("arithmetic", [0, 9]), ("json", [3, 250]), ("schema", [5, 640]),
                                        ("pylike", [7, 321]), ("stress", [17]), ("gosql", [4, 333])])
def test_sliced_layout_bit_exact(built, name, steps):
    wl, clf, orc = built(name)
    sl = _sliced(built, name)
    inf = sl.info()
    n_ids = inf["n_classes"] * inf["mask_stride_words"] // 64
    assert inf["sliced_mask_bytes"] <= inf["mask_table_bytes"] + 4 * n_ids
    sl.error_count(reset=True)
    for step in steps:
        states = wl.states(step)
        _check_step(sl, wl, orc, states, step, ref_classes=clf.classify_host(states))
    assert sl.error_count() == 0


@pytest.mark.parametrize("name", ["arithmetic", "json", "schema", "pylike"])
def test_sliced_layout_argmax_and_decode_step(built, name):
    """The calls without speculation read the sliced table through the same
    accessor: masked argmax and the one-launch decoding step equal the flat
    layout's."""
    wl, clf, orc = built(name)
    sl = _sliced(built, name)
    states = wl.states(21)
    stacks, lens, qs = pack_states(states, DEV)
    logits = wl.logits(21).to(DEV)
    t_flat = clf.compute_and_argmax(stacks, lens, qs, logits)
    t_sl = sl.compute_and_argmax(stacks, lens, qs, logits)
    torch.cuda.synchronize()
    assert torch.equal(t_flat, t_sl)
    cap = max(len(a) for _, a in states) + 64
    toks = torch.tensor(np.arange(len(states), dtype=np.int32) * 37 % wl.V, device=DEV)
    res = []
    for c in (clf, sl):
        ds = DecodeStates(c, len(states), cap, DEV).load(states)
        lg = wl.logits(22).to(DEV)
        out = torch.empty((len(states), c.W), dtype=torch.int32, device=DEV)
        st = ds.decode_step(toks, lg, out=out)
        torch.cuda.synchronize()
        res.append((st.cpu(), out.cpu(), _as_int(lg.cpu()), ds.host_states()))
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1])
    assert torch.equal(res[0][2], res[1][2])
    for (q0, s0), (q1, s1) in zip(res[0][3], res[1][3]):
        assert q0 == q1 and np.array_equal(s0, s1)


@pytest.mark.parametrize("name,layout", [("json", "flat"), ("schema", "flat"), ("schema", "sliced"),
                                         ("pylike", "flat"), ("pylike", "sliced")])
def test_predictor_never_changes_results(built, name, layout):
    """Empty, trained, and wrong everywhere (every entry one class): the
    fused and two-launch steps stay bit-exact against the oracle."""
    wl, clf, orc = built(name)
    c = clf if layout == "flat" else _sliced(built, name)
    c.set_options(speculate=True)
    n_classes = c.info()["n_classes"]
    train = [st for s in range(wl.steps, wl.steps + 20) for st in wl.states(s)]
    tstacks, tlens, tqs = pack_states(train, DEV)
    for mode in ("empty", "trained", "class0", "last"):
        if mode == "empty":
            c.predictor_fill(-1)
        elif mode == "trained":
            c.predictor_fill(-1)
            c.compute_classes(tstacks, tlens, tqs)
        else:
            c.predictor_fill(0 if mode == "class0" else n_classes - 1)
        torch.cuda.synchronize()
        for step in (2, 301):
            states = wl.states(step)
            _check_step(c, wl, orc, states, step, ref_classes=clf.classify_host(states))
    with pytest.raises(Exception):
        c.predictor_fill(n_classes)
    c.predictor_fill(-1)
    c.set_options(speculate=False)


def test_predictor_learns(built):
    """Trained on held-out prefixes of the schema workload, the predictor
    holds for most sequences of the benchmarked steps (it only changes
    speed; the count is of walks that ended in another class)."""
    wl, clf, _ = built("schema")
    clf.set_options(speculate=True)
    clf.predictor_fill(-1)
    train = [st for s in range(wl.steps, wl.steps + 200) for st in wl.states(s)]
    stacks, lens, qs = pack_states(train, DEV)
    clf.compute_classes(stacks, lens, qs)
    torch.cuda.synchronize()
    first = clf.predictor_updates(reset=True)
    assert first > 0
    lg = torch.zeros((wl.B, wl.V), dtype=torch.bfloat16, device=DEV)
    n = 50
    for s in range(n):
        st, ln, q = pack_states(wl.states(s), DEV)
        clf.compute_and_apply(st, ln, q, lg)
    torch.cuda.synchronize()
    misses = clf.predictor_updates(reset=True)
    assert misses < 0.5 * n * wl.B, misses
    clf.predictor_fill(-1)
    clf.set_options(speculate=False)


def test_stack_bound_rejects_overlong_stack(built):
    """A ragged stack whose length reaches past the stacks tensor is a
    rejected input (zero row, one count) in every bounded call, even when
    the memory past the tensor is allocated: it is never read."""
    wl, clf, orc = built("schema")
    states = wl.states(40)[:8]
    stacks, lens, qs = pack_states(states, DEV)
    n = stacks.numel()
    big = torch.zeros(n + 4096, dtype=torch.int32, device=DEV)
    big[:n] = stacks
    big[n:] = int(states[-1][1][0])       # valid symbols past the end
    view = big[:n]
    lens[-1] += 7                         # the last stack now ends 7 symbols past the view
    want = orc.masks(states)
    clf.error_count(reset=True)
    out = clf.compute_masks(view, lens, qs)
    lg = torch.zeros((len(states), wl.V), dtype=torch.bfloat16, device=DEV)
    out2 = torch.empty_like(out)
    clf.compute_and_apply(view, lens, qs, lg, out=out2)
    cls = clf.compute_classes(view, lens, qs)
    tok = clf.compute_and_argmax(view, lens, qs, lg)
    torch.cuda.synchronize()
    for o in (out, out2):
        got = o.cpu().numpy().view(np.uint32)
        assert np.array_equal(got[:-1], want[:-1]) and not got[-1].any()
    assert cls.cpu().numpy()[-1] == -1 and tok.cpu().numpy()[-1] == -1
    assert (lg[-1].view(torch.int16) == -128).all()       # 0xFF80: -inf
    assert clf.error_count(reset=True) == 4


def test_timeline_records_and_results(built):
    wl, clf, orc = built("schema")
    states = wl.states(77)
    stacks, lens, qs = pack_states(states, DEV)
    logits = wl.logits(77)
    lg = logits.to(DEV)
    out = torch.empty((wl.B, clf.W), dtype=torch.int32, device=DEV)
    n = clf.timeline_records(wl.B, torch.bfloat16)
    rec = torch.zeros((n, 4), dtype=torch.int64, device=DEV)
    clf.compute_and_apply_timeline(stacks, lens, qs, lg, rec, out=out)
    torch.cuda.synchronize()
    want = orc.masks(states)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), want)
    assert torch.equal(_as_int(lg.cpu()), _as_int(_closed_form(logits, want, wl.V)))
    r = rec.cpu().numpy().view(np.uint64)
    t_a, t_b = r[:, 1] & 0xFFFFFFFF, r[:, 1] >> 32
    t_e, meta = r[:, 2] & 0xFFFFFFFF, r[:, 2] >> 32
    assert (r[:, 0] > 0).all() and (t_a <= t_b).all() and (t_b <= t_e).all()
    per_block = 4
    assert np.array_equal(meta & 7, np.tile(np.arange(per_block), n // per_block))
    assert set((r[:, 3] & 0xFFFFFFFF).tolist()) == set(range(wl.B))
    small = torch.zeros((n - 1, 4), dtype=torch.int64, device=DEV)
    with pytest.raises(Exception):
        clf.compute_and_apply_timeline(stacks, lens, qs, lg, small)
