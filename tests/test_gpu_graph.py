"""The step captured in a HIP graph (torch.cuda.CUDAGraph): every replay,
with new inputs written into the captured buffers between replays, must
equal the same calls made eagerly."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd.psc import DecodeStates, pack_states  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_fused_step_graph_replays(built):
    wl, clf, orc = built("schema")
    B = wl.B
    steps = [wl.states(s) for s in range(30, 36)]
    max_total = max(sum(len(a) for _, a in st) for st in steps)
    g_stacks = torch.zeros(max_total, dtype=torch.int32, device=DEV)
    g_lens = torch.zeros(B, dtype=torch.int32, device=DEV)
    g_qs = torch.zeros(B, dtype=torch.int32, device=DEV)
    g_logits = torch.zeros((B, wl.V), dtype=torch.bfloat16, device=DEV)
    g_out = torch.zeros((B, clf.W), dtype=torch.int32, device=DEV)

    def load(k):
        stacks, lens, qs = pack_states(steps[k], DEV)
        g_stacks[:stacks.numel()].copy_(stacks)
        g_lens.copy_(lens)
        g_qs.copy_(qs)
        g_logits.copy_(wl.logits(30 + k).to(DEV))

    load(0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                   # warm-up outside the capture
        clf.compute_and_apply(g_stacks, g_lens, g_qs, g_logits.clone(), out=g_out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        clf.compute_and_apply(g_stacks, g_lens, g_qs, g_logits, out=g_out)
    for rep in range(3):
        for k in range(len(steps)):
            load(k)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            stacks, lens, qs = pack_states(steps[k], DEV)
            eager = wl.logits(30 + k).to(DEV)
            out = torch.empty_like(g_out)
            clf.compute_and_apply(stacks, lens, qs, eager, out=out)
            torch.cuda.synchronize()
            assert torch.equal(g_out, out), (rep, k)
            assert torch.equal(g_logits.view(torch.int16), eager.view(torch.int16)), (rep, k)
            if rep == 0:
                assert np.array_equal(g_out.cpu().numpy().view(np.uint32), orc.masks(steps[k])), k


def test_decode_step_graph_replays(built):
    """advance + fused step on device states, captured once and replayed per
    token; the states and outputs follow an eager twin exactly."""
    wl, clf, orc = built("json")
    B, cap, n = 16, 512, 40
    toks = [wl.vocab.tokenize(wl.make_document(np.random.default_rng(b), wl))[:n] for b in range(B)]
    n = min(len(t) for t in toks)
    g_tok = torch.zeros(B, dtype=torch.int32, device=DEV)
    g_logits = torch.zeros((B, wl.V), dtype=torch.float32, device=DEV)
    g_out = torch.zeros((B, clf.W), dtype=torch.int32, device=DEV)
    ds = DecodeStates(clf, B, cap, DEV)
    twin = DecodeStates(clf, B, cap, DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                   # warm-up outside the capture
        DecodeStates(clf, B, cap, DEV).advance(g_tok)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ds.advance(g_tok)
        ds.compute_and_apply(g_logits, out=g_out)
    ds.reset()
    torch.cuda.synchronize()
    for k in range(n):
        t = torch.tensor([toks[b][k] for b in range(B)], dtype=torch.int32, device=DEV)
        g_tok.copy_(t)
        logits = wl.logits(k, B=B).to(DEV)
        g_logits.copy_(logits)
        torch.cuda.synchronize()
        graph.replay()
        st = twin.advance(t)
        out = torch.empty_like(g_out)
        twin.compute_and_apply(logits, out=out)
        torch.cuda.synchronize()
        assert torch.equal(ds.status, st) and torch.equal(g_out, out), k
        assert torch.equal(g_logits.view(torch.int32), logits.view(torch.int32)), k
        assert torch.equal(ds.lens, twin.lens) and torch.equal(ds.qs, twin.qs), k
        assert torch.equal(ds.stacks, twin.stacks), k
