"""The library-owned workspace of a (device, stream) pair.  A graph captured
with asd_verify keeps the workspace address it was captured with; a later
eager call on the same stream that needs a larger workspace must leave that
buffer valid, so the graph still replays correctly."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def _batch(rng, num_requests, K, vocab):
    rows = num_requests * (K + 1)
    logits = rng.integers(-3, 4, size=(rows, vocab)).astype(np.float32)   # many ties
    draft = rng.integers(0, vocab, size=rows).astype(np.int32)
    draft[rng.random(rows) < 0.02] = vocab + 2
    lens = np.full(num_requests, K, np.int32)
    tau = rng.uniform(0.5, 3.0, num_requests).astype(np.float32)
    cap = rng.integers(0, 3, num_requests).astype(np.int32)
    budget = np.stack([rng.uniform(0, 6, num_requests), np.zeros(num_requests)],
                      axis=1).astype(np.float32)
    return logits, draft, lens, tau, cap, budget


def _device(dev, logits, draft, lens, tau, cap, budget):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(x)).to(dev)
            for x in (logits, draft, lens, tau, cap, budget)]


def _same(a, b):
    a, b = np.asarray(a), np.asarray(b)
    if a.dtype == np.float32:
        a, b = a.view(np.uint32), b.view(np.uint32)
    return np.array_equal(a, b)


def test_graph_replays_after_the_workspace_grows():
    import torch
    import paper_2608_03447_amd as asd
    dev = torch.device("cuda:0")
    torch.cuda.synchronize(dev)
    asd.asd_release()                 # every stream starts without a library workspace
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    rng = np.random.default_rng(77)

    small = _batch(rng, 4, 9, 16)     # 40 rows: the first, 1 MiB workspace
    ref_small = oracle.verify(*small)
    tl, td, tk, tt, tc, tb = _device(dev, *small)
    pristine = tb.clone()
    rows = tl.shape[0]
    acc = torch.empty(4, dtype=torch.int32, device=dev)
    nxt = torch.empty(4, dtype=torch.int32, device=dev)
    amax = torch.empty(rows, dtype=torch.int32, device=dev)
    reg = torch.empty(rows, dtype=torch.float32, device=dev)

    def call():
        asd.asd_verify(tl, td, tk, tt, tc, tb, out_accept_len=acc, out_next_token=nxt,
                       out_argmax=amax, out_regret=reg)

    def check(tag):
        got = {"accept_len": acc, "next_token": nxt, "argmax": amax, "regret": reg, "budget": tb}
        for k, v in got.items():
            g = v.cpu().numpy()
            r = ref_small[k]
            if k == "regret":
                both_nan = np.isnan(g) & np.isnan(r)
                g, r = g[~both_nan], r[~both_nan]
            assert _same(g, r), "%s: %s differs from the oracle" % (tag, k)

    with torch.cuda.stream(side):     # eager: creates the stream's workspace
        call()
    torch.cuda.synchronize(dev)
    check("eager")

    graph = torch.cuda.CUDAGraph()
    tb.copy_(pristine)
    torch.cuda.synchronize(dev)
    with torch.cuda.graph(graph, stream=side):
        call()

    def replay(tag):
        tb.copy_(pristine)
        for t in (acc, nxt, amax):
            t.fill_(-5)
        reg.fill_(float("nan"))
        torch.cuda.synchronize(dev)
        graph.replay()
        torch.cuda.synchronize(dev)
        check(tag)

    replay("replay before growth")

    # 40,000 requests x 10 rows: about 3.5 MB of workspace, so the stream's
    # workspace grows to a new buffer while the graph still holds the old one.
    large = _batch(rng, 40000, 9, 16)
    ref_large = oracle.verify(*large)
    Ll, Ld, Lk, Lt, Lc, Lb = _device(dev, *large)
    print("case workspace growth: 40,000 requests x 10 rows, V = 16 f32", flush=True)
    with torch.cuda.stream(side):
        a_l, n_l = asd.asd_verify(Ll, Ld, Lk, Lt, Lc, Lb)
    torch.cuda.synchronize(dev)
    assert np.array_equal(a_l.cpu().numpy(), ref_large["accept_len"])
    assert np.array_equal(n_l.cpu().numpy(), ref_large["next_token"])
    assert _same(Lb.cpu().numpy(), ref_large["budget"])

    for k in range(3):
        replay("replay %d after growth" % k)
