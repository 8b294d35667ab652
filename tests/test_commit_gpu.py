"""GPU commit step (Sec. 3.3) and graph-captured decoding rounds, against the
oracle and against eager execution."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def t(a, dtype=None):
    a = np.ascontiguousarray(a if dtype is None else np.asarray(a, dtype=dtype))
    return torch.from_numpy(a).to(DEV)


@pytest.mark.parametrize("cfg", [2, 5])
def test_commit_matches_oracle(cfg):
    w = W.make_config(cfg, batch=40 if cfg == 2 else 300)
    rng = np.random.default_rng(cfg)
    n = w.num_requests
    cap = 24
    start = rng.integers(0, 12, n).astype(np.int64)
    start[::7] = cap - 3                                  # some will not fit
    start[3] = -1                                         # invalid length
    tokens0 = rng.integers(-5, 5, size=(n, cap)).astype(np.int32)
    budget = t(w.budget.copy())
    acc, nxt = asd.asd_verify(t(w.logits.view(np.int16)).view(torch.bfloat16), t(w.draft_tokens),
                              t(w.block_lens), t(w.tau), t(w.exc_cap), budget)
    tok = t(tokens0.copy())
    sl = t(start.copy())
    done = torch.empty(n, dtype=torch.int32, device=DEV)
    asd.asd_commit(t(w.draft_tokens), t(w.block_lens), acc, nxt, tok, sl, out_committed=done)
    torch.cuda.synchronize()
    ref = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    r_tok, r_sl, r_done = oracle.commit(w.draft_tokens, w.block_lens, ref["accept_len"],
                                        ref["next_token"], tokens0, start)
    assert np.array_equal(tok.cpu().numpy(), r_tok)
    assert np.array_equal(sl.cpu().numpy(), r_sl)
    assert np.array_equal(done.cpu().numpy(), r_done)
    assert r_done.min() == 0 and r_done.max() > 1


def _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len):
    n = w.rows_per_call
    for b in range(blocks):
        lg = logits[b * n:(b + 1) * n]
        dr = draft[b * n:(b + 1) * n]
        asd.asd_verify_ws(lg, dr, lens, tau, cap, budget, ws, out_accept_len=acc[b],
                          out_next_token=nxt[b])
        asd.asd_commit(dr, lens, acc[b], nxt[b], tokens, seq_len)


def test_graph_captured_rounds_match_eager_and_oracle():
    blocks = 16
    w = W.make_config(1, batch=blocks)
    logits, draft = t(w.logits), t(w.draft_tokens)
    lens, tau, cap = t(w.block_lens), t(w.tau), t(w.exc_cap)
    nbytes = asd.asd_workspace_bytes(torch.float32, w.vocab, 1, w.rows_per_call)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    capacity = blocks * 9 + 1
    pristine = (t(w.budget.copy()), torch.zeros((1, capacity), dtype=torch.int32, device=DEV),
                torch.zeros(1, dtype=torch.int64, device=DEV))
    budget, tokens, seq_len = (x.clone() for x in pristine)
    acc = torch.empty((blocks, 1), dtype=torch.int32, device=DEV)
    nxt = torch.empty((blocks, 1), dtype=torch.int32, device=DEV)

    # eager
    _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len)
    torch.cuda.synchronize()
    eager = [x.cpu().numpy().copy() for x in (budget, tokens, seq_len, acc, nxt)]

    # oracle: the same rounds on the host
    ledger = w.budget.copy()
    r_tok = np.zeros((1, capacity), np.int32)
    r_sl = np.zeros(1, np.int64)
    for b in range(blocks):
        lg, dr = w.call(b)
        out = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ledger)
        ledger = out["budget"]
        r_tok, r_sl, _ = oracle.commit(dr, w.block_lens, out["accept_len"], out["next_token"],
                                       r_tok, r_sl)
        assert eager[3][b, 0] == out["accept_len"][0] and eager[4][b, 0] == out["next_token"][0]
    assert np.array_equal(eager[0].view(np.uint32), ledger.view(np.uint32))
    assert np.array_equal(eager[1], r_tok) and np.array_equal(eager[2], r_sl)

    # captured once, replayed three times from the pristine state
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        for x, p in zip((budget, tokens, seq_len), pristine):
            x.copy_(p)
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=side):
        _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len)
    for replay in range(3):
        for x, p in zip((budget, tokens, seq_len), pristine):
            x.copy_(p)
        acc.fill_(-5)
        nxt.fill_(-5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [x.cpu().numpy() for x in (budget, tokens, seq_len, acc, nxt)]
        for a, b in zip(got, eager):
            assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                  b.view(np.uint32) if b.dtype == np.float32 else b), replay
