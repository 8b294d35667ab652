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


def _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len,
            fused=False):
    n = w.rows_per_call
    for b in range(blocks):
        lg = logits[b * n:(b + 1) * n]
        dr = draft[b * n:(b + 1) * n]
        if fused:
            asd.asd_verify_commit(lg, dr, lens, tau, cap, budget, tokens, seq_len, workspace=ws,
                                  out_accept_len=acc[b], out_next_token=nxt[b])
        else:
            asd.asd_verify_ws(lg, dr, lens, tau, cap, budget, ws, out_accept_len=acc[b],
                              out_next_token=nxt[b])
            asd.asd_commit(dr, lens, acc[b], nxt[b], tokens, seq_len)


@pytest.mark.parametrize("cfg,library_ws", [(2, True), (5, True), (5, False)])
def test_verify_commit_matches_oracle_and_the_two_calls(cfg, library_ws):
    """asd_verify_commit equals asd_verify then asd_commit, and the oracle's
    verify then commit, on every output (requests that do not fit included)."""
    w = W.make_config(cfg, batch=40 if cfg == 2 else 300)
    rng = np.random.default_rng(10 + cfg)
    n = w.num_requests
    cap = 24
    start = rng.integers(0, 12, n).astype(np.int64)
    start[::7] = cap - 3
    start[3] = -1
    tokens0 = rng.integers(-5, 5, size=(n, cap)).astype(np.int32)
    logits = t(w.logits.view(np.int16)).view(torch.bfloat16)
    ws = None
    if not library_ws:
        ws = torch.zeros(asd.asd_workspace_bytes(torch.bfloat16, w.vocab, n, w.rows_per_call),
                         dtype=torch.uint8, device=DEV)
    budget = t(w.budget.copy())
    tok, sl = t(tokens0.copy()), t(start.copy())
    done = torch.empty(n, dtype=torch.int32, device=DEV)
    amax = torch.empty(w.rows_per_call, dtype=torch.int32, device=DEV)
    acc, nxt = asd.asd_verify_commit(logits, t(w.draft_tokens), t(w.block_lens), t(w.tau),
                                     t(w.exc_cap), budget, tok, sl, out_committed=done,
                                     out_argmax=amax, workspace=ws)
    # the two calls
    budget2 = t(w.budget.copy())
    tok2, sl2 = t(tokens0.copy()), t(start.copy())
    done2 = torch.empty(n, dtype=torch.int32, device=DEV)
    acc2, nxt2 = asd.asd_verify(logits, t(w.draft_tokens), t(w.block_lens), t(w.tau),
                                t(w.exc_cap), budget2)
    asd.asd_commit(t(w.draft_tokens), t(w.block_lens), acc2, nxt2, tok2, sl2, out_committed=done2)
    torch.cuda.synchronize()
    ref = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    r_tok, r_sl, r_done = oracle.commit(w.draft_tokens, w.block_lens, ref["accept_len"],
                                        ref["next_token"], tokens0, start)
    got = [x.cpu().numpy() for x in (acc, nxt, budget, tok, sl, done, amax)]
    two = [x.cpu().numpy() for x in (acc2, nxt2, budget2, tok2, sl2, done2)]
    want = [ref["accept_len"], ref["next_token"], ref["budget"], r_tok, r_sl, r_done,
            ref["argmax"]]
    for k, (g, r) in enumerate(zip(got, want)):
        assert np.array_equal(g.view(np.uint32) if g.dtype == np.float32 else g,
                              r.view(np.uint32) if r.dtype == np.float32 else r), k
    for k, (g, r) in enumerate(zip(got, two)):
        assert np.array_equal(g.view(np.uint32) if g.dtype == np.float32 else g,
                              r.view(np.uint32) if r.dtype == np.float32 else r), k
    assert r_done.min() == 0 and r_done.max() > 1


def test_verify_commit_with_offsets_and_unverified_requests():
    """Explicit offsets with a gap, requests whose rows do not fit (they commit
    nothing and keep their lengths) and one with K < 0, read as K = 0 (it commits
    its one emitted token)."""
    rng = np.random.default_rng(78)
    vocab, rows = 3000, 120
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    y = np.argmax(z, axis=1)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
    lens = np.array([8, 0, 5, -1, 8, 3, 12, 8], dtype=np.int32)
    offs = np.array([0, 10, 12, 20, 30, 117, 100, -4], dtype=np.int64)
    n = len(lens)
    budget0 = np.tile(np.array([[3.0, 0.5]], np.float32), (n, 1))
    tau = np.full(n, 2.0, np.float32)
    capx = np.full(n, 1, np.int32)
    capacity = 16
    start = np.array([0, 3, 15, 2, 4, 0, 1, 0], dtype=np.int64)
    tokens0 = np.full((n, capacity), -9, np.int32)
    budget = t(budget0.copy())
    tok, sl = t(tokens0.copy()), t(start.copy())
    done = torch.empty(n, dtype=torch.int32, device=DEV)
    acc, nxt = asd.asd_verify_commit(t(z), t(draft), t(lens), t(tau), t(capx), budget, tok, sl,
                                     row_offsets=t(offs), out_committed=done)
    torch.cuda.synchronize()
    ref = oracle.verify(z, draft, lens, tau, capx, budget0, offs)
    r_tok, r_sl, r_done = oracle.commit(draft, lens, ref["accept_len"], ref["next_token"],
                                        tokens0, start, offs)
    assert np.array_equal(acc.cpu().numpy(), ref["accept_len"])
    assert np.array_equal(nxt.cpu().numpy(), ref["next_token"])
    assert np.array_equal(tok.cpu().numpy(), r_tok)
    assert np.array_equal(sl.cpu().numpy(), r_sl)
    assert np.array_equal(done.cpu().numpy(), r_done)
    assert list(r_done[[3, 5, 7]]) == [1, 0, 0]


@pytest.mark.parametrize("fused", [False, True])
def test_graph_captured_rounds_match_eager_and_oracle(fused):
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
    _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len, fused)
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
        _rounds(w, blocks, logits, draft, lens, tau, cap, budget, ws, acc, nxt, tokens, seq_len,
                fused)
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


def test_checkpoint_resume_across_sessions_is_bit_identical(tmp_path):
    """Workload 1's 64 sequential rounds (verify and commit, asd_verify_commit)
    run as two sessions: after 32 rounds the request state -- the ledger
    (B, s) of Sec. 3.2 and the committed tokens and length of Sec. 3.3 -- is
    copied to the host and saved to a file, the library's workspaces are
    released and every device buffer is dropped; a second session loads the
    file into fresh device buffers and runs the other 32 rounds.  The result
    equals the uninterrupted 64-round run and the oracle's verify then commit,
    bit for bit."""
    w = W.make_config(1)
    n = w.rows_per_call
    capacity = w.blocks * (int(w.block_lens.max()) + 1)
    logits_all, draft_all = w.logits, w.draft_tokens

    def session(first, last, ledger, tokens, seq_len):
        lg = t(logits_all[first * n:last * n])
        dr = t(draft_all[first * n:last * n])
        lens, tau, cap = t(w.block_lens), t(w.tau), t(w.exc_cap)
        budget, tok, sl = t(ledger), t(tokens), t(seq_len)
        for b in range(last - first):
            asd.asd_verify_commit(lg[b * n:(b + 1) * n], dr[b * n:(b + 1) * n], lens, tau, cap,
                                  budget, tok, sl)
        torch.cuda.synchronize()
        return budget.cpu().numpy(), tok.cpu().numpy(), sl.cpu().numpy()

    ledger0 = w.budget.copy()
    tokens0 = np.zeros((1, capacity), np.int32)
    seq0 = np.zeros(1, np.int64)
    print("case checkpoint/resume: workload 1, 64 rounds uninterrupted", flush=True)
    whole = session(0, w.blocks, ledger0, tokens0, seq0)

    print("case checkpoint/resume: 32 rounds, save, release, 32 rounds", flush=True)
    first = session(0, 32, ledger0, tokens0, seq0)
    path = tmp_path / "asd_state.npz"
    np.savez(path, ledger=first[0], tokens=first[1], seq_len=first[2])
    del first
    torch.cuda.synchronize()
    asd.asd_release()
    torch.cuda.empty_cache()
    with np.load(path) as f:
        state = (f["ledger"].copy(), f["tokens"].copy(), f["seq_len"].copy())
    resumed = session(32, w.blocks, *state)

    ledger = ledger0.copy()
    r_tok, r_sl = tokens0.copy(), seq0.copy()
    for b in range(w.blocks):
        lg, dr = w.call(b)
        r = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ledger)
        ledger = r["budget"]
        r_tok, r_sl, _ = oracle.commit(dr, w.block_lens, r["accept_len"], r["next_token"],
                                       r_tok, r_sl)
    for got in (whole, resumed):
        assert np.array_equal(got[0].view(np.uint32), ledger.view(np.uint32))
        assert np.array_equal(got[1], r_tok)
        assert np.array_equal(got[2], r_sl)
    assert ledger[0, 1] > 0 and r_sl[0] > w.blocks      # exceptions were accepted


@pytest.mark.parametrize("num_requests", [3000, 8193, 70000])
def test_commit_packed_layout_any_request_count(num_requests):
    """asd_commit with row_offsets NULL at batch sizes above the 1,024 that
    one wavefront per request can sum on its own: against the oracle, with
    negative and zero K, accepted lengths out of range, unverified requests
    and tokens that do not fit."""
    rng = np.random.default_rng(num_requests)
    n = num_requests
    lens = rng.integers(-1, 7, n).astype(np.int32)
    k = np.maximum(lens, 0)
    rows = int(np.sum(k + 1))
    draft = rng.integers(0, 1000, rows).astype(np.int32)
    acc = np.minimum(rng.integers(0, 8, n), k).astype(np.int32)
    acc[rng.random(n) < 0.01] = 9                                 # outside [0, K]
    nxt = rng.integers(0, 1000, n).astype(np.int32)
    nxt[rng.random(n) < 0.02] = -1                                # not verified
    capacity = 12
    start = rng.integers(0, 6, n).astype(np.int64)
    start[rng.random(n) < 0.05] = capacity - 2                     # may not fit
    tokens0 = rng.integers(-5, 5, size=(n, capacity)).astype(np.int32)
    print("case commit packed: %d requests, %d rows" % (n, rows), flush=True)
    tok, sl = t(tokens0.copy()), t(start.copy())
    done = torch.empty(n, dtype=torch.int32, device=DEV)
    asd.asd_commit(t(draft), t(lens), t(acc), t(nxt), tok, sl, out_committed=done)
    torch.cuda.synchronize()
    r_tok, r_sl, r_done = oracle.commit(draft, lens, acc, nxt, tokens0, start)
    assert np.array_equal(tok.cpu().numpy(), r_tok)
    assert np.array_equal(sl.cpu().numpy(), r_sl)
    assert np.array_equal(done.cpu().numpy(), r_done)
    assert (r_done == 0).any() and (r_done > 1).any()
