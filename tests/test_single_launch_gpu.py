"""Small calls (few row tiles and requests) run as one launch when the call
uses a library workspace: the last row tile to finish runs the scan, found
through a counter in the workspace header that every call leaves at zero.
These tests check that form against the oracle and against the two-launch
form (a caller workspace), over random small calls, 1,000 repeated calls,
graph replays and two streams in flight."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W
from asd_gpu import device_logits
from test_fuzz_gpu import _run_block

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.mark.parametrize("block,large_vocab,caller", [
    (0, False, False), (1, False, False), (2, True, False), (3, True, False),
    (0, False, True), (2, True, True)])
def test_random_small_calls_match_the_oracle(block, large_vocab, caller):
    """At most eight requests: with the library workspace most of these calls
    take the single launch (with whole rows or split rows, commit or not, raw
    gate, explicit offsets, special values); with a caller workspace the same
    calls take two launches."""
    _run_block(np.random.default_rng(9000 + block), "small %d%s" % (block, " caller" if caller
                                                                     else ""),
               large_vocab, max_requests=8, caller_workspace=caller, cases=40)


def _workload1_tensors():
    w = W.make_config(1)
    lens, tau, cap = (torch.from_numpy(x).to(DEV) for x in (w.block_lens, w.tau, w.exc_cap))
    return w, device_logits(w.logits, DEV), torch.from_numpy(w.draft_tokens).to(DEV), lens, tau, cap


def test_repeated_single_launch_calls_are_bit_identical():
    """1,000 calls of workload 1's first block from the same ledger: the
    counter is back at zero after every call, so each call equals the first
    and the oracle."""
    w, logits, draft, lens, tau, cap = _workload1_tensors()
    n = w.rows_per_call
    lg, dr = logits[:n], draft[:n]
    pristine = torch.from_numpy(w.budget.copy()).to(DEV)
    calls = 1000
    acc = torch.empty((calls, 1), dtype=torch.int32, device=DEV)
    nxt = torch.empty((calls, 1), dtype=torch.int32, device=DEV)
    spent = torch.empty((calls, 2), dtype=torch.float32, device=DEV)
    amax = torch.empty((calls, n), dtype=torch.int32, device=DEV)
    budget = pristine.clone()
    print("case single launch: 1,000 calls of workload 1's first block", flush=True)
    for c in range(calls):
        budget.copy_(pristine)
        asd.asd_verify(lg, dr, lens, tau, cap, budget, out_accept_len=acc[c], out_next_token=nxt[c],
                       out_argmax=amax[c])
        spent[c].copy_(budget[0])
    torch.cuda.synchronize()
    l0, d0 = w.call(0)
    ref = oracle.verify(l0, d0, w.block_lens, w.tau, w.exc_cap, w.budget)
    assert (acc.cpu().numpy() == ref["accept_len"]).all()
    assert (nxt.cpu().numpy() == ref["next_token"]).all()
    assert (amax.cpu().numpy() == ref["argmax"][None, :]).all()
    assert (spent.cpu().numpy().view(np.uint32) == ref["budget"][0].view(np.uint32)).all()


def test_small_call_rounds_replay_from_a_graph():
    """Eight sequential rounds (verify and commit): the eager calls take the
    single launch, the captured ones the two-launch form; the rounds are
    captured once and replayed three times from the pristine state, and every
    replay equals the oracle."""
    w, logits, draft, lens, tau, cap = _workload1_tensors()
    n = w.rows_per_call
    rounds = 8
    pristine = torch.from_numpy(w.budget.copy()).to(DEV)
    budget = pristine.clone()
    capacity = rounds * 9
    tokens = torch.zeros((1, capacity), dtype=torch.int32, device=DEV)
    seq_len = torch.zeros(1, dtype=torch.int64, device=DEV)
    acc = torch.empty((rounds, 1), dtype=torch.int32, device=DEV)
    nxt = torch.empty((rounds, 1), dtype=torch.int32, device=DEV)

    def run():
        for b in range(rounds):
            asd.asd_verify_commit(logits[b * n:(b + 1) * n], draft[b * n:(b + 1) * n], lens, tau,
                                  cap, budget, tokens, seq_len, out_accept_len=acc[b],
                                  out_next_token=nxt[b])

    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):          # the stream's library workspace exists before capture
        run()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run()
    ledger = w.budget.copy()
    r_tok = np.zeros((1, capacity), np.int32)
    r_sl = np.zeros(1, np.int64)
    r_acc, r_nxt = [], []
    for b in range(rounds):
        lg, dr = w.call(b)
        r = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ledger)
        ledger = r["budget"]
        r_acc.append(r["accept_len"])
        r_nxt.append(r["next_token"])
        r_tok, r_sl, _ = oracle.commit(dr, w.block_lens, r["accept_len"], r["next_token"],
                                       r_tok, r_sl)
    print("case single launch: graph of 8 rounds, 3 replays", flush=True)
    for replay in range(3):
        budget.copy_(pristine)
        tokens.zero_()
        seq_len.zero_()
        acc.fill_(-5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(acc.cpu().numpy(), np.stack(r_acc)), replay
        assert np.array_equal(nxt.cpu().numpy(), np.stack(r_nxt)), replay
        assert np.array_equal(budget.cpu().numpy().view(np.uint32), ledger.view(np.uint32)), replay
        assert np.array_equal(tokens.cpu().numpy(), r_tok), replay
        assert np.array_equal(seq_len.cpu().numpy(), r_sl), replay


def test_single_launch_on_two_streams_in_flight():
    """Two streams, each with its own library workspace and counter, issue
    single-launch calls concurrently; each sequence equals the oracle."""
    w, logits, draft, lens, tau, cap = _workload1_tensors()
    n = w.rows_per_call
    streams = [torch.cuda.Stream(DEV), torch.cuda.Stream(DEV)]
    budgets = [torch.from_numpy(w.budget.copy()).to(DEV) for _ in streams]
    accs = [torch.empty((w.blocks, 1), dtype=torch.int32, device=DEV) for _ in streams]
    nxts = [torch.empty((w.blocks, 1), dtype=torch.int32, device=DEV) for _ in streams]
    torch.cuda.synchronize()
    print("case single launch: two streams x 64 rounds", flush=True)
    for b in range(w.blocks):
        for k, st in enumerate(streams):
            with torch.cuda.stream(st):
                asd.asd_verify(logits[b * n:(b + 1) * n], draft[b * n:(b + 1) * n], lens, tau,
                               cap, budgets[k], out_accept_len=accs[k][b],
                               out_next_token=nxts[k][b])
    torch.cuda.synchronize()
    ledger = w.budget.copy()
    r_acc, r_nxt = [], []
    for b in range(w.blocks):
        lg, dr = w.call(b)
        r = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ledger)
        ledger = r["budget"]
        r_acc.append(r["accept_len"])
        r_nxt.append(r["next_token"])
    for k in range(2):
        assert np.array_equal(accs[k].cpu().numpy(), np.stack(r_acc)), k
        assert np.array_equal(nxts[k].cpu().numpy(), np.stack(r_nxt)), k
        assert np.array_equal(budgets[k].cpu().numpy().view(np.uint32), ledger.view(np.uint32)), k
