"""Randomized parity sweep: many verifier calls with random shapes (whole rows
and split plans), layouts, controls and special values, each compared bit for
bit with the oracle (accept lengths, next tokens, per-row argmax and regret,
the ledger, the commit and the device error word)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W
from asd_gpu import describe, device_logits, mismatches

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

SPECIAL_F32 = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00000,
                        0x7F800001, 0xFF800001, 0x3F800000, 0xBF800000, 0x00000001, 0x80000001],
                       dtype=np.uint32)


def _case(rng, large_vocab=False, max_requests=None):
    """One random call.  With `large_vocab` the vocabulary is 8,191 to 151,936
    entries and there are at most six requests, so rows are split over several
    workgroups (a split plan); otherwise V <= 5,003 and rows are whole.
    `max_requests` bounds the number of requests further."""
    dtype = "bf16" if rng.random() < 0.6 else "f32"
    if large_vocab:
        vocab = int(rng.choice([8191, 16385, 32000, 50257, 129280, 151936]))
        n = int(rng.integers(1, 7))
    else:
        vocab = int(rng.choice([1, 2, 7, 64, 257, 1000, 1031, 4096, 5003]))
        n = int(rng.integers(1, 40))
    if max_requests is not None:
        n = min(n, int(rng.integers(1, max_requests + 1)))
    lens = rng.integers(-2, 20, n).astype(np.int32)
    offsets = None
    rows = int(np.sum(np.maximum(lens, 0) + 1))
    if rng.random() < 0.3:
        # Explicit offsets: requests in order with gaps between them (never
        # overlapping, so each row belongs to at most one request), and a few
        # moved out of the batch.
        pos, offs = 0, []
        for k in lens:
            pos += int(rng.integers(0, 3))
            offs.append(pos)
            pos += max(int(k), 0) + 1
        rows = pos + int(rng.integers(0, 4))
        offsets = np.array(offs, dtype=np.int64)
        bad = rng.random(n) < 0.1
        offsets[bad] = rng.choice(np.array([-1, rows, rows + 7], np.int64), int(bad.sum()))
    z = (rng.integers(-12, 13, size=(rows, vocab)) / 4.0).astype(np.float32)
    if rng.random() < 0.5:
        z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    if rng.random() < 0.4:                        # special values in a few places
        k = int(rng.integers(1, 1 + rows))
        z.reshape(-1)[rng.integers(0, z.size, k)] = rng.choice(SPECIAL_F32, k).view(np.float32)
    if dtype == "bf16":
        bits = (z.view(np.uint32) >> 16).astype(np.uint16)    # truncation keeps NaN and inf
        logits = bits
        y = oracle.argmax_rows(bits)
    else:
        logits = z
        y = oracle.argmax_rows(z)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(-1, vocab + 1, rows)).astype(np.int32)
    tau = rng.choice(np.array([-1.0, 0.0, 0.25, 0.5, 1.0, 2.0, np.inf, np.nan], np.float32), n)
    cap = rng.choice(np.array([0, 1, 2, 5, 2**31 - 1], np.int32), n)
    tot = rng.choice(np.array([0.0, -0.0, 0.5, 2.0, 8.0, np.inf], np.float32), n)
    spent = np.minimum(rng.choice(np.array([0.0, 0.25, 1.0], np.float32), n), tot)
    budget = np.stack([tot, spent], axis=1).astype(np.float32)
    raw_gate = bool(rng.random() < 0.25)
    return dtype, logits, draft, lens, offsets, tau, cap, budget, raw_gate


@pytest.mark.parametrize("block", range(6))
def test_random_calls_match_the_oracle(block):
    _run_block(np.random.default_rng(5000 + block), "fuzz %d" % block, large_vocab=False)


@pytest.mark.parametrize("block", range(2))
def test_random_split_plan_calls_match_the_oracle(block):
    _run_block(np.random.default_rng(7000 + block), "fuzz-split %d" % block, large_vocab=True)


def _run_block(rng, name, large_vocab, max_requests=None, caller_workspace=False, cases=25):
    """`cases` random calls against the oracle.  With `caller_workspace` every
    call gets a workspace of its own (so the two-launch form runs); otherwise
    the library's, where small calls run as one launch."""
    for case in range(cases):
        dtype, logits, draft, lens, offsets, tau, cap, budget, raw_gate = _case(
            rng, large_vocab, max_requests)
        rows, vocab = logits.shape
        n = len(lens)
        label = "%s.%d: %s rows %d vocab %d requests %d offsets %s raw_gate %s" % (
            name, case, dtype, rows, vocab, n, offsets is not None, raw_gate)
        print(label, flush=True)
        ref = oracle.verify(logits, draft, lens, tau, cap, budget, offsets, raw_gate=raw_gate)
        capacity = 24
        start = rng.integers(-1, 12, n).astype(np.int64)
        tokens0 = np.full((n, capacity), -5, np.int32)
        r_tok, r_sl, r_done = oracle.commit(draft, lens, ref["accept_len"], ref["next_token"],
                                            tokens0, start, offsets)
        tl = device_logits(logits, DEV)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
        tb = t(budget.copy())
        amax = torch.full((rows,), -7, dtype=torch.int32, device=DEV)
        regret = torch.full((rows,), float("nan"), dtype=torch.float32, device=DEV)
        to = None if offsets is None else t(offsets)
        torch.cuda.synchronize()
        asd.asd_device_error(clear=True)
        use_commit = (not raw_gate) and rng.random() < 0.5
        ws = None
        if caller_workspace:
            ws = torch.full((asd.asd_workspace_bytes(tl.dtype, vocab, n, rows),), 0xA5,
                            dtype=torch.uint8, device=DEV)
        if use_commit:
            tok, sl = t(tokens0.copy()), t(start.copy())
            done = torch.empty(n, dtype=torch.int32, device=DEV)
            acc, nxt = asd.asd_verify_commit(tl, t(draft), t(lens), t(tau), t(cap), tb, tok, sl,
                                             row_offsets=to, out_argmax=amax, out_regret=regret,
                                             out_committed=done, workspace=ws)
        else:
            acc, nxt = asd.asd_verify_ex(tl, t(draft), t(lens), t(tau), t(cap), tb,
                                         flags=asd.ASD_GATE_RAW if raw_gate else 0,
                                         workspace=ws, row_offsets=to, out_argmax=amax,
                                         out_regret=regret)
        torch.cuda.synchronize()
        word = asd.asd_device_error(clear=True)
        g = {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
             "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
             "budget": tb.cpu().numpy()}
        bad = mismatches(g, ref)
        assert not bad, "%s differs in %s: %s" % (label, bad, describe(g, ref))
        expect = ref["error"]
        if use_commit:
            assert np.array_equal(tok.cpu().numpy(), r_tok), label
            assert np.array_equal(sl.cpu().numpy(), r_sl), label
            assert np.array_equal(done.cpu().numpy(), r_done), label
            if np.any((ref["next_token"] >= 0) & (r_done == 0)):
                expect |= asd.ASD_DEVERR_COMMIT
        assert word == expect, "%s: error word %d, expected %d" % (label, word, expect)
