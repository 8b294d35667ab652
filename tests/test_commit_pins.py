"""Pins of the oracle's commit step (Sec. 3.3; Algorithm 1's return)."""
import json
import os

import numpy as np

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_figure1_emitted_sequences():
    # ASD emits A B E F G then recovers with H; strict emits A B then E'
    # (Figure 1 caption, Sec. 1).  Ids: A..H = 0..7, E' = 8.
    with open(os.path.join(GOLDEN, "fig1_asd_example.json")) as f:
        fx = json.load(f)
    logits = np.array(fx["logits"], dtype=np.float32)
    draft = np.array(fx["draft_tokens"], dtype=np.int32)
    for mode, expect in (("asd", [0, 1, 4, 5, 6, 7]), ("strict", [0, 1, 8])):
        p = fx[mode]
        out = oracle.verify(logits, draft, [6], [p["tau"]], [p["exc_cap"]],
                            [[p["budget_total"], p["budget_spent"]]])
        tok, sl, done = oracle.commit(draft, [6], out["accept_len"], out["next_token"],
                                      np.full((1, 10), -9, np.int32), [0])
        assert tok[0, :sl[0]].tolist() == expect and done[0] == len(expect)
        assert np.all(tok[0, sl[0]:] == -9)


def test_strict_commits_the_target_greedy_trajectory_and_asd_differs_only_at_exceptions():
    """With B = 0 every committed token is the target's greedy token of its row
    (the strict rule preserves the greedy trajectory); with B > 0 the committed
    tokens differ from the greedy ones exactly at the accepted mismatches, at
    most M per block."""
    w = W.make_config(1, vocab=2000)
    cap_tokens = 64 * 9 + 4
    for total in (0.0, 4.0):
        ledger = np.array([[total, 0.0]], np.float32)
        tok = np.full((1, cap_tokens), -1, np.int32)
        sl = np.array([0], np.int64)
        greedy = []
        for b in range(w.blocks):
            lg, dr = w.call(b)
            out = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ledger)
            ledger = out["budget"]
            a = int(out["accept_len"][0])
            before = int(sl[0])
            tok, sl, done = oracle.commit(dr, w.block_lens, out["accept_len"],
                                          out["next_token"], tok, sl)
            assert done[0] == a + 1 and sl[0] == before + a + 1
            greedy.extend(out["argmax"][:a + 1].tolist())
            diff = np.sum(tok[0, before:before + a + 1] != out["argmax"][:a + 1])
            assert diff <= int(w.exc_cap[0]) if total > 0 else diff == 0
        committed = tok[0, :sl[0]].tolist()
        if total == 0.0:
            assert committed == greedy
        else:
            assert committed != greedy and ledger[0, 1] <= ledger[0, 0]


def test_commit_skips_what_does_not_fit():
    draft = np.array([5, 6, 7, 0, 1, 2, 3, 0], dtype=np.int32)
    lens = [3, 3]
    acc = np.array([2, 3], np.int32)
    nxt = np.array([9, 8], np.int32)
    tok, sl, done = oracle.commit(draft, lens, acc, nxt, np.zeros((2, 5), np.int32), [2, 2])
    assert tok[0].tolist() == [0, 0, 5, 6, 9] and sl[0] == 5 and done[0] == 3
    assert tok[1].tolist() == [0] * 5 and sl[1] == 2 and done[1] == 0      # 2 + 4 > 5
    tok, sl, done = oracle.commit(draft, lens, acc, nxt, np.zeros((2, 5), np.int32), [0, 1])
    assert tok[1].tolist() == [0, 1, 2, 3, 8] and sl[1] == 5               # 1 + 4 fits exactly
    tok, sl, done = oracle.commit(draft, lens, acc, np.array([-1, 8], np.int32),
                                  np.zeros((2, 9), np.int32), [0, -3])
    assert done.tolist() == [0, 0] and sl.tolist() == [0, -3]


def test_negative_block_length_commits_like_zero():
    """A negative K is read as 0 by the verifier (one bonus row), so its request
    emits one token, the argmax of that row, and the commit takes it."""
    logits = np.zeros((4, 3), dtype=np.float32)
    logits[0, 2] = 1.0
    logits[1, 1] = 1.0
    draft = np.array([2, 0, 1, 0], dtype=np.int32)
    lens = [-2, 2]
    out = oracle.verify(logits, draft, lens, [1.0] * 2, [1] * 2, [[0.0, 0.0]] * 2)
    assert out["accept_len"].tolist() == [0, 0] and out["next_token"].tolist() == [2, 1]
    tok, sl, done = oracle.commit(draft, lens, out["accept_len"], out["next_token"],
                                  np.full((2, 4), -1, np.int32), [1, 0])
    assert tok[0].tolist() == [-1, 2, -1, -1] and sl[0] == 2 and done[0] == 1
    assert tok[1].tolist() == [1, -1, -1, -1] and sl[1] == 1 and done[1] == 1
