"""Pins of the oracle's opportunity statistic (Sec. 3.1, Eq. 4)."""
import json
import os

import numpy as np

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _taus(raw):
    return np.array([np.inf if t == "inf" else t for t in raw], dtype=np.float32)


def test_figure1_opportunity_counts():
    with open(os.path.join(GOLDEN, "fig1_asd_example.json")) as f:
        fx = json.load(f)
    with open(os.path.join(GOLDEN, "fig1_opportunity.json")) as f:
        op = json.load(f)
    logits = np.array(fx["logits"], dtype=np.float32)
    draft = np.array(fx["draft_tokens"], dtype=np.int32)
    out = oracle.verify(logits, draft, [6], [1.0], [1], [[1.0, 0.0]])
    counts, m = oracle.opportunity(draft, out["argmax"], out["regret"], fx["vocab"], [6],
                                   _taus(op["taus"]), op["ps"])
    assert m == op["expected_mismatches"]
    assert counts.tolist() == op["expected_counts"]


def run_lengths(draft, y, lens):
    """Independent formulation: for every draft position, the length of the run
    of target-greedy drafts that starts right after it (a reverse scan)."""
    out = []
    o = 0
    for K in lens:
        match = (draft[o:o + K] == y[o:o + K]).astype(np.int64)
        run = np.zeros(K, dtype=np.int64)
        after = 0
        for i in range(K - 1, -1, -1):
            run[i] = after
            after = after + 1 if match[i] else 0
        out.append((match, run))
        o += K + 1
    return out


def test_counts_equal_run_length_formulation_and_p0_identity():
    rng = np.random.default_rng(44)
    taus = np.array([0.0, 0.5, 1.0, 3.0, np.inf], dtype=np.float32)
    ps = np.array([0, 1, 2, 3, 5, 8], dtype=np.int32)
    for trial in range(40):
        w = W.make_config(int(rng.choice([2, 3, 5])), seed=trial, batch=int(rng.integers(1, 9)),
                          vocab=int(rng.integers(50, 400)))
        out = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
        counts, m = oracle.opportunity(w.draft_tokens, out["argmax"], out["regret"], w.vocab,
                                       w.block_lens, taus, ps)
        expect = np.zeros_like(counts)
        total = 0
        o = 0
        for K, (match, run) in zip(w.block_lens, run_lengths(w.draft_tokens, out["argmax"],
                                                              w.block_lens)):
            r = out["regret"][o:o + K]
            for i in np.flatnonzero(match == 0):
                total += 1
                for a, t in enumerate(taus):
                    if r[i] <= t:
                        expect[a] += (run[i] >= ps).astype(np.uint64)
            o += K + 1
        assert m == total
        assert np.array_equal(counts, expect)
        # p = 0: the fraction of mismatches with r <= tau
        assert counts[-1, 0] == m
        # monotone: nondecreasing in tau, nonincreasing in p
        assert np.all(np.diff(counts.astype(np.int64), axis=0) >= 0)
        assert np.all(np.diff(counts.astype(np.int64), axis=1) <= 0)


def test_counts_skip_invalid_requests():
    draft = np.array([1, 2, 3, 0, 0, 0], dtype=np.int32)
    y = np.array([1, 9, 3, 0, 0, 0], dtype=np.int32)
    reg = np.array([0.0, 1.0, 0.0, 0.0, 0.0, 0.0], dtype=np.float32)
    c1, m1 = oracle.opportunity(draft, y, reg, 10, [3, -1, 9], [2.0], [0, 1, 2],
                                row_offsets=[0, 3, 4])
    assert m1 == 1 and c1.tolist() == [[1, 1, 0]]
