"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself:
  * the paper's Figure 1 example (golden fixture),
  * exact greedy verification (Eq. 2), written independently here, which
    Algorithm 1 must reproduce when B = 0 (and when M = 0 or g < 0),
  * brute force over every prefix and every accepted-mismatch subset, in
    exact rational arithmetic, for the longest feasible prefix (Eqs. 9-12),
  * the paper's invariants (s' <= B after Eq. 13; Proposition 1),
  * numpy.argmax for the argmax order (Eq. 1), NaNs included: numpy's argmax
    returns the first NaN of a row, which is the order the verifier takes.
"""
import json
import math
import os
from fractions import Fraction
from itertools import combinations

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------- helpers

def strict_greedy(logits_f32, draft, lens, offsets=None):
    """Exact greedy verification, Eq. 2, with numpy's first-occurrence argmax."""
    y = np.argmax(logits_f32, axis=1)
    acc, nxt = [], []
    o = 0
    for i, K in enumerate(lens):
        K = int(K)
        if offsets is not None:
            o = int(offsets[i])
        a = 0
        while a < K and int(draft[o + a]) == int(y[o + a]):
            a += 1
        acc.append(a)
        nxt.append(int(y[o + a]))
        o += K + 1
    return np.array(acc), np.array(nxt)


# -------------------------------------------------------- Figure 1 example

def _fig1():
    with open(os.path.join(GOLDEN, "fig1_asd_example.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("mode", ["asd", "strict"])
def test_figure1_example(mode):
    fx = _fig1()
    logits = np.array(fx["logits"], dtype=np.float32)
    draft = np.array(fx["draft_tokens"], dtype=np.int32)
    p = fx[mode]
    out = oracle.verify(logits, draft, [fx["block_len"]], [p["tau"]], [p["exc_cap"]],
                        [[p["budget_total"], p["budget_spent"]]])
    exp = p["expected"]
    assert out["accept_len"][0] == exp["accept_len"]
    assert out["next_token"][0] == exp["next_token"]
    assert out["budget"][0, 1] == np.float32(exp["budget_spent"])
    assert list(out["argmax"]) == fx["row_argmax"]


def test_figure1_bf16_same_outcome():
    fx = _fig1()
    logits = W.f32_to_bf16(np.array(fx["logits"], dtype=np.float32))
    draft = np.array(fx["draft_tokens"], dtype=np.int32)
    p = fx["asd"]
    out = oracle.verify(logits, draft, [6], [p["tau"]], [p["exc_cap"]],
                        [[p["budget_total"], p["budget_spent"]]])
    assert (out["accept_len"][0], out["next_token"][0]) == (5, 7)


# ------------------------------------------------------ B = 0 is strict greedy

@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_zero_budget_is_strict_greedy(cfg):
    w = W.make_config(cfg, batch=6 if cfg != 1 else 4, vocab=4000)
    zero = np.zeros_like(w.budget)
    zero[:, 1] = 0.5                       # s is left untouched on the B = 0 path
    for b in range(w.blocks):
        lg, dr = w.call(b)
        out = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, zero)
        lf = lg if w.dtype == "f32" else W.bf16_to_f32(lg)
        acc, nxt = strict_greedy(lf, dr, w.block_lens)
        assert np.array_equal(out["accept_len"], acc)
        assert np.array_equal(out["next_token"], nxt)
        assert np.array_equal(out["budget"], zero)


def _tie_block(rng, K, V):
    """Integer logits in a tiny range so ties for the maximum are common."""
    logits = rng.integers(-2, 3, size=(K + 1, V)).astype(np.float32)
    y = np.argmax(logits, axis=1)
    draft = np.where(rng.random(K + 1) < 0.6, y, rng.integers(0, V, K + 1)).astype(np.int32)
    return logits, draft


def test_zero_budget_negative_zero_and_random_ties():
    rng = np.random.default_rng(11)
    for trial in range(300):
        K, V = int(rng.integers(0, 9)), int(rng.integers(1, 7))
        logits, draft = _tie_block(rng, K, V)
        total = -0.0 if trial % 2 else 0.0
        out = oracle.verify(logits, draft, [K], [rng.choice([0.25, 1.0, np.inf])],
                            [int(rng.integers(0, 5))], [[total, 0.0]])
        acc, nxt = strict_greedy(logits, draft, [K])
        assert out["accept_len"][0] == acc[0] and out["next_token"][0] == nxt[0]


def test_zero_cap_or_negative_gate_is_strict_greedy():
    rng = np.random.default_rng(5)
    for _ in range(300):
        K, V = int(rng.integers(0, 9)), int(rng.integers(1, 7))
        logits, draft = _tie_block(rng, K, V)
        acc, nxt = strict_greedy(logits, draft, [K])
        a = oracle.verify(logits, draft, [K], [1.0], [0], [[5.0, 0.0]])
        b = oracle.verify(logits, draft, [K], [-0.5], [4], [[5.0, 0.0]])
        for out in (a, b):
            assert out["accept_len"][0] == acc[0] and out["next_token"][0] == nxt[0]
            assert out["budget"][0, 1] == 0.0


def test_tie_mismatch_differs_from_strict_only_when_budget_positive():
    # The draft takes a value tied for the maximum at a higher index: a token-ID
    # mismatch with zero regret.  B = 0 must stop there; B > 0 accepts it at no
    # cost (it still counts against the cap), which is why B = 0 dispatches to
    # token-ID greedy instead of accepting r = 0 mismatches.
    logits = np.array([[1.0, 3.0, 3.0, 0.0],
                       [0.0, 0.0, 0.0, 2.0],
                       [2.0, 0.0, 0.0, 0.0]], dtype=np.float32)
    draft = np.array([2, 3, 0], dtype=np.int32)
    strict = oracle.verify(logits, draft, [2], [0.25], [1], [[0.0, 0.0]])
    asd = oracle.verify(logits, draft, [2], [0.25], [1], [[1.0, 0.0]])
    capped = oracle.verify(logits, draft, [2], [0.25], [0], [[1.0, 0.0]])
    assert (strict["accept_len"][0], strict["next_token"][0]) == (0, 1)
    assert (asd["accept_len"][0], asd["next_token"][0]) == (2, 0)
    assert asd["budget"][0, 1] == 0.0
    assert (capped["accept_len"][0], capped["next_token"][0]) == (0, 1)


# ---------------------------------------- brute force: longest feasible prefix

def _frac(v):
    return Fraction(float(v))


def brute_force_block(logits, draft, K, g, M, B, s, raw_gate=False):
    """Longest feasible prefix by Eqs. 9-12, two independent ways, exactly.
    With ``raw_gate`` every mismatch must satisfy r <= g instead of r / q <= g."""
    V = logits.shape[1]
    y = np.argmax(logits, axis=1)
    valid = [(0 <= int(draft[i]) < V) for i in range(K)]
    mism = [i for i in range(K) if not valid[i] or int(draft[i]) != int(y[i])]
    r = {}
    for i in mism:
        r[i] = (_frac(logits[i, y[i]]) - _frac(logits[i, draft[i]])) if valid[i] else None

    def gate_ok(i):
        if r[i] is None:
            return False
        q = 1 if raw_gate else K - (i + 1) + 1
        if math.isinf(g):
            return g > 0
        return r[i] <= _frac(g) * q

    room = None if math.isinf(B) else _frac(B) - _frac(s)

    def set_ok(S):
        if len(S) > M:
            return False
        if not all(gate_ok(i) for i in S):
            return False
        total = sum((r[i] for i in S), Fraction(0))
        return room is None or total <= room

    # (1) every prefix t checked against Eqs. 9-11 directly.
    best_t = 0
    for t in range(K + 1):
        if set_ok([i for i in mism if i < t]):
            best_t = t
    # (2) every subset of mismatch positions; a prefix is covered up to the
    #     first mismatch the subset leaves out (contiguity).
    best_s = 0
    for n in range(len(mism) + 1):
        for S in combinations(mism, n):
            if not set_ok(S):
                continue
            left_out = [i for i in mism if i not in S]
            best_s = max(best_s, left_out[0] if left_out else K)
    assert best_t == best_s
    return best_t, int(y[best_t])


def test_longest_feasible_prefix_brute_force():
    rng = np.random.default_rng(2608)
    gates = [-1.0, 0.0, 0.25, 0.5, 1.0, 1.5, np.inf]
    caps = [0, 1, 2, 3, 2**31 - 1]
    n_nontrivial = 0
    for trial in range(1500):
        K, V = int(rng.integers(0, 9)), int(rng.integers(1, 6))
        # Dyadic logits (multiples of 1/4 in [-2, 2]): every fp32 sum below is exact.
        logits = (rng.integers(-8, 9, size=(K + 1, V)) / 4.0).astype(np.float32)
        y = np.argmax(logits, axis=1)
        draft = np.where(rng.random(K + 1) < 0.55, y, rng.integers(0, V, K + 1)).astype(np.int32)
        if trial % 7 == 0 and K > 0:
            draft[int(rng.integers(0, K))] = int(rng.choice([-1, V, 2**31 - 1]))
        g = float(rng.choice(gates))
        M = int(rng.choice(caps))
        B = float(rng.choice([0.25, 0.5, 1.0, 2.0, 3.75, np.inf]))
        s = float(rng.choice([0.0, 0.25, 0.5])) if not math.isinf(B) else 0.0
        s = min(s, B)
        out = oracle.verify(logits, draft, [K], [g], [M], [[B, s]])
        a, nxt = brute_force_block(logits, draft, K, g, M, B, s)
        assert out["accept_len"][0] == a, (trial, K, V, g, M, B, s)
        assert out["next_token"][0] == nxt
        strict_a = strict_greedy(logits, draft, [K])[0][0]
        n_nontrivial += int(a > strict_a)
    assert n_nontrivial > 100          # the brute force exercised accepted mismatches


def test_raw_gate_variant_brute_force():
    """The raw-gate variant (r <= g at every accepted mismatch) against the
    same two-way brute force; it never accepts more than the paper's gate for
    g >= 0 (q >= 1), and equals it when every mismatch sits at q = 1."""
    rng = np.random.default_rng(2609)
    gates = [-1.0, 0.0, 0.25, 0.5, 1.0, 1.5, np.inf]
    n_differ = 0
    for trial in range(1200):
        K, V = int(rng.integers(0, 9)), int(rng.integers(1, 6))
        logits = (rng.integers(-8, 9, size=(K + 1, V)) / 4.0).astype(np.float32)
        y = np.argmax(logits, axis=1)
        draft = np.where(rng.random(K + 1) < 0.55, y, rng.integers(0, V, K + 1)).astype(np.int32)
        g = float(rng.choice(gates))
        M = int(rng.choice([0, 1, 2, 3, 2**31 - 1]))
        B = float(rng.choice([0.25, 1.0, 2.0, 3.75, np.inf]))
        raw = oracle.verify(logits, draft, [K], [g], [M], [[B, 0.0]], raw_gate=True)
        norm = oracle.verify(logits, draft, [K], [g], [M], [[B, 0.0]])
        a, nxt = brute_force_block(logits, draft, K, g, M, B, 0.0, raw_gate=True)
        assert raw["accept_len"][0] == a and raw["next_token"][0] == nxt, (trial, K, g, M, B)
        if g >= 0:
            assert raw["accept_len"][0] <= norm["accept_len"][0]
        n_differ += int(raw["accept_len"][0] != norm["accept_len"][0])
        if K > 0 and np.all(draft[:K - 1] == y[:K - 1]):      # only position K can mismatch
            assert raw["accept_len"][0] == norm["accept_len"][0]
    assert n_differ > 50               # the two gates were told apart
    # B = 0 dispatches to strict greedy under either gate
    logits = np.array([[0.0, 1.0], [1.0, 0.0], [0.0, 1.0]], dtype=np.float32)
    draft = np.array([0, 0, 0], dtype=np.int32)
    out = oracle.verify(logits, draft, [2], [np.inf], [5], [[0.0, 0.0]], raw_gate=True)
    assert (out["accept_len"][0], out["next_token"][0]) == (0, 1)


# --------------------------------------------------------- paper invariants

def test_ledger_never_exceeds_budget_and_cap_holds():
    """s' <= B by construction (Eq. 13); at most M exceptions per block (Eq. 10);
    accepted matches add no exception (Proposition 1)."""
    rng = np.random.default_rng(99)
    for trial in range(400):
        K, V = int(rng.integers(1, 17)), int(rng.integers(2, 40))
        logits = rng.normal(0.0, 1.0, size=(K + 1, V)).astype(np.float32)
        y = np.argmax(logits, axis=1)
        order = np.argsort(-logits, axis=1, kind="stable")
        draft = np.where(rng.random(K + 1) < 0.5, y, order[:, 1]).astype(np.int32)
        B = np.float32(rng.uniform(0.01, 3.0))
        s = np.float32(rng.uniform(0.0, 1.0)) * B
        M = int(rng.integers(0, 5))
        g = np.float32(rng.uniform(0.0, 2.0))
        out = oracle.verify(logits, draft, [K], [g], [M], [[B, s]])
        a = int(out["accept_len"][0])
        s_new = out["budget"][0, 1]
        assert s_new <= B
        assert s_new >= s
        mism = int(np.sum(draft[:a] != y[:a]))
        assert mism <= M
        if mism == 0:
            assert s_new == s               # no exception, no spend
        else:
            assert s_new > s or np.all(out["regret"][:a][draft[:a] != y[:a]] == 0)


def test_ledger_sum_matches_accepted_regrets():
    # s' - s is the regret of the accepted mismatches (Eq. 13).  With dyadic
    # values the fp32 arithmetic is exact and the check is a real identity.
    rng = np.random.default_rng(7)
    for _ in range(300):
        K, V = int(rng.integers(1, 12)), int(rng.integers(2, 9))
        logits = (rng.integers(-8, 9, size=(K + 1, V)) / 4.0).astype(np.float32)
        y = np.argmax(logits, axis=1)
        draft = np.where(rng.random(K + 1) < 0.5, y, rng.integers(0, V, K + 1)).astype(np.int32)
        out = oracle.verify(logits, draft, [K], [np.inf], [99], [[100.0, 1.5]])
        a = int(out["accept_len"][0])
        exact = sum(Fraction(float(logits[i, y[i]])) - Fraction(float(logits[i, draft[i]]))
                    for i in range(a) if draft[i] != y[i])
        assert Fraction(float(out["budget"][0, 1])) - Fraction(1.5) == exact


def test_monotone_in_controls_and_unbounded_accepts_all():
    rng = np.random.default_rng(3)
    for _ in range(200):
        K, V = int(rng.integers(1, 12)), int(rng.integers(2, 30))
        logits = rng.normal(0.0, 2.0, size=(K + 1, V)).astype(np.float32)
        y = np.argmax(logits, axis=1)
        draft = np.where(rng.random(K + 1) < 0.6, y, rng.integers(0, V, K + 1)).astype(np.int32)
        strict_a = strict_greedy(logits, draft, [K])[0][0]
        prev = -1
        for g in (0.0, 0.1, 0.5, 1.0, 4.0, np.inf):
            a = oracle.verify(logits, draft, [K], [g], [2], [[6.0, 0.0]])["accept_len"][0]
            assert a >= prev and a >= strict_a
            prev = a
        prev = -1
        for M in (0, 1, 2, 5, 100):
            a = oracle.verify(logits, draft, [K], [1.0], [M], [[6.0, 0.0]])["accept_len"][0]
            assert a >= prev
            prev = a
        prev = -1
        for B in (0.01, 0.5, 2.0, 8.0, np.inf):
            a = oracle.verify(logits, draft, [K], [1.0], [3], [[B, 0.0]])["accept_len"][0]
            assert a >= prev
            prev = a
        out = oracle.verify(logits, draft, [K], [np.inf], [2**31 - 1], [[np.inf, 0.0]])
        assert out["accept_len"][0] == K and out["next_token"][0] == y[K]


def test_out_of_range_draft_is_never_accepted():
    logits = np.zeros((3, 4), dtype=np.float32)
    logits[:, 1] = 1.0
    for bad in (-1, 4, 2**31 - 1):
        draft = np.array([1, bad, 0], dtype=np.int32)
        out = oracle.verify(logits, draft, [2], [np.inf], [2**31 - 1], [[np.inf, 0.0]])
        assert out["accept_len"][0] == 1 and out["next_token"][0] == 1
        assert out["regret"][1] == np.inf


def test_negative_block_length_reads_as_zero_and_bad_rows_are_not_verified():
    logits = np.zeros((5, 3), dtype=np.float32)
    logits[2, 1] = 1.0
    draft = np.zeros(5, dtype=np.int32)
    out = oracle.verify(logits, draft, [1, -1, 2], [1.0] * 3, [1] * 3,
                        [[1.0, 0.25]] * 3, row_offsets=[0, 2, 3])
    # K = -1 is K = 0: the request's one row at o = 2 is its bonus row
    assert list(out["accept_len"]) == [1, 0, 0]
    assert list(out["next_token"]) == [0, 1, -1]      # row 3 + 2 is past the end
    assert list(out["budget"][:, 1]) == [0.25, 0.25, 0.25]
    assert out["regret"][2] == 0.0 and not np.signbit(out["regret"][2])
    assert out["error"] == oracle.ERR_NEGATIVE_K | oracle.ERR_ROWS
    # the packed layout gives a negative K one row, like K = 0
    neg = oracle.verify(logits, draft, [1, -7, 1], [1.0] * 3, [1] * 3, [[1.0, 0.25]] * 3)
    zero = oracle.verify(logits, draft, [1, 0, 1], [1.0] * 3, [1] * 3, [[1.0, 0.25]] * 3)
    for k in ("accept_len", "next_token", "budget", "argmax"):
        assert np.array_equal(neg[k], zero[k])
    assert neg["error"] == oracle.ERR_NEGATIVE_K and zero["error"] == 0
    ok = oracle.verify(logits, draft, [1, 2], [1.0] * 2, [1] * 2, [[1.0, 0.0]] * 2)
    assert ok["error"] == 0


def test_ledger_carried_across_sessions():
    """Checkpoint/resume: the ledger is the only state; splitting 64 sequential
    blocks into two sessions with a host round-trip changes nothing."""
    w = W.make_config(1, batch=16, vocab=3000)
    def run(blocks, budget):
        res = []
        for b in blocks:
            lg, dr = w.call(b)
            out = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, budget)
            budget = out["budget"]
            res.append((int(out["accept_len"][0]), int(out["next_token"][0])))
        return res, budget
    full, b_full = run(range(16), w.budget)
    first, b_mid = run(range(8), w.budget)
    saved = json.loads(json.dumps(b_mid.tolist()))
    second, b_end = run(range(8, 16), np.array(saved, dtype=np.float32))
    assert full == first + second
    assert np.array_equal(b_full, b_end)
    assert b_full[0, 1] <= b_full[0, 0]


# ------------------------------------------------------------- argmax (Eq. 1)

def test_argmax_matches_numpy_on_finite_values_with_signed_zeros_and_infs():
    rng = np.random.default_rng(1)
    for _ in range(200):
        R, V = int(rng.integers(1, 6)), int(rng.integers(1, 70))
        pool = np.array([-np.inf, -1.5, -0.0, 0.0, 0.5, 2.0, np.inf], dtype=np.float32)
        x = rng.choice(pool, size=(R, V)).astype(np.float32)
        assert np.array_equal(oracle.argmax_rows(x), np.argmax(x, axis=1))
        xb = W.f32_to_bf16(np.nan_to_num(x, posinf=3e38, neginf=-3e38))
        assert np.array_equal(oracle.argmax_rows(xb), np.argmax(W.bf16_to_f32(xb), axis=1))


def test_argmax_with_nans_matches_numpy_first_nan():
    """numpy.argmax returns the first NaN of a row (NaN propagates through its
    maximum); the verifier's order ranks every NaN, of either sign and any
    payload, above +inf and all NaNs equal, so the two must agree everywhere."""
    rng = np.random.default_rng(4)
    specials = np.array([0x7FC00000, 0x7F800001, 0x7FFFFFFF, 0xFFC00000, 0xFF800001,
                         0xFFFFFFFF, 0x7F800000, 0xFF800000, 0x80000000, 0x00000000,
                         0x3F800000, 0xBF800000], dtype=np.uint32).view(np.float32)
    for _ in range(400):
        R, V = int(rng.integers(1, 4)), int(rng.integers(1, 40))
        x = rng.choice(specials, size=(R, V)).astype(np.float32)
        with np.errstate(invalid="ignore"):
            assert np.array_equal(oracle.argmax_rows(x), np.argmax(x, axis=1))
        xb = (x.view(np.uint32) >> 16).astype(np.uint16)      # exact: low halves are zero
        wide = (xb.astype(np.uint32) << 16).view(np.float32)
        assert np.array_equal(oracle.argmax_rows(xb), np.argmax(wide, axis=1))
    # every NaN pattern of bf16 ranks above +inf and below no other NaN
    nans = np.array([0x7F81, 0x7FC0, 0x7FFF, 0xFF81, 0xFFC0, 0xFFFF], dtype=np.uint16)
    for n in nans:
        row = np.array([[0x7F80, n, 0x3F80, n ^ 0x8000]], dtype=np.uint16)
        assert oracle.argmax_rows(row)[0] == 1


def test_regret_is_one_fp32_subtraction():
    rng = np.random.default_rng(8)
    logits = rng.normal(0, 3, size=(41, 257)).astype(np.float32)
    y = np.argmax(logits, axis=1)
    draft = rng.integers(0, 257, 41).astype(np.int32)
    lens = [40]
    out = oracle.verify(logits, draft, lens, [1.0], [1], [[1.0, 0.0]])
    rows = np.arange(40)
    expect = logits[rows, y[:40]] - logits[rows, draft[:40]]       # numpy float32 '-'
    assert np.array_equal(out["regret"][:40].view(np.uint32), expect.view(np.uint32))
    assert out["regret"][40] == 0.0 and not np.signbit(out["regret"][40])


def test_budget_reading_keeps_ledger_within_budget_where_the_other_form_fails():
    """Reading of Eq. 9: fl32(s + C) <= B keeps s' <= B exactly.  The other
    binary32 form C <= fl32(B - s) admits cases where s + C rounds above B."""
    rng = np.random.default_rng(12)
    found = 0
    for _ in range(200000):
        B = np.float32(rng.uniform(0.5, 8.0))
        s = np.float32(rng.uniform(0.0, 1.0) * B)
        C = np.float32(B - s) + np.float32(rng.integers(0, 3)) * np.spacing(np.float32(B - s))
        if C <= np.float32(B - s) and np.float32(s + C) > B:
            found += 1
            logits = np.array([[0.0, C], [0.0, 0.0]], dtype=np.float32)
            out = oracle.verify(logits, np.array([0, 0], np.int32), [1], [np.inf], [1], [[B, s]])
            assert out["accept_len"][0] == 0 and out["budget"][0, 1] == s
        if found >= 5:
            break
    assert found >= 1


def test_lmhead_logits_exact_regime_equals_integer_matmul():
    rng = np.random.default_rng(21)
    for d in (64, 512, 5120):
        h = rng.integers(-2, 3, size=(7, d))
        w = rng.integers(-2, 3, size=(33, d))
        z = oracle.lmhead_logits(W.f32_to_bf16(h.astype(np.float32)),
                                 W.f32_to_bf16(w.astype(np.float32)))
        assert z.dtype == np.float32
        assert np.array_equal(z, (h.astype(np.int64) @ w.T).astype(np.float32))
    # a zero sum is +0 even when every product is -0
    z = oracle.lmhead_logits(W.f32_to_bf16(np.zeros((1, 4), np.float32)),
                             W.f32_to_bf16(-np.ones((1, 4), np.float32)))
    assert z[0, 0] == 0.0 and not np.signbit(z[0, 0])


# ------------------------------------------------------- metamorphic checks

def _batch(rng, n, vocab):
    lens = rng.integers(0, 10, n).astype(np.int32)
    rows = int(np.sum(lens + 1))
    z = (rng.integers(-8, 9, size=(rows, vocab)) / 4.0).astype(np.float32)
    y = np.argmax(z, axis=1)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(0, vocab, rows)).astype(np.int32)
    tau = rng.choice(np.array([0.25, 1.0, 2.0, np.inf], np.float32), n)
    cap = rng.choice(np.array([0, 1, 3], np.int32), n)
    budget = np.stack([rng.choice(np.array([0.0, 1.0, 4.0], np.float32), n),
                       np.zeros(n, np.float32)], 1)
    return z, draft, lens, tau, cap, budget


def test_requests_are_independent_split_and_permuted():
    """Algorithm 1 runs per request: a batch verified at once equals its two
    halves verified apart, and a permutation of the requests (their rows moved
    with them through explicit offsets, with unused rows between) permutes the
    outputs."""
    rng = np.random.default_rng(61)
    for _ in range(60):
        n, vocab = int(rng.integers(2, 12)), int(rng.integers(1, 20))
        z, draft, lens, tau, cap, budget = _batch(rng, n, vocab)
        whole = oracle.verify(z, draft, lens, tau, cap, budget)
        k = int(rng.integers(1, n))
        cut = int(np.sum(lens[:k] + 1))
        a = oracle.verify(z[:cut], draft[:cut], lens[:k], tau[:k], cap[:k], budget[:k])
        b = oracle.verify(z[cut:], draft[cut:], lens[k:], tau[k:], cap[k:], budget[k:])
        for key in ("accept_len", "next_token", "budget"):
            assert np.array_equal(whole[key], np.concatenate([a[key], b[key]]))
        # permuted requests, rows laid out in the new order with gaps
        perm = rng.permutation(n)
        starts = np.concatenate([[0], np.cumsum(lens + 1)])[:-1]
        blocks, offs, pos = [], [], 0
        for i in perm:
            pos += int(rng.integers(0, 3))
            offs.append(pos)
            blocks.append((pos, starts[i], lens[i] + 1))
            pos += lens[i] + 1
        rows2 = pos + 1
        z2 = np.full((rows2, vocab), -9.0, np.float32)
        d2 = np.zeros(rows2, np.int32)
        for dst, src, cnt in blocks:
            z2[dst:dst + cnt] = z[src:src + cnt]
            d2[dst:dst + cnt] = draft[src:src + cnt]
        p = oracle.verify(z2, d2, lens[perm], tau[perm], cap[perm], budget[perm],
                          row_offsets=np.array(offs, np.int64))
        for key in ("accept_len", "next_token", "budget"):
            assert np.array_equal(p[key], whole[key][perm])
