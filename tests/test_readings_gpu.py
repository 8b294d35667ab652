"""GPU parity where the paper is silent: the argmax order of NaN logits, a
negative block length, the raw-gate variant, and the device error word.

Bar: bit-exact with the oracle (a regret that is NaN on both sides counts as
equal).  Row shapes are chosen so that the row kernel runs both as one tile per
row and split over many tiles, on rows whose base is not 16-byte aligned (odd
vocabularies), so a NaN can sit in the streamed middle of a tile, in the
unaligned head or tail of a row, or in a tile of its own.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W
from asd_gpu import describe, device_logits, gpu_verify, mismatches, oracle_verify

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

NAN_F32 = np.array([0x7FC00000, 0x7F800001, 0x7FFFFFFF, 0xFFC00000, 0xFF800001, 0xFFFFFFFF],
                   dtype=np.uint32)
NAN_BF16 = np.array([0x7FC0, 0x7F81, 0x7FFF, 0xFFC0, 0xFF81, 0xFFFF], dtype=np.uint16)


def check(logits, draft, lens, tau, cap, budget, row_offsets=None, label="", raw_gate=False):
    print("case %s: rows %d vocab %d dtype %s raw_gate %s" % (
        label, logits.shape[0], logits.shape[1], logits.dtype, raw_gate), flush=True)
    g = gpu_verify(logits, draft, lens, tau, cap, budget, row_offsets,
                   flags=asd.ASD_GATE_RAW if raw_gate else None)
    r = oracle_verify(logits, draft, lens, tau, cap, budget, row_offsets, raw_gate=raw_gate)
    bad = mismatches(g, r)
    assert not bad, "%s differs in %s: %s" % (label, bad, describe(g, r))
    return g, r


def _nan_logits(rng, rows, vocab, dtype, where):
    """Gaussian rows (all below zero for "negative") with NaNs planted per
    `where`; returns logits in the requested dtype (bf16 as bit patterns)."""
    z = rng.normal(0.0, 2.0, size=(rows, vocab)).astype(np.float32)
    if where == "negative":
        z = -np.abs(z) - np.float32(0.5)
    if dtype == "bf16":
        bits, nan_pool = W.f32_to_bf16(z), NAN_BF16
    else:
        bits, nan_pool = z.view(np.uint32).copy(), NAN_F32
    if where == "only_negative":
        nan_pool = nan_pool[3:]
    elif where == "only_positive":
        nan_pool = nan_pool[:3]
    for r in range(rows):
        n = int(rng.integers(0, 4)) if where != "inf_first" else 1
        if where == "edges":
            cols = rng.choice(np.r_[0:min(8, vocab), max(0, vocab - 8):vocab], size=n)
        else:
            cols = rng.integers(0, vocab, n)
        bits[r, cols] = rng.choice(nan_pool, n)
        if where == "inf_first":
            bits[r, 0] = 0x7F80 if dtype == "bf16" else 0x7F800000
    return bits if dtype == "bf16" else bits.view(np.float32)


# rows, vocab, block lengths: split over many tiles, split over a few, one
# tile per row (odd vocabulary: unaligned rows with heads and tails)
SHAPES = [(9, 151936, [8]), (40, 50001, [3] * 10), (600, 4099, [14] * 40)]


@pytest.mark.parametrize("where", ["random", "edges", "negative", "inf_first", "only_negative",
                                   "only_positive"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", range(len(SHAPES)))
def test_nan_logits_rank_above_everything_first_wins(shape, dtype, where):
    rows, vocab, lens = SHAPES[shape]
    rng = np.random.default_rng(1000 * shape + 10 * len(where) + (dtype == "f32"))
    logits = _nan_logits(rng, rows, vocab, dtype, where)
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(0, vocab, rows)).astype(np.int32)
    n = len(lens)
    g, r = check(logits, draft, np.array(lens, np.int32), 1.0, 2, [[4.0, 0.0]] * n,
                 label="nan-%s-%s-%d" % (where, dtype, shape))
    if where not in ("negative",):
        assert np.any(r["regret"] != r["regret"])     # some NaN regret was exercised


def test_nan_in_one_split_tile_of_an_otherwise_positive_row():
    """One NaN with the sign bit set, alone in a late tile of a split row whose
    other tiles hold large positive values: only the NaN detection of the raw
    pass can find it."""
    rng = np.random.default_rng(5)
    vocab = 151936
    for dtype in ("bf16", "f32"):
        z = rng.uniform(1.0, 2.0, size=(3, vocab)).astype(np.float32)
        z[:, 7] = 1e30
        logits = W.f32_to_bf16(z) if dtype == "bf16" else z
        if dtype == "bf16":
            logits[0, vocab - 3] = 0xFF81
            logits[1, 100000] = 0xFFFF
            logits[2, 123457] = 0x7FC1
        else:
            b = logits.view(np.uint32)
            b[0, vocab - 3] = 0xFF800001
            b[1, 100000] = 0xFFFFFFFF
            b[2, 123457] = 0x7FC00001
        draft = np.array([7, 7, 5], dtype=np.int32)
        g, _ = check(logits, draft, np.array([2], np.int32), 1.0, 1, [[1.0, 0.0]],
                     label="late-nan-" + dtype)
        assert g["argmax"].tolist() == [vocab - 3, 100000, 123457]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_log_probability_rows(dtype):
    """Rows of log-probabilities (all <= 0): every tile is ranked with exact
    sign-magnitude keys."""
    rng = np.random.default_rng(11 if dtype == "bf16" else 12)
    rows, vocab = 68, 32000
    z = rng.normal(0, 3, size=(rows, vocab))
    lp = (z - np.log(np.exp(z - z.max(1, keepdims=True)).sum(1, keepdims=True))
          - z.max(1, keepdims=True)).astype(np.float32)
    lp[:, 3] = 0.0                       # a zero log-probability in some rows
    lp[::2, 3] = -1.0
    logits = W.f32_to_bf16(lp) if dtype == "bf16" else lp
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
    check(logits, draft, np.array([16] * 4, np.int32), 0.5, 2, [[3.0, 0.0]] * 4,
          label="logprob-" + dtype)


# ------------------------------------------------------- negative K, errors

def _error_word(clear=False):
    torch.cuda.synchronize()
    return asd.asd_device_error(clear=clear)


def test_negative_block_lengths_read_as_zero_and_set_the_error_word():
    rng = np.random.default_rng(21)
    vocab = 5000
    lens = np.array([4, -1, 0, -7, 3, -1], dtype=np.int32)
    rows = int(np.sum(np.maximum(lens, 0) + 1))
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    logits = W.f32_to_bf16(z)
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
    budget = [[2.0, 0.25]] * len(lens)
    _error_word(clear=True)
    assert _error_word() == 0
    g, r = check(logits, draft, lens, 1.0, 2, budget, label="negative-k")
    assert r["error"] == oracle.ERR_NEGATIVE_K
    assert _error_word(clear=True) == asd.ASD_DEVERR_NEGATIVE_K
    assert _error_word() == 0                            # cleared
    assert np.all(g["next_token"] >= 0)                  # every request verified
    # rows outside the batch as well, with explicit offsets
    offs = np.array([0, 5, 6, 7, rows - 2, -1], dtype=np.int64)
    g, r = check(logits, draft, lens, 1.0, 2, budget, row_offsets=offs, label="negative-k-offs")
    assert r["error"] == oracle.ERR_NEGATIVE_K | oracle.ERR_ROWS
    assert _error_word(clear=True) == asd.ASD_DEVERR_NEGATIVE_K | asd.ASD_DEVERR_ROWS
    # a clean call leaves the word at zero
    clean = np.array([4, 0, 2], dtype=np.int32)
    rows_c = int(np.sum(clean + 1))
    check(logits[:rows_c], draft[:rows_c], clean, 1.0, 2, [[2.0, 0.0]] * 3, label="clean")
    assert _error_word() == 0


def test_commit_sets_the_error_word_for_what_does_not_fit():
    rng = np.random.default_rng(22)
    w = W.make_config(2, batch=12)
    n = w.num_requests
    cap = 40
    start = rng.integers(0, 10, n).astype(np.int64)
    budget = torch.from_numpy(w.budget.copy()).to(DEV)
    tl = device_logits(w.logits, DEV)
    td = torch.from_numpy(w.draft_tokens).to(DEV)
    tk = torch.from_numpy(w.block_lens).to(DEV)
    tt = torch.from_numpy(w.tau).to(DEV)
    tc = torch.from_numpy(w.exc_cap).to(DEV)
    _error_word(clear=True)
    acc, nxt = asd.asd_verify(tl, td, tk, tt, tc, budget)
    tok = torch.zeros((n, cap), dtype=torch.int32, device=DEV)
    sl = torch.from_numpy(start.copy()).to(DEV)
    asd.asd_commit(td, tk, acc, nxt, tok, sl)
    assert _error_word() == 0                            # everything fit
    sl = torch.from_numpy(np.full(n, cap - 2, np.int64)).to(DEV)
    asd.asd_commit(td, tk, acc, nxt, tok, sl)          # a + 1 tokens fit only if a <= 1
    ref = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    expect = asd.ASD_DEVERR_COMMIT if np.any(ref["accept_len"] > 1) else 0
    assert _error_word(clear=True) == expect
    # the fused verify-and-commit path reports the same
    budget = torch.from_numpy(w.budget.copy()).to(DEV)
    sl = torch.from_numpy(np.array([-1] + [0] * (n - 1), np.int64)).to(DEV)
    asd.asd_verify_commit(tl, td, tk, tt, tc, budget, tok, sl)
    assert _error_word(clear=True) == asd.ASD_DEVERR_COMMIT


# ------------------------------------------------------------ raw gate

@pytest.mark.parametrize("cfg,batch", [(1, 1), (2, 16), (3, 32), (5, 64)])
def test_raw_gate_variant_matches_oracle(cfg, batch):
    w = W.make_config(cfg, batch=batch)
    lg, dr = (w.call(0) if cfg == 1 else (w.logits, w.draft_tokens))
    g, r = check(lg, dr, w.block_lens, w.tau, w.exc_cap, w.budget, w.row_offsets,
                 label="raw-gate-%d" % cfg, raw_gate=True)
    norm = oracle.verify(lg, dr, w.block_lens, w.tau, w.exc_cap, w.budget, w.row_offsets)
    assert np.all(r["accept_len"] <= norm["accept_len"])


def test_raw_gate_on_dyadic_blocks_differs_where_the_brute_force_says():
    rng = np.random.default_rng(23)
    n, K, vocab = 300, 8, 64
    rows = n * (K + 1)
    logits = (rng.integers(-8, 9, size=(rows, vocab)) / 4.0).astype(np.float32)
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.5, y, rng.integers(0, vocab, rows)).astype(np.int32)
    lens = np.full(n, K, np.int32)
    tau = rng.choice(np.array([0.25, 0.5, 1.0, 1.5], np.float32), n)
    budget = np.stack([np.full(n, 3.75, np.float32), np.zeros(n, np.float32)], 1)
    g_raw, r_raw = check(logits, draft, lens, tau, 3, budget, label="dyadic-raw", raw_gate=True)
    g_norm, r_norm = check(logits, draft, lens, tau, 3, budget, label="dyadic-norm")
    assert np.sum(r_raw["accept_len"] != r_norm["accept_len"]) > 10


def test_verify_ex_without_flags_equals_verify_and_takes_a_workspace():
    w = W.make_config(3, batch=24)
    base = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    ex = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget, flags=0)
    nbytes = asd.asd_workspace_bytes(torch.bfloat16, w.logits.shape[1], w.num_requests,
                                     w.logits.shape[0])
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    exw = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget,
                     flags=0, workspace=ws)
    for k in ("accept_len", "next_token", "argmax", "budget"):
        assert np.array_equal(base[k], ex[k]) and np.array_equal(base[k], exw[k]), k
    assert np.array_equal(base["regret"].view(np.uint32), ex["regret"].view(np.uint32))
    with pytest.raises(asd.AsdError):
        gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget, flags=6)
