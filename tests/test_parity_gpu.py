"""Parity of the HIP verifier with the CPU oracle, through the C ABI.

Bar: bit-exact.  accept lengths, next tokens and per-row argmax are compared
as integers; regrets and the ledger as binary32 bit patterns (a regret that is
NaN on both sides counts as equal: the payload of a NaN produced by an
arithmetic operation is not part of the contract).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from asd_gpu import describe, gpu_verify, mismatches, oracle_verify

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def check(logits, draft, lens, tau, cap, budget, row_offsets=None, label=""):
    print("case %s: rows %d vocab %d dtype %s" % (label, logits.shape[0], logits.shape[1],
                                                   logits.dtype), flush=True)
    g = gpu_verify(logits, draft, lens, tau, cap, budget, row_offsets)
    r = oracle_verify(logits, draft, lens, tau, cap, budget, row_offsets)
    bad = mismatches(g, r)
    assert not bad, "%s differs in %s: %s" % (label, bad, describe(g, r))
    return g


def check_workload(w, label):
    return check(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget,
                 w.row_offsets, label)


# ------------------------------------------------------------ paper example

@pytest.mark.parametrize("mode", ["asd", "strict"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_figure1_example(mode, dtype):
    with open(os.path.join(GOLDEN, "fig1_asd_example.json")) as f:
        fx = json.load(f)
    logits = np.array(fx["logits"], dtype=np.float32)
    if dtype == "bf16":
        logits = W.f32_to_bf16(logits)
    p = fx[mode]
    g = check(logits, np.array(fx["draft_tokens"], np.int32), [fx["block_len"]], [p["tau"]],
              [p["exc_cap"]], [[p["budget_total"], p["budget_spent"]]], label="fig1")
    exp = p["expected"]
    assert g["accept_len"][0] == exp["accept_len"]
    assert g["next_token"][0] == exp["next_token"]
    assert g["budget"][0, 1] == np.float32(exp["budget_spent"])


# ------------------------------------------------- the five workloads, full size

@pytest.mark.parametrize("cfg,variant", [(2, "asd"), (3, "asd"), (4, "asd"), (4, "asd_b8"),
                                         (4, "strict"), (5, "asd")])
def test_workload_full_size(cfg, variant):
    w = W.make_config(cfg, variant=variant)
    g = check_workload(w, w.name)
    if variant == "strict":
        # B = 0 must equal exact greedy verification: stop at the first
        # token-ID mismatch, ledger unchanged.
        z = w.logits
        y = np.argmax(z, axis=1)
        for i in range(w.num_requests):
            o = i * 33
            a = 0
            while a < 32 and w.draft_tokens[o + a] == y[o + a]:
                a += 1
            assert g["accept_len"][i] == a and g["next_token"][i] == y[o + a]
        assert np.array_equal(g["budget"], w.budget)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workload_seeds_0_to_9(cfg):
    """Every workload at seeds 0..9, reduced in batch (full vocabulary), bit-exact."""
    for seed in range(10):
        w = W.make_config(cfg, seed=seed, batch={1: 3, 2: 6, 3: 6, 4: 4, 5: 24}[cfg])
        if w.blocks > 1:
            lg, dr = w.call(seed % w.blocks)
            check(lg, dr, w.block_lens, w.tau, w.exc_cap, w.budget, label="%s seed %d" % (
                w.name, seed))
        else:
            check_workload(w, "%s seed %d" % (w.name, seed))


def test_workload1_sequential_blocks_carry_the_ledger_on_device():
    """64 sequential calls of one request; the ledger stays in device memory."""
    w = W.make_config(1)
    dev = torch.device("cuda:0")
    import paper_2608_03447_amd as asd
    budget = torch.from_numpy(w.budget.copy()).to(dev)
    lens = torch.from_numpy(w.block_lens).to(dev)
    tau = torch.from_numpy(w.tau).to(dev)
    cap = torch.from_numpy(w.exc_cap).to(dev)
    logits_all = torch.from_numpy(w.logits).to(dev)
    draft_all = torch.from_numpy(w.draft_tokens).to(dev)
    n = w.rows_per_call
    outs = []
    for b in range(w.blocks):
        acc, nxt = asd.asd_verify(logits_all[b * n:(b + 1) * n], draft_all[b * n:(b + 1) * n],
                                  lens, tau, cap, budget)
        outs.append((acc, nxt))
    torch.cuda.synchronize()
    ref_budget = w.budget.copy()
    for b in range(w.blocks):
        lg, dr = w.call(b)
        ref = oracle_verify(lg, dr, w.block_lens, w.tau, w.exc_cap, ref_budget)
        ref_budget = ref["budget"]
        assert outs[b][0].item() == ref["accept_len"][0], b
        assert outs[b][1].item() == ref["next_token"][0], b
    assert np.array_equal(budget.cpu().numpy().view(np.uint32), ref_budget.view(np.uint32))
    assert ref_budget[0, 1] > 0          # exceptions were accepted and carried


# ------------------------------------------------ shapes: tiles and ragged tails

VOCABS = [1, 2, 3, 7, 8, 9, 15, 16, 17, 255, 256, 257, 1000, 2048, 4095, 32003, 50257, 151936]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("vocab", VOCABS)
def test_vocab_sizes_and_row_alignment(dtype, vocab):
    rng = np.random.default_rng(vocab)
    B = 5
    lens = rng.integers(0, 6, B).astype(np.int32)
    rows = int(np.sum(lens + 1))
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    peak = rng.integers(0, vocab, rows)
    z[np.arange(rows), peak] += 3.0
    logits = W.f32_to_bf16(z) if dtype == "bf16" else z
    zf = W.bf16_to_f32(logits) if dtype == "bf16" else logits
    y = np.argmax(zf, axis=1)
    second = np.argsort(-zf, axis=1, kind="stable")[:, min(1, vocab - 1)]
    draft = np.where(rng.random(rows) < 0.6, y, second).astype(np.int32)
    tau = rng.uniform(0.5, 3.0, B).astype(np.float32)
    budget = np.stack([rng.uniform(0, 8, B), np.zeros(B)], axis=1).astype(np.float32)
    check(logits, draft, lens, tau, 2, budget, label="vocab%d-%s" % (vocab, dtype))


@pytest.mark.parametrize("rows", [1, 2, 3, 9, 31, 257, 600, 2500])
def test_row_counts_select_split_plans(rows):
    # Few rows split each row over several workgroups, many rows do not.
    rng = np.random.default_rng(rows)
    vocab = 65536 + 24
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    logits = W.f32_to_bf16(z)
    lens = np.array([rows - 1], dtype=np.int32)
    draft = rng.integers(0, vocab, rows).astype(np.int32)
    check(logits, draft, lens, 1.0, 1, [[4.0, 0.0]], label="rows%d" % rows)


def test_argmax_in_every_position_of_a_row():
    # Put the single greatest value at every column class: head, vector lanes,
    # each element of a vector, split boundaries, and the tail.
    vocab = 70001
    cols = list(range(0, 40)) + list(range(vocab - 40, vocab)) + \
        [4096 * k + d for k in range(1, 17) for d in (-1, 0, 1, 7, 8)]
    cols = sorted(set(c for c in cols if 0 <= c < vocab))
    rows = len(cols)
    for dtype in ("bf16", "f32"):
        z = np.full((rows, vocab), -1.0, dtype=np.float32)
        z[np.arange(rows), cols] = 5.0
        logits = W.f32_to_bf16(z) if dtype == "bf16" else z
        draft = np.array(cols, dtype=np.int32)
        g = check(logits, draft, [rows - 1], 1.0, 1, [[1.0, 0.0]], label="positions-" + dtype)
        assert np.array_equal(g["argmax"], np.array(cols))


# ------------------------------------------------------- special values, ties

SPECIAL_BITS = np.array([0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x007fffff,
                         0x3f800000, 0xbf800000, 0x7f800000, 0xff800000, 0x7fc00000,
                         0xffc00000, 0x7f800001, 0x7fbfffff, 0xff800001, 0x40000000,
                         0x40400000, 0x3e800000], dtype=np.uint32)


@pytest.mark.parametrize("seed", range(6))
def test_special_values_and_ties(seed):
    rng = np.random.default_rng(100 + seed)
    for dtype in ("f32", "bf16"):
        B = int(rng.integers(1, 12))
        lens = rng.integers(0, 9, B).astype(np.int32)
        rows = int(np.sum(lens + 1))
        vocab = int(rng.choice([5, 64, 300, 1031, 4096, 20000]))
        dyadic = (rng.integers(-6, 7, size=(rows, vocab)) / 4.0).astype(np.float32)
        special = SPECIAL_BITS[rng.integers(0, len(SPECIAL_BITS), size=(rows, vocab))].view(
            np.float32)
        use_special = rng.random((rows, vocab)) < (0.3 if seed % 2 else 0.02)
        z = np.where(use_special, special, dyadic).astype(np.float32)
        logits = (z.view(np.uint32) >> 16).astype(np.uint16) if dtype == "bf16" else z
        draft = rng.integers(-2, vocab + 2, rows).astype(np.int32)
        zf = W.bf16_to_f32(logits) if dtype == "bf16" else logits
        y = np.argmax(np.nan_to_num(zf, nan=-np.inf), axis=1)
        draft = np.where(rng.random(rows) < 0.5, y, draft).astype(np.int32)
        tau = rng.choice(np.array([-1.0, 0.0, 0.25, 1.0, np.inf, np.nan], np.float32), B)
        cap = rng.choice(np.array([0, 1, 3, 2**31 - 1], np.int32), B)
        tot = rng.choice(np.array([0.0, -0.0, 0.5, 2.0, np.inf, 1e-30], np.float32), B)
        spent = np.minimum(rng.choice(np.array([0.0, -0.0, 0.25], np.float32), B), tot)
        budget = np.stack([tot, spent], axis=1).astype(np.float32)
        check(logits, draft, lens, tau, cap, budget, label="special%d-%s" % (seed, dtype))


# ---------------------------------------------- layouts and invalid requests

def test_explicit_row_offsets_with_gaps_and_invalid_requests():
    rng = np.random.default_rng(77)
    vocab, rows = 3000, 120
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    logits = W.f32_to_bf16(z)
    y = np.argmax(W.bf16_to_f32(logits), axis=1)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
    lens = np.array([8, 0, 5, -1, 8, 3, 12, 8], dtype=np.int32)
    offs = np.array([0, 10, 12, 20, 30, 117, 100, -4], dtype=np.int64)
    budget = np.tile(np.array([[3.0, 0.5]], np.float32), (8, 1))
    g = check(logits, draft, lens, 2.0, 1, budget, row_offsets=offs, label="offsets")
    assert list(g["next_token"][[5, 7]]) == [-1, -1]          # rows outside the batch
    assert g["next_token"][3] == y[20] and g["accept_len"][3] == 0   # K = -1 read as 0


def test_zero_length_blocks_emit_the_bonus_token():
    rng = np.random.default_rng(3)
    vocab = 2000
    lens = np.zeros(40, dtype=np.int32)
    z = rng.normal(0, 1, size=(40, vocab)).astype(np.float32)
    g = check(z, rng.integers(0, vocab, 40).astype(np.int32), lens, 1.0, 1, [[1.0, 0.0]] * 40,
              label="k0")
    assert np.array_equal(g["next_token"], np.argmax(z, axis=1))
    assert np.all(g["accept_len"] == 0)


def test_long_blocks_cross_scan_windows():
    rng = np.random.default_rng(9)
    vocab = 1024
    lens = np.array([31, 32, 33, 64, 100, 0, 1], dtype=np.int32)
    rows = int(np.sum(lens + 1))
    z = rng.normal(0, 1, size=(rows, vocab)).astype(np.float32)
    y = np.argmax(z, axis=1)
    second = np.argsort(-z, axis=1, kind="stable")[:, 1]
    draft = np.where(rng.random(rows) < 0.9, y, second).astype(np.int32)
    check(z, draft, lens, np.inf, 2**31 - 1, [[np.inf, 0.0]] * 7, label="long-inf")
    check(z, draft, lens, 0.5, 3, [[6.0, 1.0]] * 7, label="long")


# ------------------------------------------------- determinism, workspace, streams

@pytest.mark.parametrize("cfg,batch", [(2, 8), (5, 40)])
def test_repeated_calls_are_bit_identical(cfg, batch):
    """1,000 calls on the same inputs (a split plan and a ragged batch): every
    output equals the first call's bit for bit, compared on the device."""
    import paper_2608_03447_amd as asd
    from asd_gpu import device_logits
    w = W.make_config(cfg, batch=batch)
    first = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    assert not mismatches(first, oracle_verify(w.logits, w.draft_tokens, w.block_lens, w.tau,
                                               w.exc_cap, w.budget))
    dev = torch.device("cuda:0")
    tl = device_logits(w.logits, dev)
    td, tk = torch.from_numpy(w.draft_tokens).to(dev), torch.from_numpy(w.block_lens).to(dev)
    tt, tc = torch.from_numpy(w.tau).to(dev), torch.from_numpy(w.exc_cap).to(dev)
    pristine = torch.from_numpy(w.budget.copy()).to(dev)
    ref = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in first.items()}
    rows = w.rows_per_call
    amax = torch.empty(rows, dtype=torch.int32, device=dev)
    regret = torch.empty(rows, dtype=torch.float32, device=dev)
    tb = pristine.clone()
    for call in range(1000):
        tb.copy_(pristine)
        amax.fill_(-7)
        regret.fill_(float("nan"))
        acc, nxt = asd.asd_verify(tl, td, tk, tt, tc, tb, out_argmax=amax, out_regret=regret)
        assert (torch.equal(acc, ref["accept_len"]) and torch.equal(nxt, ref["next_token"])
                and torch.equal(amax, ref["argmax"])
                and torch.equal(tb.view(torch.int32), ref["budget"].view(torch.int32))
                and torch.equal(regret.view(torch.int32), ref["regret"].view(torch.int32))), call


def test_caller_workspace_matches_library_workspace():
    import paper_2608_03447_amd as asd
    w = W.make_config(2, batch=4)
    nbytes = asd.asd_workspace_bytes(torch.bfloat16, w.vocab, w.num_requests,
                                     w.logits.shape[0])
    assert nbytes > 0
    # Any content will do: nothing in the workspace is carried between calls.
    ws = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda:0")
    a = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget,
                   workspace=ws)
    b = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget,
                   workspace=ws)
    r = oracle_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    assert not mismatches(a, r) and not mismatches(b, r)
    small = torch.zeros(nbytes - 256, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(asd.AsdError):
        gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget,
                   workspace=small)


def test_two_streams_in_flight():
    import paper_2608_03447_amd as asd
    dev = torch.device("cuda:0")
    ws_ = [W.make_config(2, seed=s, batch=16) for s in (21, 22)]
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    res = []
    tensors = []
    for w in ws_:
        tensors.append(dict(
            logits=torch.from_numpy(w.logits.view(np.int16)).to(dev).view(torch.bfloat16),
            draft=torch.from_numpy(w.draft_tokens).to(dev),
            lens=torch.from_numpy(w.block_lens).to(dev),
            tau=torch.from_numpy(w.tau).to(dev), cap=torch.from_numpy(w.exc_cap).to(dev),
            budget=torch.from_numpy(w.budget.copy()).to(dev)))
    torch.cuda.synchronize()
    for _ in range(5):
        for k, (t, s) in enumerate(zip(tensors, streams)):
            with torch.cuda.stream(s):
                t["budget"].copy_(torch.from_numpy(ws_[k].budget).to(dev))
                res.append(asd.asd_verify(t["logits"], t["draft"], t["lens"], t["tau"],
                                          t["cap"], t["budget"]))
    torch.cuda.synchronize()
    for k, w in enumerate(ws_):
        r = oracle_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
        for j in range(5):
            acc, nxt = res[2 * j + k]
            assert np.array_equal(acc.cpu().numpy(), r["accept_len"])
            assert np.array_equal(nxt.cpu().numpy(), r["next_token"])


def test_alternating_shapes_share_one_workspace():
    """Calls of different shapes on one stream share the library workspace: a
    many-row call (one workgroup per row) must not disturb the split counters
    of a later few-row call (several workgroups per row), and back."""
    rng = np.random.default_rng(31)
    shapes = [(2700, 4000, "bf16"), (9, 32000, "f32"), (544, 20000, "bf16"),
              (3, 151936, "bf16"), (2000, 3000, "f32"), (9, 32000, "f32"), (17, 70000, "bf16")]
    for rows, vocab, dtype in shapes:
        z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
        logits = W.f32_to_bf16(z) if dtype == "bf16" else z
        zf = W.bf16_to_f32(logits) if dtype == "bf16" else logits
        y = np.argmax(zf, axis=1)
        draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
        check(logits, draft, [rows - 1], 2.0, 2, [[5.0, 0.0]],
              label="alternate-%d-%d-%s" % (rows, vocab, dtype))


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_without_optional_per_row_outputs(cfg):
    """The serving path: no out_argmax / out_regret (split and unsplit plans)."""
    import paper_2608_03447_amd as asd
    w = W.make_config(cfg, batch=None if cfg != 3 else 40)
    lg, dr = w.call(0)
    dev = torch.device("cuda:0")
    from asd_gpu import device_logits
    budget = torch.from_numpy(w.budget.copy()).to(dev)
    acc, nxt = asd.asd_verify(device_logits(lg, dev), torch.from_numpy(dr).to(dev),
                              torch.from_numpy(w.block_lens).to(dev),
                              torch.from_numpy(w.tau).to(dev),
                              torch.from_numpy(w.exc_cap).to(dev), budget)
    torch.cuda.synchronize()
    r = oracle_verify(lg, dr, w.block_lens, w.tau, w.exc_cap, w.budget)
    assert np.array_equal(acc.cpu().numpy(), r["accept_len"])
    assert np.array_equal(nxt.cpu().numpy(), r["next_token"])
    assert np.array_equal(budget.cpu().numpy().view(np.uint32), r["budget"].view(np.uint32))


# ------------------------------------------ vocabulary-sharded verification

def sharded_verify(logits, draft, lens, tau, cap, budget, num_shards, row_offsets=None):
    """Split every row into num_shards column shards (equal widths, the last
    narrower), reduce each shard separately, then finish from the partials."""
    import paper_2608_03447_amd as asd
    from asd_gpu import device_logits
    dev = torch.device("cuda:0")
    rows, vocab = logits.shape
    width = -(-vocab // num_shards)
    n = len(lens)
    td = torch.from_numpy(np.ascontiguousarray(draft, dtype=np.int32)).to(dev)
    parts = torch.empty((num_shards, rows, 4), dtype=torch.int32, device=dev)
    full = device_logits(logits, dev)
    for k in range(num_shards):
        shard = full[:, k * width:min((k + 1) * width, vocab)].contiguous()
        asd.asd_shard_argmax(shard, k * width, vocab, td, out_partials=parts[k])
    tb = torch.from_numpy(np.array(budget, dtype=np.float32).reshape(n, 2)).to(dev)
    amax = torch.full((rows,), -7, dtype=torch.int32, device=dev)
    regret = torch.full((rows,), float("nan"), dtype=torch.float32, device=dev)
    to = None if row_offsets is None else torch.from_numpy(
        np.ascontiguousarray(row_offsets, dtype=np.int64)).to(dev)
    acc, nxt = asd.asd_verify_partials(
        parts, width, vocab, td, torch.from_numpy(np.asarray(lens, dtype=np.int32)).to(dev),
        torch.from_numpy(np.ascontiguousarray(np.broadcast_to(np.asarray(tau, np.float32), (n,)))).to(dev),
        torch.from_numpy(np.ascontiguousarray(np.broadcast_to(np.asarray(cap, np.int32), (n,)))).to(dev),
        tb, row_offsets=to, out_argmax=amax, out_regret=regret)
    torch.cuda.synchronize()
    return {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
            "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
            "budget": tb.cpu().numpy()}


@pytest.mark.parametrize("cfg,shards", [(3, 8), (3, 3), (4, 8), (5, 8), (5, 1), (2, 2)])
def test_vocabulary_sharded_equals_unsharded(cfg, shards):
    w = W.make_config(cfg, batch=None if cfg != 3 else 64)
    print("case sharded workload %d x %d shards" % (cfg, shards), flush=True)
    g = sharded_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget, shards)
    r = oracle_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    bad = mismatches(g, r)
    assert not bad, "%s differs in %s: %s" % (w.name, bad, describe(g, r))


@pytest.mark.parametrize("vocab,shards", [(1000, 7), (50257, 8), (17, 4), (9, 9), (300, 2)])
def test_sharded_special_values_ragged_widths_and_offsets(vocab, shards):
    rng = np.random.default_rng(vocab + shards)
    for dtype in ("bf16", "f32"):
        lens = rng.integers(0, 7, 6).astype(np.int32)
        rows = int(np.sum(lens + 1)) + 3
        offs = np.concatenate([[0], np.cumsum(lens + 1)[:-1]]).astype(np.int64) + 2
        dyadic = (rng.integers(-6, 7, size=(rows, vocab)) / 4.0).astype(np.float32)
        special = SPECIAL_BITS[rng.integers(0, len(SPECIAL_BITS), size=(rows, vocab))].view(np.float32)
        z = np.where(rng.random((rows, vocab)) < 0.1, special, dyadic).astype(np.float32)
        logits = (z.view(np.uint32) >> 16).astype(np.uint16) if dtype == "bf16" else z
        zf = W.bf16_to_f32(logits) if dtype == "bf16" else logits
        y = np.argmax(np.nan_to_num(zf, nan=-np.inf), axis=1)
        draft = np.where(rng.random(rows) < 0.6, y, rng.integers(-1, vocab + 1, rows)).astype(np.int32)
        budget = np.stack([rng.choice([0.0, 1.0, 4.0], 6), np.zeros(6)], axis=1).astype(np.float32)
        g = sharded_verify(logits, draft, lens, 1.0, 2, budget, shards, row_offsets=offs)
        r = oracle_verify(logits, draft, lens, 1.0, 2, budget, row_offsets=offs)
        bad = mismatches(g, r)
        assert not bad, "vocab %d shards %d %s differs in %s: %s" % (vocab, shards, dtype, bad,
                                                                     describe(g, r))


@pytest.mark.parametrize("num_requests", [1023, 1024, 1025, 3000])
def test_sharded_packed_offsets_both_paths(num_requests):
    """Up to 1,024 requests each scan wavefront sums its own packed offset;
    above that a one-workgroup scan writes them first."""
    rng = np.random.default_rng(num_requests)
    vocab = 640
    lens = rng.integers(0, 5, num_requests).astype(np.int32)
    rows = int(np.sum(lens + 1))
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    logits = W.f32_to_bf16(z)
    y = np.argmax(W.bf16_to_f32(logits), axis=1)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(0, vocab, rows)).astype(np.int32)
    budget = np.stack([rng.uniform(0, 6, num_requests), np.zeros(num_requests)], axis=1).astype(np.float32)
    g = sharded_verify(logits, draft, lens, 2.0, 1, budget, 3)
    r = oracle_verify(logits, draft, lens, 2.0, 1, budget)
    bad = mismatches(g, r)
    assert not bad, "%d requests differ in %s: %s" % (num_requests, bad, describe(g, r))


# ------------------------------------------------ per-wavefront key choice

def _mixed_sign_blocks(rng, rows, vocab, block, dtype):
    """Rows built from `block`-element runs that are either all negative or
    mixed-sign, so that within one tile some wavefronts meet a positive number
    in their first group and others do not; a few rows hold only negatives and
    signed zeros (the maximum is then +-0 and the first zero wins)."""
    z = -rng.uniform(0.25, 6.0, size=(rows, vocab)).astype(np.float32)
    for r in range(rows):
        kind = rng.integers(0, 4)
        if kind == 0:                               # zeros only, both signs
            cols = rng.integers(0, vocab, int(rng.integers(1, 6)))
            z[r, cols] = rng.choice(np.array([0.0, -0.0], np.float32), cols.size)
        elif kind == 1:                             # one negative maximum, tied twice
            a, b = rng.integers(0, vocab, 2)
            z[r, a] = z[r, b] = np.float32(-0.125)
        else:                                       # positive runs here and there
            for start in range(0, vocab, block):
                if rng.random() < 0.15:
                    n = min(block, vocab - start)
                    z[r, start:start + n] = rng.normal(0, 2, n).astype(np.float32)
            if kind == 3:                           # the maximum late in the row
                z[r, int(rng.integers(vocab // 2, vocab))] = np.float32(30.0)
    return W.f32_to_bf16(z) if dtype == "bf16" else z


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rows,vocab", [(300, 32768), (9, 151936), (40, 50001)])
def test_wavefronts_choose_raw_or_sign_magnitude_keys(dtype, rows, vocab):
    rng = np.random.default_rng(rows + vocab + (dtype == "f32"))
    block = 512 if dtype == "bf16" else 256        # 64 lanes x one 16-byte vector
    logits = _mixed_sign_blocks(rng, rows, vocab, block, dtype)
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(0, vocab, rows)).astype(np.int32)
    K = 2 if rows % 3 == 0 else (rows // 3 if rows >= 3 else 0)
    lens = np.full(rows // (K + 1), K, np.int32)
    used = int(np.sum(lens + 1))
    check(logits[:used], draft[:used], lens, 1.0, 2, [[4.0, 0.0]] * len(lens),
          label="wave-modes-%s-%dx%d" % (dtype, rows, vocab))


# ------------------------------------------------------------- scale limits

def test_very_long_block():
    """K = 3,000: the scan walks 47 windows of 64 positions."""
    rng = np.random.default_rng(31)
    vocab = 512
    lens = np.array([3000, 5], dtype=np.int32)
    rows = int(np.sum(lens + 1))
    z = rng.normal(0, 1, size=(rows, vocab)).astype(np.float32)
    y = np.argmax(z, axis=1)
    second = np.argsort(-z, axis=1, kind="stable")[:, 1]
    draft = np.where(rng.random(rows) < 0.97, y, second).astype(np.int32)
    check(z, draft, lens, np.inf, 2**31 - 1, [[np.inf, 0.0]] * 2, label="k3000-inf")
    check(z, draft, lens, 0.01, 40, [[30.0, 0.0]] * 2, label="k3000")


def test_seventy_thousand_requests():
    """A large scan grid and the row kernel's one-workgroup offset scan over
    70,000 block lengths (K in 0..2, some negative)."""
    rng = np.random.default_rng(32)
    n, vocab = 70000, 64
    lens = rng.integers(-1, 3, n).astype(np.int32)
    rows = int(np.sum(np.maximum(lens, 0) + 1))
    table = W.f32_to_bf16(np.arange(-8, 9, dtype=np.float32) / 4)   # dyadic values, many ties
    logits = table[rng.integers(0, table.size, size=(rows, vocab), dtype=np.int8)]
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(0, vocab, rows)).astype(np.int32)
    tau = rng.uniform(0, 2, n).astype(np.float32)
    budget = np.stack([rng.uniform(0, 4, n), np.zeros(n)], 1).astype(np.float32)
    check(logits, draft, lens, tau, 2, budget, label="70k-requests")


def test_vocabulary_of_a_million_splits_at_the_cap():
    """V = 2^20 over 9 rows: the plan wants more than 64 splits and takes 64."""
    rng = np.random.default_rng(33)
    vocab, rows = 1 << 20, 9
    z = rng.normal(0, 2, size=(rows, vocab)).astype(np.float32)
    z[3, vocab - 1] = 50.0                       # the maximum in the last split
    z[5, 0] = 50.0                               # and in the first
    logits = W.f32_to_bf16(z)
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.5, y, rng.integers(0, vocab, rows)).astype(np.int32)
    check(logits, draft, np.array([8], np.int32), 2.0, 2, [[6.0, 0.0]], label="v2^20")
    check(z, draft, np.array([8], np.int32), 2.0, 2, [[6.0, 0.0]], label="v2^20-f32")


# ------------------------------------------------------- metamorphic checks

def test_requests_are_independent_split_and_permuted_on_the_gpu():
    """A ragged batch verified at once equals its halves verified apart, and a
    permutation of its requests (rows moved with them, unused rows between)
    permutes every output; all three agree with the oracle bit for bit."""
    rng = np.random.default_rng(71)
    w = W.make_config(5, batch=96, vocab=20000)
    n = w.num_requests
    lens = w.block_lens
    whole = check_workload(w, "independence-whole")
    k = 37
    cut = int(np.sum(lens[:k] + 1))
    a = check(w.logits[:cut], w.draft_tokens[:cut], lens[:k], w.tau[:k], w.exc_cap[:k],
              w.budget[:k], label="independence-first")
    b = check(w.logits[cut:], w.draft_tokens[cut:], lens[k:], w.tau[k:], w.exc_cap[k:],
              w.budget[k:], label="independence-second")
    for key in ("accept_len", "next_token", "budget"):
        assert np.array_equal(whole[key], np.concatenate([a[key], b[key]])), key
    perm = rng.permutation(n)
    starts = np.concatenate([[0], np.cumsum(lens + 1)])[:-1]
    offs, pos, moves = [], 0, []
    for i in perm:
        pos += int(rng.integers(0, 4))
        offs.append(pos)
        moves.append((pos, starts[i], lens[i] + 1))
        pos += lens[i] + 1
    rows2 = pos + 3
    z2 = np.zeros((rows2, w.vocab), np.uint16)
    d2 = np.zeros(rows2, np.int32)
    for dst, src, cnt in moves:
        z2[dst:dst + cnt] = w.logits[src:src + cnt]
        d2[dst:dst + cnt] = w.draft_tokens[src:src + cnt]
    p = check(z2, d2, lens[perm], w.tau[perm], w.exc_cap[perm], w.budget[perm],
              row_offsets=np.array(offs, np.int64), label="independence-permuted")
    for key in ("accept_len", "next_token", "budget"):
        assert np.array_equal(p[key], whole[key][perm]), key
