"""LM-head-fused verification (hidden states x output weights, argmax in the
epilogue) against the oracle.

Exact regime: small dyadic inputs whose products and every partial sum are
representable in binary32, so any accumulation order gives the exact logits
and every output must match bit for bit -- including ties for the maximum,
which such inputs produce often.  Realistic regime: random bf16 inputs, where
the matrix cores round in an order of their own; the argmax must agree wherever
the top-two gap exceeds the accumulated rounding bound, and the chosen token's
exact logit must lie within that bound of the exact maximum.
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def _run(hidden, weight, draft, lens, tau, cap, budget, offsets=None, outputs=True):
    import torch
    import paper_2608_03447_amd as asd
    from asd_gpu import device_logits
    dev = torch.device("cuda:0")
    rows = hidden.shape[0]
    n = len(lens)
    tb = torch.from_numpy(np.array(budget, dtype=np.float32).reshape(n, 2)).to(dev)
    amax = torch.full((rows,), -7, dtype=torch.int32, device=dev)
    regret = torch.full((rows,), float("nan"), dtype=torch.float32, device=dev)
    to = None if offsets is None else torch.from_numpy(np.asarray(offsets, np.int64)).to(dev)
    acc, nxt = asd.asd_lmhead_verify(
        device_logits(hidden, dev), device_logits(weight, dev),
        torch.from_numpy(np.ascontiguousarray(draft, dtype=np.int32)).to(dev),
        torch.from_numpy(np.asarray(lens, np.int32)).to(dev),
        torch.from_numpy(np.array(np.broadcast_to(np.asarray(tau, np.float32), (n,)))).to(dev),
        torch.from_numpy(np.array(np.broadcast_to(np.asarray(cap, np.int32), (n,)))).to(dev),
        tb, row_offsets=to, out_argmax=amax if outputs else None,
        out_regret=regret if outputs else None)
    torch.cuda.synchronize()
    return {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
            "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
            "budget": tb.cpu().numpy()}


def _exact_inputs(rng, rows, vocab, d):
    """Dyadic hidden states and weights whose every partial sum is exact in
    binary32, and drafts that are the greedy token, the runner-up or invalid."""
    hidden = W.f32_to_bf16(rng.integers(-2, 3, size=(rows, d)).astype(np.float32))
    weight = W.f32_to_bf16((rng.integers(-2, 3, size=(vocab, d)) / 2.0).astype(np.float32))
    z = oracle.lmhead_logits(hidden, weight)
    y = np.argmax(z, axis=1)
    second = np.argsort(-z, axis=1, kind="stable")[:, min(1, vocab - 1)]
    draft = np.where(rng.random(rows) < 0.6, y, second).astype(np.int32)
    draft[rng.random(rows) < 0.05] = -1
    draft[rng.random(rows) < 0.02] = vocab + 3
    return hidden, weight, draft


@pytest.mark.parametrize("rows,vocab,d", [(9, 100, 128), (130, 1027, 128), (300, 5000, 256),
                                          (17, 257, 5120), (1, 1, 128), (260, 3000, 384),
                                          (600, 1300, 640), (257, 513, 128)])
def test_exact_regime_bit_exact(rows, vocab, d):
    from asd_gpu import describe, mismatches
    rng = np.random.default_rng(rows * 7 + vocab + d)
    hidden = W.f32_to_bf16(rng.integers(-2, 3, size=(rows, d)).astype(np.float32))
    weight = W.f32_to_bf16((rng.integers(-2, 3, size=(vocab, d)) / 2.0).astype(np.float32))
    z = oracle.lmhead_logits(hidden, weight)
    y = np.argmax(z, axis=1)
    second = np.argsort(-z, axis=1, kind="stable")[:, min(1, vocab - 1)]
    draft = np.where(rng.random(rows) < 0.6, y, second).astype(np.int32)
    draft[rng.random(rows) < 0.05] = -1
    lens = []
    left = rows
    while left > 0:
        k = int(min(left - 1, rng.integers(0, 9)))
        lens.append(k)
        left -= k + 1
    budget = np.stack([rng.uniform(0, 6, len(lens)), np.zeros(len(lens))], axis=1)
    print("case lmhead exact rows %d vocab %d d %d" % (rows, vocab, d), flush=True)
    g = _run(hidden, weight, draft, lens, 1.0, 2, budget)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget)
    bad = mismatches(g, r)
    assert not bad, "differs in %s: %s" % (bad, describe(g, r))


@pytest.mark.parametrize("rows,vocab,d", [(130, 1027, 128), (40, 5000, 256), (300, 640, 128)])
def test_nonfinite_and_negative_rows_bit_exact(rows, vocab, d):
    """Rows that the epilogue cannot rank by raw patterns: every logit negative,
    NaNs among infinities, infinities only, NaN everywhere and all-zero rows,
    mixed with ordinary rows.  Coordinates 0-2 are reserved: weights 1 (a bias
    that makes a row negative when its hidden value is -256), weights in
    {-1, 0, 1} (inf there gives NaN where the weight is 0 and +-inf elsewhere),
    and weights +-0.5 (inf there gives +-inf only)."""
    from asd_gpu import describe, mismatches
    rng = np.random.default_rng(rows + vocab + d)
    h = rng.integers(-2, 3, size=(rows, d)).astype(np.float32)
    w = (rng.integers(-2, 3, size=(vocab, d)) / 2.0).astype(np.float32)
    h[:, :3] = 0.0
    w[:, 0] = 1.0
    w[:, 1] = rng.integers(-1, 2, size=vocab)
    w[:, 2] = rng.choice([-0.5, 0.5], size=vocab)
    kind = rng.integers(0, 7, size=rows)
    h[kind == 1, 0] = -256.0                      # every logit negative
    h[kind == 2, 1] = np.inf                      # NaN where w = 0, +-inf elsewhere
    h[kind == 3, 2] = np.inf                      # +-inf only
    h[kind == 4, 2] = -np.inf
    h[kind == 5, 3] = np.nan                      # NaN in every column
    h[kind == 6] = 0.0                            # every logit zero
    hidden, weight = W.f32_to_bf16(h), W.f32_to_bf16(w)
    z = oracle.lmhead_logits(hidden, weight)
    assert np.isnan(z[kind == 2]).any() and np.isinf(z[kind == 3]).all()
    assert (z[kind == 1] < 0).all()
    draft = rng.integers(0, vocab, rows).astype(np.int32)
    draft[rng.random(rows) < 0.05] = vocab + 1
    lens = []
    left = rows
    while left > 0:
        k = int(min(left - 1, rng.integers(0, 9)))
        lens.append(k)
        left -= k + 1
    budget = np.stack([rng.uniform(0, 6, len(lens)), np.zeros(len(lens))], axis=1)
    print("case lmhead nonfinite rows %d vocab %d d %d" % (rows, vocab, d), flush=True)
    g = _run(hidden, weight, draft, lens, 1.0, 2, budget)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget)
    bad = mismatches(g, r)
    assert not bad, "differs in %s: %s" % (bad, describe(g, r))


# The three launches the bench times: the headline batch at d = 5,120 and at
# d = 4,096, and workload 5's ragged rows at d = 7,168 with V = 129,280.
BENCH_SHAPES = [(3, 5120), (3, 4096), (5, 7168)]


@pytest.mark.parametrize("config,d", BENCH_SHAPES)
def test_full_size_every_output_bit_exact(config, d):
    """Every row and every request of a benched launch, exact regime.  Hidden
    states in {-2..2} and weights in {-1, -1/2, 0, 1/2, 1} are drawn on the
    device; the oracle forms all R x V logits exactly on the host (weights
    copied back in chunks), drafts are drawn from those logits (greedy token,
    runner-up or uniform), and the workload's own requests, gates, caps and
    budgets are verified.  Every per-row argmax and regret and every request's
    accepted length, next token and ledger must match bit for bit."""
    import torch
    import paper_2608_03447_amd as asd
    from asd_gpu import describe, mismatches
    dev = torch.device("cuda:0")
    w = W.make_config(config)
    rows, vocab = w.rows_per_call, w.vocab
    print("case lmhead full size: workload %d, %d rows x d %d x V %d" % (config, rows, d, vocab),
          flush=True)
    g = torch.Generator(device=dev).manual_seed(7700 + d)
    hidden = torch.randint(-2, 3, (rows, d), generator=g, device=dev).to(torch.bfloat16)
    weight = (torch.randint(-2, 3, (vocab, d), generator=g, device=dev).to(torch.float32) / 2.0
              ).to(torch.bfloat16)
    h_bits = hidden.view(torch.int16).cpu().numpy().view(np.uint16)
    z = np.empty((rows, vocab), np.float32)
    for c in range(0, vocab, 8192):
        z[:, c:c + 8192] = oracle.lmhead_logits(
            h_bits, weight[c:c + 8192].view(torch.int16).cpu().numpy().view(np.uint16))
    rng = np.random.default_rng(d + config)
    top = np.argmax(z, axis=1)
    at_top = z[np.arange(rows), top].copy()
    z[np.arange(rows), top] = -np.inf           # the runner-up: greatest other column
    second = np.argmax(z, axis=1)
    z[np.arange(rows), top] = at_top
    u = rng.random(rows)
    draft = np.where(u < 0.6, top, np.where(u < 0.9, second, rng.integers(0, vocab, rows)))
    draft = draft.astype(np.int32)
    draft[rng.random(rows) < 0.01] = vocab + 5            # outside the vocabulary
    budget = w.budget.copy()
    got = _run_device(hidden, weight, draft, w, budget)
    ref = oracle.verify(z, draft, w.block_lens, w.tau, w.exc_cap, budget, w.row_offsets)
    accepted_mismatch = (ref["budget"][:, 1] != budget[:, 1]).sum()
    print("  oracle: mean a %.2f, %d requests spent budget" % (ref["accept_len"].mean(),
                                                               accepted_mismatch), flush=True)
    assert accepted_mismatch > 0
    bad = mismatches(got, ref)
    assert not bad, "differs in %s: %s" % (bad, describe(got, ref))


def _run_device(hidden, weight, draft, w, budget):
    """asd_lmhead_verify on device tensors with a workload's requests."""
    import torch
    import paper_2608_03447_amd as asd
    dev = hidden.device
    rows = hidden.shape[0]
    tb = torch.from_numpy(budget.copy()).to(dev)
    amax = torch.full((rows,), -7, dtype=torch.int32, device=dev)
    regret = torch.full((rows,), float("nan"), dtype=torch.float32, device=dev)
    offs = None if w.row_offsets is None else torch.from_numpy(w.row_offsets).to(dev)
    acc, nxt = asd.asd_lmhead_verify(
        hidden, weight, torch.from_numpy(draft).to(dev), torch.from_numpy(w.block_lens).to(dev),
        torch.from_numpy(w.tau).to(dev), torch.from_numpy(w.exc_cap).to(dev), tb,
        row_offsets=offs, out_argmax=amax, out_regret=regret)
    torch.cuda.synchronize(dev)
    return {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
            "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
            "budget": tb.cpu().numpy()}


def test_maximum_hidden_size_bit_exact():
    """d = 2^20, the largest hidden size the call accepts: the copies reach
    their largest offsets (255 rows of 2 MB) and the K loop runs 16,384
    steps.  Exact regime: every partial sum is a multiple of 1/2 below 2^22."""
    from asd_gpu import describe, mismatches
    rng = np.random.default_rng(20)
    rows, vocab, d = 4, 257, 1 << 20
    hidden = W.f32_to_bf16(rng.integers(-2, 3, size=(rows, d)).astype(np.float32))
    weight = W.f32_to_bf16((rng.integers(-2, 3, size=(vocab, d)) / 2.0).astype(np.float32))
    draft = rng.integers(0, vocab, rows).astype(np.int32)
    print("case lmhead rows %d vocab %d d %d" % (rows, vocab, d), flush=True)
    g = _run(hidden, weight, draft, [3], 1.0, 2, [[4.0, 0.0]])
    r = oracle.lmhead_verify(hidden, weight, draft, [3], 1.0, 2, [[4.0, 0.0]])
    bad = mismatches(g, r)
    assert not bad, "differs in %s: %s" % (bad, describe(g, r))


def _fuzz_case(seed):
    """One random exact-regime case: shape, row kinds (as in the non-finite
    test), drafts and batch layout all drawn from the seed."""
    rng = np.random.default_rng(1000 + seed)
    rows = int(rng.integers(1, 700))
    vocab = int(rng.integers(1, 3000))
    d = int(rng.choice([128, 256, 384, 512]))
    h = rng.integers(-2, 3, size=(rows, d)).astype(np.float32)
    w = (rng.integers(-2, 3, size=(vocab, d)) / 2.0).astype(np.float32)
    h[:, :3] = 0.0
    w[:, 0] = 1.0
    w[:, 1] = rng.integers(-1, 2, size=vocab)
    w[:, 2] = rng.choice([-0.5, 0.5], size=vocab)
    p_special = rng.choice([0.0, 0.05, 0.3])
    kind = np.where(rng.random(rows) < p_special, rng.integers(1, 7, size=rows), 0)
    h[kind == 1, 0] = -256.0
    h[kind == 2, 1] = np.inf
    h[kind == 3, 2] = np.inf
    h[kind == 4, 2] = -np.inf
    h[kind == 5, 3] = np.nan
    h[kind == 6] = 0.0
    draft = rng.integers(0, vocab, rows).astype(np.int32)
    draft[rng.random(rows) < 0.05] = -1
    lens = []
    left = rows
    while left > 0:
        k = int(min(left - 1, rng.integers(0, 12)))
        lens.append(k)
        left -= k + 1
    budget = np.stack([rng.uniform(0, 6, len(lens)), np.zeros(len(lens))], axis=1)
    return rows, vocab, d, W.f32_to_bf16(h), W.f32_to_bf16(w), draft, lens, budget


@pytest.mark.parametrize("seed", range(40))
def test_fuzz_exact_regime_bit_exact(seed):
    """Random shapes (ragged row and column tiles, partly valid column quarters,
    one to four K steps) with ordinary and special rows mixed: every output
    bit-exact against the oracle."""
    from asd_gpu import describe, mismatches
    rows, vocab, d, hidden, weight, draft, lens, budget = _fuzz_case(seed)
    print("case lmhead fuzz seed %d rows %d vocab %d d %d" % (seed, rows, vocab, d), flush=True)
    g = _run(hidden, weight, draft, lens, 1.0, 2, budget)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget)
    bad = mismatches(g, r)
    assert not bad, "seed %d differs in %s: %s" % (seed, bad, describe(g, r))


def test_realistic_regime_within_rounding_bound():
    rng = np.random.default_rng(12)
    rows, vocab, d = 200, 4000, 1024
    hidden = W.f32_to_bf16(rng.normal(0, 1, size=(rows, d)).astype(np.float32))
    weight = W.f32_to_bf16(rng.normal(0, d ** -0.5, size=(vocab, d)).astype(np.float32))
    draft = rng.integers(0, vocab, rows).astype(np.int32)
    lens = [rows - 1]
    g = _run(hidden, weight, draft, lens, 1.0, 1, [[1.0, 0.0]])
    h64 = W.bf16_to_f32(hidden).astype(np.float64)
    w64 = W.bf16_to_f32(weight).astype(np.float64)
    z = h64 @ w64.T
    bound = 2.0 * d * 2.0 ** -24 * (np.abs(h64) @ np.abs(w64).T).max(axis=1)
    order = np.argsort(-z, axis=1, kind="stable")
    gap = z[np.arange(rows), order[:, 0]] - z[np.arange(rows), order[:, 1]]
    decided = gap > 2 * bound
    assert decided.mean() > 0.9
    assert np.array_equal(g["argmax"][decided], order[decided, 0])
    exact_at_gpu = z[np.arange(rows), g["argmax"]]
    assert np.all(z.max(axis=1) - exact_at_gpu <= 2 * bound)
    r_exact = z.max(axis=1)[:-1] - z[np.arange(rows - 1), draft[:-1]]
    assert np.all(np.abs(g["regret"][:-1] - r_exact) <= 4 * bound[:-1])


def test_explicit_row_offsets_in_any_order():
    """Requests listed in an order other than their rows' (explicit offsets)."""
    from asd_gpu import describe, mismatches
    rng = np.random.default_rng(31)
    rows, vocab, d = 260, 700, 256
    hidden, weight, draft = _exact_inputs(rng, rows, vocab, d)
    lens, o = [], 0
    offs = []
    while o < rows:
        k = int(min(rows - o - 1, rng.integers(0, 9)))
        lens.append(k)
        offs.append(o)
        o += k + 1
    perm = rng.permutation(len(lens))
    lens = np.asarray(lens, np.int32)[perm]
    offs = np.asarray(offs, np.int64)[perm]
    n = len(lens)
    tau = rng.uniform(0.2, 2.0, n).astype(np.float32)
    cap = rng.integers(0, 4, n).astype(np.int32)
    budget = np.stack([rng.uniform(0, 6, n), rng.uniform(0, 1, n)], axis=1)
    print("case lmhead offsets rows %d requests %d" % (rows, n), flush=True)
    g = _run(hidden, weight, draft, lens, tau, cap, budget, offsets=offs)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, tau, cap, budget.astype(np.float32),
                             row_offsets=offs)
    bad = mismatches(g, r)
    assert not bad, "differs in %s: %s" % (bad, describe(g, r))


def test_many_requests_use_the_offsets_pass():
    """More than 1,024 requests without offsets: the packed offsets come from a
    separate pass instead of each scan wavefront."""
    from asd_gpu import describe, mismatches
    rng = np.random.default_rng(32)
    n = 1100
    lens = rng.integers(0, 3, n).astype(np.int32)
    rows, vocab, d = int((lens + 1).sum()), 300, 128
    hidden, weight, draft = _exact_inputs(rng, rows, vocab, d)
    budget = np.stack([rng.uniform(0, 4, n), np.zeros(n)], axis=1)
    print("case lmhead many requests rows %d requests %d" % (rows, n), flush=True)
    g = _run(hidden, weight, draft, lens, 1.0, 2, budget)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget)
    bad = mismatches(g, r)
    assert not bad, "differs in %s: %s" % (bad, describe(g, r))


def test_optional_outputs_may_be_omitted():
    rng = np.random.default_rng(33)
    rows, vocab, d = 130, 1027, 128
    hidden, weight, draft = _exact_inputs(rng, rows, vocab, d)
    lens = [8] * 14 + [3]
    budget = np.stack([rng.uniform(0, 6, 15), np.zeros(15)], axis=1)
    g = _run(hidden, weight, draft, lens, 1.0, 2, budget, outputs=False)
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget)
    assert np.array_equal(g["accept_len"], r["accept_len"])
    assert np.array_equal(g["next_token"], r["next_token"])
    assert np.array_equal(g["budget"].view(np.uint32), r["budget"].view(np.uint32))


def test_graph_capture_replays_match_eager():
    """The call allocates nothing once the stream's workspace exists, so it can
    be captured; every replay equals the eager call and the oracle."""
    import torch
    import paper_2608_03447_amd as asd
    from asd_gpu import device_logits
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(34)
    rows, vocab, d = 300, 5000, 256
    hidden, weight, draft = _exact_inputs(rng, rows, vocab, d)
    lens = [9] * 30
    n = len(lens)
    budget0 = np.stack([rng.uniform(0, 6, n), np.zeros(n)], axis=1).astype(np.float32)
    th, tw = device_logits(hidden, dev), device_logits(weight, dev)
    td = torch.from_numpy(draft).to(dev)
    tl = torch.from_numpy(np.asarray(lens, np.int32)).to(dev)
    tt = torch.full((n,), 1.0, dtype=torch.float32, device=dev)
    tc = torch.full((n,), 2, dtype=torch.int32, device=dev)
    pristine = torch.from_numpy(budget0).to(dev)
    tb = pristine.clone()
    amax = torch.empty(rows, dtype=torch.int32, device=dev)
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):       # eager call: creates this stream's workspace
        acc, nxt = asd.asd_lmhead_verify(th, tw, td, tl, tt, tc, tb, out_argmax=amax)
    torch.cuda.synchronize()
    eager = [x.cpu().numpy().copy() for x in (acc, nxt, tb, amax)]
    r = oracle.lmhead_verify(hidden, weight, draft, lens, 1.0, 2, budget0)
    assert np.array_equal(eager[0], r["accept_len"]) and np.array_equal(eager[1], r["next_token"])
    assert np.array_equal(eager[2].view(np.uint32), r["budget"].view(np.uint32))
    assert np.array_equal(eager[3], r["argmax"])
    graph = torch.cuda.CUDAGraph()
    tb.copy_(pristine)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=side):
        asd.asd_lmhead_verify(th, tw, td, tl, tt, tc, tb, out_accept_len=acc, out_next_token=nxt,
                              out_argmax=amax)
    for replay in range(3):
        tb.copy_(pristine)
        acc.fill_(-5)
        nxt.fill_(-5)
        amax.fill_(-5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [x.cpu().numpy() for x in (acc, nxt, tb, amax)]
        for a, b in zip(got, eager):
            assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                  b.view(np.uint32) if b.dtype == np.float32 else b), replay
