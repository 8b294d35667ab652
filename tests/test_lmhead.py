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


def _run(hidden, weight, draft, lens, tau, cap, budget, offsets=None):
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
        torch.from_numpy(np.ascontiguousarray(np.broadcast_to(np.float32(tau), (n,)))).to(dev),
        torch.from_numpy(np.ascontiguousarray(np.broadcast_to(np.int32(cap), (n,)))).to(dev),
        tb, row_offsets=to, out_argmax=amax, out_regret=regret)
    torch.cuda.synchronize()
    return {"accept_len": acc.cpu().numpy(), "next_token": nxt.cpu().numpy(),
            "argmax": amax.cpu().numpy(), "regret": regret.cpu().numpy(),
            "budget": tb.cpu().numpy()}


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
