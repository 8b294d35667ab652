"""GPU opportunity statistic (Eq. 4) against the oracle: integer counts, exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W
from asd_gpu import gpu_verify

pytestmark = pytest.mark.gpu

TAUS = np.array([0.0, 0.5, 1.0, 2.0, 4.0, 8.0, np.inf], dtype=np.float32)
PS = np.array([0, 1, 2, 3, 4, 6, 8, 12], dtype=np.int32)


def gpu_counts(draft, amax, regret, vocab, lens, taus, ps, row_offsets=None, repeat=1):
    dev = torch.device("cuda:0")
    counts = torch.zeros((len(taus), len(ps)), dtype=torch.int64, device=dev)
    mism = torch.zeros(1, dtype=torch.int64, device=dev)
    args = [torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in
            (draft.astype(np.int32), amax.astype(np.int32), regret.astype(np.float32))]
    offs = None if row_offsets is None else torch.from_numpy(
        np.ascontiguousarray(row_offsets, dtype=np.int64)).to(dev)
    for _ in range(repeat):
        asd.asd_opportunity(*args, vocab, torch.from_numpy(np.asarray(lens, np.int32)).to(dev),
                            torch.from_numpy(taus).to(dev), torch.from_numpy(ps).to(dev), counts,
                            mism, row_offsets=offs)
    torch.cuda.synchronize()
    return counts.cpu().numpy().astype(np.uint64), int(mism.item())


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_opportunity_matches_oracle_on_workloads(cfg):
    w = W.make_config(cfg, batch=None if cfg != 3 else 64)
    print("case opportunity workload %d" % cfg, flush=True)
    g = gpu_verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    counts, m = gpu_counts(w.draft_tokens, g["argmax"], g["regret"], w.vocab, w.block_lens,
                           TAUS, PS)
    ref_v = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
    ref_c, ref_m = oracle.opportunity(w.draft_tokens, ref_v["argmax"], ref_v["regret"], w.vocab,
                                      w.block_lens, TAUS, PS)
    assert m == ref_m and np.array_equal(counts, ref_c)
    assert m > 0 and counts[-1, 1] > 0


@pytest.mark.parametrize("num_requests,explicit", [
    (1, False), (3, False), (4, False), (5, False), (1023, False), (1024, False), (1025, False),
    (3000, False), (3000, True), (8193, False), (70000, False), (70000, True)])
def test_opportunity_offsets_across_workgroups_and_accumulation(num_requests, explicit):
    """Packed (row_offsets NULL) or explicit offsets, from one request to 70,000:
    above 8,192 packed requests each workgroup takes 64 requests."""
    rng = np.random.default_rng(num_requests)
    vocab = 300
    lens = rng.integers(0, 14, num_requests).astype(np.int32)
    rows = int(np.sum(lens + 1))
    y = rng.integers(0, vocab, rows).astype(np.int32)
    draft = np.where(rng.random(rows) < 0.7, y, rng.integers(-1, vocab + 1, rows)).astype(np.int32)
    regret = rng.choice(np.array([0.0, 0.25, 1.0, 3.0, np.inf, np.nan], np.float32), rows)
    offs = None if not explicit else np.concatenate(
        [[0], np.cumsum(lens.astype(np.int64) + 1)[:-1]])
    print("case opportunity: %d requests, %s offsets" % (num_requests,
                                                         "explicit" if explicit else "packed"),
          flush=True)
    counts, m = gpu_counts(draft, y, regret, vocab, lens, TAUS, PS, row_offsets=offs, repeat=2)
    ref_c, ref_m = oracle.opportunity(draft, y, regret, vocab, lens, TAUS, PS)
    assert m == 2 * ref_m and np.array_equal(counts, 2 * ref_c)


def test_opportunity_long_blocks_cross_64_position_chunks():
    rng = np.random.default_rng(64)
    vocab = 100
    lens = np.array([63, 64, 65, 127, 128, 129, 200, 0, 1], dtype=np.int32)
    rows = int(np.sum(lens + 1))
    y = rng.integers(0, vocab, rows).astype(np.int32)
    for p_match in (0.5, 0.95, 1.0):
        draft = np.where(rng.random(rows) < p_match, y, rng.integers(0, vocab, rows)).astype(np.int32)
        draft[[10, 70, 200]] = -1                        # a few invalid ids
        regret = rng.uniform(0, 2, rows).astype(np.float32)
        ps = np.array([0, 1, 5, 30, 63, 64, 65, 100, 199], dtype=np.int32)
        counts, m = gpu_counts(draft, y, regret, vocab, lens, TAUS, ps)
        ref_c, ref_m = oracle.opportunity(draft, y, regret, vocab, lens, TAUS, ps)
        assert m == ref_m and np.array_equal(counts, ref_c), p_match


def test_opportunity_explicit_offsets_and_invalid_requests():
    rng = np.random.default_rng(5)
    vocab, rows = 50, 80
    y = rng.integers(0, vocab, rows).astype(np.int32)
    draft = np.where(rng.random(rows) < 0.6, y, rng.integers(0, vocab, rows)).astype(np.int32)
    regret = rng.uniform(0, 3, rows).astype(np.float32)
    lens = np.array([5, -2, 9, 30, 4], dtype=np.int32)
    offs = np.array([0, 6, 7, 60, 74], dtype=np.int64)
    counts, m = gpu_counts(draft, y, regret, vocab, lens, TAUS, PS, row_offsets=offs)
    ref_c, ref_m = oracle.opportunity(draft, y, regret, vocab, lens, TAUS, PS, row_offsets=offs)
    assert m == ref_m and np.array_equal(counts, ref_c)
