"""asd_row_pass (the verifier's row pass alone, on the call's own tile grid)
against the CPU oracle, through the C ABI.

Each tile's partial is decoded here (white box: a packed (key, column) whose
unsigned maximum ranks rows as Eq. 1 does, the binary32 bits of that value, and
the draft token's logit in the tile that holds its column).  Combined over the
S tiles of a row they must give the oracle's argmax, that logit's bits, and the
draft logit's bits, exactly.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03447_amd as asd
import workloads as W
from asd_gpu import device_logits

pytestmark = pytest.mark.gpu

SPECIAL_BITS = np.array([0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x3f800000, 0xbf800000,
                         0x7f800000, 0xff800000, 0x7fc00000, 0xffc00000, 0x7f800001, 0xff800001],
                        dtype=np.uint32)


def f32_bits(logits):
    """Each logit's binary32 bit pattern (bf16 patterns widened)."""
    if logits.dtype == np.uint16:
        return logits.astype(np.uint32) << 16
    return np.ascontiguousarray(logits).view(np.uint32)


def run_and_check(logits, draft, label):
    rows, vocab = logits.shape
    print("case %s: rows %d vocab %d dtype %s" % (label, rows, vocab, logits.dtype), flush=True)
    dev = torch.device("cuda:0")
    tl = device_logits(logits, dev)
    td = torch.from_numpy(np.ascontiguousarray(draft, dtype=np.int32)).to(dev)
    splits = asd.asd_row_splits(tl.dtype, vocab, rows)
    parts = asd.asd_row_pass(tl, td)
    torch.cuda.synchronize()
    assert splits >= 1 and tuple(parts.shape) == (rows, splits, 4)
    w = parts.cpu().numpy().view(np.uint32)
    packed = w[:, :, 0].astype(np.uint64) | (w[:, :, 1].astype(np.uint64) << np.uint64(32))
    best = np.argmax(packed, axis=1)                 # unsigned maximum over the tiles
    take = np.arange(rows)
    col = (np.uint64(0xffffffff) - (packed[take, best] & np.uint64(0xffffffff))).astype(np.int64)
    bits = w[take, best, 2]
    draft_bits = np.bitwise_or.reduce(w[:, :, 3], axis=1)

    y = oracle.argmax_rows(logits)
    zb = f32_bits(logits)
    assert np.array_equal(col, y.astype(np.int64)), "%s: argmax differs in %d rows" % (
        label, int(np.sum(col != y)))
    assert np.array_equal(bits, zb[take, y]), "%s: max bits differ" % label
    valid = (draft >= 0) & (draft < vocab)
    want = np.where(valid, zb[take, np.clip(draft, 0, vocab - 1)], 0).astype(np.uint32)
    assert np.array_equal(draft_bits, want), "%s: draft logit bits differ" % label
    return splits


@pytest.mark.parametrize("cfg,batch", [(2, None), (3, 16), (4, 8), (5, 24)])
def test_row_pass_matches_oracle_on_workloads(cfg, batch):
    w = W.make_config(cfg, batch=batch)
    rows = w.rows_per_call
    logits = w.logits[:rows]
    draft = w.draft_tokens[:rows]
    splits = run_and_check(logits, draft, "workload %d" % cfg)
    if cfg == 2:
        assert splits > 1        # 544 rows of 151,936 bf16: the call splits them


@pytest.mark.parametrize("rows,vocab,dtype", [(1, 151936, "bf16"), (3, 32000, "f32"),
                                              (7, 1001, "bf16"), (300, 1001, "f32"),
                                              (2, 9, "bf16"), (40, 65536, "bf16"),
                                              (1200, 5003, "bf16")])
def test_row_pass_special_values_and_ragged_tiles(rows, vocab, dtype):
    rng = np.random.default_rng(rows * 7919 + vocab)
    z = rng.normal(0, 3, size=(rows, vocab)).astype(np.float32)
    special = SPECIAL_BITS[rng.integers(0, len(SPECIAL_BITS), size=(rows, vocab))].view(np.float32)
    frac = rng.choice([0.0, 0.001, 0.3], size=(rows, 1))
    z = np.where(rng.random((rows, vocab)) < frac, special, z).astype(np.float32)
    z[rows // 2] = -np.abs(z[rows // 2])                    # a row with no positive number
    logits = W.f32_to_bf16(z) if dtype == "bf16" else z
    y = oracle.argmax_rows(logits)
    draft = np.where(rng.random(rows) < 0.5, y, rng.integers(-2, vocab + 2, rows)).astype(np.int32)
    run_and_check(logits, draft, "%d x %d %s" % (rows, vocab, dtype))


def test_row_splits_matches_the_verifier_workspace_plan():
    """The split count asd_row_pass uses is the one asd_verify plans: the
    verifier's workspace holds one 16-byte partial per tile when S > 1."""
    for rows, vocab, dt in [(544, 151936, torch.bfloat16), (4352, 151936, torch.bfloat16),
                            (9, 32000, torch.float32), (2112, 151936, torch.float32)]:
        s = asd.asd_row_splits(dt, vocab, rows)
        assert 1 <= s <= 64
        code = asd.ASD_BF16 if dt == torch.bfloat16 else asd.ASD_F32
        ws = asd.asd_workspace_bytes(code, vocab, 1, rows)
        if s > 1:
            assert ws >= rows * s * 16
