"""The read probe behind the bench's practical read ceiling: it reads every
16-byte vector of every row (a value planted in any one vector reaches the
fold of the lane that reads it)."""
import numpy as np
import pytest
import torch

import paper_2608_03447_amd as asd

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
MARK = np.array([0x9E3779B9], dtype=np.uint32).view(np.int32)[0]


@pytest.mark.parametrize("rows,vecs", [(3, 4 * 256 + 3), (1, 1), (5, 4 * 256 * 3), (2, 300)])
def test_read_probe_folds_every_vector(rows, vecs):
    row_bytes = 16 * vecs
    print("probe rows %d vecs %d" % (rows, vecs), flush=True)
    buf = torch.zeros(rows * row_bytes // 4, dtype=torch.int32, device=DEV)
    out = torch.zeros(1, dtype=torch.int32, device=DEV)
    asd.asd_read_probe(buf, rows, row_bytes, out)
    torch.cuda.synchronize()
    assert out.item() == 0                          # an all-zero fold writes nothing
    words = buf.view(rows, vecs * 4)
    for r, v in {(rows - 1, vecs - 1), (0, 0), (rows // 2, vecs // 2)}:
        words.zero_()
        words[r, 4 * v + 1] = int(MARK)             # one word of vector v of row r
        out.zero_()
        asd.asd_read_probe(buf, rows, row_bytes, out)
        torch.cuda.synchronize()
        assert out.item() == int(MARK), (r, v)


@pytest.mark.parametrize("workgroups,steps", [(1, 1), (3, 5), (300, 2)])
def test_mfma_probe_runs_every_step(workgroups, steps):
    """With every operand 1.0 each accumulator of thread 0 ends at 64 * steps,
    so its 128 accumulators sum to 8192 * steps (exact in binary32)."""
    print("mfma probe workgroups %d steps %d" % (workgroups, steps), flush=True)
    ops = torch.ones(24 * 8 * 4, dtype=torch.bfloat16, device=DEV)
    out = torch.zeros(workgroups, dtype=torch.int32, device=DEV)
    asd.asd_mfma_probe(ops, workgroups, steps, out)
    torch.cuda.synchronize()
    expect = np.array([8192.0 * steps], dtype=np.float32).view(np.int32)[0]
    assert (out.cpu().numpy() == expect).all()
