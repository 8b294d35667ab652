"""Host-side parts of bench.py, on the CPU: the acceptance diagnostics count
what the verifier's outputs say (the outputs here come from the oracle)."""
import os
import sys
import types

import numpy as np
import torch

import oracle

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


class _OracleAsd:
    """Stands in for the binding: fills the output tensors from the oracle."""

    @staticmethod
    def asd_verify(lg, dr, lens, tau, cap, budget, out_accept_len, out_next_token,
                   out_argmax, out_regret):
        out = oracle.verify(lg.numpy(), dr.numpy(), lens.numpy(), tau.numpy(), cap.numpy(),
                            budget.numpy())
        out_accept_len.copy_(torch.from_numpy(out["accept_len"]))
        out_next_token.copy_(torch.from_numpy(out["next_token"]))
        out_argmax.copy_(torch.from_numpy(out["argmax"]))
        out_regret.copy_(torch.from_numpy(np.nan_to_num(out["regret"], nan=0.0)))
        budget.copy_(torch.from_numpy(out["budget"]))


def test_acceptance_diagnostics_classify_every_stop():
    V, K = 8, 4
    # Five requests of K = 4; row p of a request has its greedy token at p % V.
    rows = 5 * (K + 1)
    z = np.zeros((rows, V), np.float32)
    for r in range(rows):
        z[r, r % V] = 3.0
    y = np.arange(rows) % V
    draft = y.copy().astype(np.int32)
    # request 0: every draft matches              -> end of block
    # request 1: B = 0 and a mismatch at p = 1   -> strict dispatch
    # request 2: mismatch with regret 3 > g q    -> gate
    # request 3: cap M = 0                       -> cap
    # request 4: budget 1 < regret 3             -> budget
    for req in (1, 2, 3, 4):
        o = req * (K + 1)
        draft[o + 1] = (y[o + 1] + 1) % V
    tau = np.array([1.0, 1.0, 0.1, 10.0, 10.0], np.float32)
    cap = np.array([2, 2, 2, 0, 2], np.int32)
    budget = np.array([[8, 0], [0, 0], [8, 0], [8, 0], [1, 0]], np.float32)
    w = types.SimpleNamespace(rows_per_call=rows, num_requests=5,
                              block_lens=np.full(5, K, np.int32), tau=tau, exc_cap=cap)
    acc = torch.zeros(5, dtype=torch.int32)
    nxt = torch.zeros(5, dtype=torch.int32)
    calls = [(torch.from_numpy(z), torch.from_numpy(draft), acc, nxt)]
    got = bench.acceptance_diagnostics(_OracleAsd, torch, w, calls,
                                       torch.from_numpy(w.block_lens), torch.from_numpy(tau),
                                       torch.from_numpy(cap), torch.from_numpy(budget))
    assert got["stop_reasons"] == {"end_of_block": 1, "strict_dispatch": 1, "gate": 1,
                                   "cap": 1, "budget": 1}
    assert got["blocks"] == 5
    assert got["mean_accept_len"] == (4 + 1 + 1 + 1 + 1) / 5
    assert got["mean_strict_accept_len"] == (4 + 1 + 1 + 1 + 1) / 5
    assert got["mean_accepted_exceptions"] == 0
    assert got["mean_budget_spent"] == 0


def test_acceptance_diagnostics_count_accepted_exceptions():
    V, K = 8, 4
    z = np.zeros((K + 1, V), np.float32)
    for r in range(K + 1):
        z[r, r] = 3.0
        z[r, (r + 1) % V] = 2.5                    # runner-up half a logit below
    draft = np.arange(K + 1, dtype=np.int32)
    draft[0] = 1                                   # regret 0.5 at p = 0
    draft[2] = 3                                   # regret 0.5 at p = 2
    w = types.SimpleNamespace(rows_per_call=K + 1, num_requests=1,
                              block_lens=np.array([K], np.int32),
                              tau=np.array([1.0], np.float32), exc_cap=np.array([2], np.int32))
    budget = np.array([[4.0, 0.0]], np.float32)
    calls = [(torch.from_numpy(z), torch.from_numpy(draft), torch.zeros(1, dtype=torch.int32),
              torch.zeros(1, dtype=torch.int32))]
    got = bench.acceptance_diagnostics(_OracleAsd, torch, w, calls,
                                       torch.from_numpy(w.block_lens), torch.from_numpy(w.tau),
                                       torch.from_numpy(w.exc_cap), torch.from_numpy(budget))
    assert got["mean_accept_len"] == 4 and got["mean_strict_accept_len"] == 0
    assert got["mean_accepted_exceptions"] == 2
    assert got["mean_budget_spent"] == 1.0
    assert got["stop_reasons"]["end_of_block"] == 1


def test_workload_tag_names_the_shape():
    class Wk:
        num_requests, vocab, dtype, blocks = 256, 151936, "bf16", 1
    assert bench.workload_tag(3, Wk) == "b256_k16_v151936_bf16"
    Wk.blocks = 64
    assert bench.workload_tag(1, Wk).endswith("_seq64")


def test_threaded_oracle_pieces_reproduce_the_whole_call():
    import workloads as W
    for cfg in (3, 5):
        w = W.make_config(cfg, batch=24, vocab=3000)
        ref = oracle.verify(w.logits, w.draft_tokens, w.block_lens, w.tau, w.exc_cap, w.budget)
        whole = (ref["accept_len"][None], ref["next_token"][None], ref["budget"])
        got = bench.threaded_oracle(w, whole, 0.01, max_threads=4)
        assert got["kind"] == "oracle" and 1 <= got["cores"] <= 4 and got["value"] > 0
        assert got["sample"].endswith("True")


def test_host_info_reports_cpu_count():
    info = bench.host_info()
    assert info["nproc"] == os.cpu_count()
