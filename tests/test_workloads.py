"""The seeded input generators: determinism, the published SplitMix64
sequence, and the shape of each workload (peak margin, draft mix)."""
import numpy as np
import pytest

import workloads as W


def test_splitmix64_matches_published_sequence():
    # First outputs of SplitMix64 seeded with 1234567 (the reference sequence
    # printed with Vigna's splitmix64.c test driver).
    expect = [6457827717110365317, 3203168211198807973, 9817491932198370423,
              4593380528125082431, 16408922859458223821]
    assert [W.splitmix64_at(1234567, k) for k in range(5)] == expect


def test_generation_is_deterministic_and_seed_dependent():
    a = W.make_config(3, batch=2, vocab=5000)
    b = W.make_config(3, batch=2, vocab=5000)
    c = W.make_config(3, seed=99, batch=2, vocab=5000)
    assert np.array_equal(a.logits, b.logits) and np.array_equal(a.draft_tokens, b.draft_tokens)
    assert not np.array_equal(a.logits, c.logits)


def test_rows_do_not_depend_on_batch_size():
    small = W.make_config(2, batch=2, vocab=3000)
    big = W.make_config(2, batch=5, vocab=3000)
    n = small.logits.shape[0]
    assert np.array_equal(small.logits, big.logits[:n])


@pytest.mark.parametrize("cfg,margin", [(1, 3.0), (2, 4.0), (5, 3.5)])
def test_planted_peak_is_the_unique_greedy_token(cfg, margin):
    w = W.make_config(cfg, batch=4, vocab=20000)
    z = w.logits if w.dtype == "f32" else W.bf16_to_f32(w.logits)
    rows = np.arange(z.shape[0])
    top = z[rows, w.peak_col]
    runner = z[rows, w.runner_col]
    assert np.all(np.argmax(z, axis=1) == w.peak_col)
    gap = top - runner
    assert np.all(np.abs(gap - margin) <= 0.07)


def test_noise_moments():
    w = W.make_config(3, batch=2, vocab=151936)
    z = W.bf16_to_f32(w.logits).astype(np.float64)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 2.0) < 0.01


def test_draft_mix_proportions():
    w = W.make_config(3, batch=64, vocab=2000)
    K = 16
    rows = np.arange(w.logits.shape[0])
    draft_rows = rows[(rows % (K + 1)) != K]
    d = w.draft_tokens[draft_rows]
    p = np.mean(d == w.peak_col[draft_rows])
    r = np.mean(d == w.runner_col[draft_rows])
    assert abs(p - 0.75) < 0.03 and abs(r - 0.15) < 0.03


def test_near_tie_config_has_exact_duplicate_maxima():
    w = W.make_config(4, batch=64, vocab=3000)
    z = w.logits
    rows = np.arange(z.shape[0])
    gap = z[rows, w.peak_col] - z[rows, w.runner_col]
    assert np.all((gap >= 0) & (gap <= 0.5))
    ties = np.mean(gap == 0)
    assert 0.002 < ties < 0.03
    strict = W.make_config(4, batch=2, vocab=3000, variant="strict")
    assert np.all(strict.budget == 0)


def test_ragged_config_layout():
    w = W.make_config(5, batch=300, vocab=1000)
    assert w.block_lens.min() >= 1 and w.block_lens.max() <= 8
    assert w.logits.shape[0] == int(np.sum(w.block_lens + 1))
    assert np.all((w.tau >= 0.5) & (w.tau <= 3.0))
    assert np.all((w.budget[:, 0] >= 0) & (w.budget[:, 0] <= 10))


def test_bf16_round_trip():
    x = np.array([1.0, -2.5, 3.1415926, 1e-3, -0.0], dtype=np.float32)
    b = W.f32_to_bf16(x)
    assert np.array_equal(W.bf16_to_f32(b)[[0, 1]], x[[0, 1]])
    assert b[4] == 0x8000
