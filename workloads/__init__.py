"""Seeded synthetic workloads for the ASD verifier.

This module holds no verifier arithmetic.  It writes host buffers that both
the CPU oracle and the GPU library read, so inputs are identical on the two
sides by construction.  The heavy per-element work (normal draws, planting a
greedy peak) is in ``gen.c``; this file only lays out the five workload
shapes and draws the per-row and per-request choices.

The shapes stand in for target logits of the paper's Qwen3-14B
(|V| = 151,936) and DeepSeek-class (|V| = 129,280) targets; the paper's
datasets and weights are not used.

Row recipe (every config): z = N(0, sigma^2) noise rounded to the dtype; a
peak column p drawn uniformly; the greatest other value m (first column w);
z[p] = round(m + c).  p is then the greedy token, w the runner-up.  A draft
takes p, w or a uniform token with the config's probabilities; the bonus row
of every block gets a uniform token, which the verifier ignores.
"""
import ctypes
import dataclasses
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "gen.c")
LIBRARY = os.path.join(HERE, "libasdgen.so")

F32, BF16 = 0, 1

# Stream ids of the counter-based generator, one per kind of draw.
_S_NOISE, _S_PEAK, _S_MARGIN, _S_TIE, _S_ROLE, _S_UNIFORM, _S_LENS, _S_TAU, _S_BUDGET = range(1, 10)


def build_generator(verbose: bool = False) -> str:
    cmd = ["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
           "-Wall", SOURCE, "-o", LIBRARY + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIBRARY + ".tmp", LIBRARY)
    return LIBRARY


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build_generator()
        lib = ctypes.CDLL(LIBRARY)
        u64, i64, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p
        lib.gen_splitmix64_at.argtypes = [u64, u64]
        lib.gen_splitmix64_at.restype = u64
        lib.gen_u01.argtypes = [u64, u64, i64, vp]
        lib.gen_u01.restype = None
        lib.gen_normal_rows.argtypes = [u64, ctypes.c_int, i64, i64, i64, ctypes.c_double, vp]
        lib.gen_normal_rows.restype = None
        lib.gen_plant_rows.argtypes = [ctypes.c_int, i64, i64, vp, vp, vp, vp]
        lib.gen_plant_rows.restype = None
        lib.gen_num_threads.argtypes = []
        lib.gen_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def splitmix64_at(seed: int, k: int) -> int:
    return int(_load().gen_splitmix64_at(seed & (2**64 - 1), k & (2**64 - 1)))


def stream_key(seed: int, config: int, stream: int) -> int:
    """Key of one stream of draws for (seed, config)."""
    return splitmix64_at(splitmix64_at(seed, config), stream)


def u01(key: int, k0: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    if n:
        _load().gen_u01(key, k0, n, _p(out))
    return out


def uniform_index(key: int, k0: int, n: int, high: int) -> np.ndarray:
    """n draws uniform over {0, ..., high-1}."""
    return np.minimum((u01(key, k0, n) * high).astype(np.int64), high - 1)


@dataclasses.dataclass
class Workload:
    """Inputs of one or more verifier calls.

    ``logits`` is [rows, vocab] float32, or uint16 bf16 bit patterns.  For
    ``blocks > 1`` (sequential decoding of one batch) call b reads rows
    ``[b * rows_per_call, (b + 1) * rows_per_call)`` with the same per-request
    arrays, and the budget ledger is carried from call to call.
    """
    name: str
    dtype: str                      # "bf16" or "f32"
    vocab: int
    logits: np.ndarray
    draft_tokens: np.ndarray        # int32 [rows]
    block_lens: np.ndarray          # int32 [num_requests]
    tau: np.ndarray                 # float32 [num_requests]  (local gate g)
    exc_cap: np.ndarray             # int32 [num_requests]    (block cap M)
    budget: np.ndarray              # float32 [num_requests, 2] = (B, s)
    peak_col: np.ndarray            # int64 [rows]  planted greedy column
    runner_col: np.ndarray          # int32 [rows]  runner-up column
    row_offsets: Optional[np.ndarray] = None
    blocks: int = 1

    @property
    def num_requests(self) -> int:
        return int(self.block_lens.shape[0])

    @property
    def rows_per_call(self) -> int:
        return int(self.logits.shape[0] // self.blocks)

    @property
    def logit_bytes_per_call(self) -> int:
        return self.rows_per_call * self.vocab * self.logits.itemsize

    def call(self, b: int):
        """Per-call slices: (logits, draft_tokens) of sequential call b."""
        n = self.rows_per_call
        return self.logits[b * n:(b + 1) * n], self.draft_tokens[b * n:(b + 1) * n]


def _rows(seed, config, dtype, vocab, nrows, sigma, margin, mix, block_lens_per_call, blocks,
          tie_rate=0.0, margin_uniform=None):
    """Logits, drafts and planted columns for ``blocks`` calls of the given layout."""
    code = BF16 if dtype == "bf16" else F32
    gen = _load()
    logits = np.empty((nrows, vocab), dtype=np.uint16 if code == BF16 else np.float32)
    gen.gen_normal_rows(stream_key(seed, config, _S_NOISE), code, vocab, 0, nrows, float(sigma),
                        _p(logits))
    peak = uniform_index(stream_key(seed, config, _S_PEAK), 0, nrows, vocab)
    if margin_uniform is not None:
        lo, hi = margin_uniform
        marg = (lo + (hi - lo) * u01(stream_key(seed, config, _S_MARGIN), 0, nrows)).astype(np.float32)
    else:
        marg = np.full(nrows, margin, dtype=np.float32)
    if tie_rate > 0.0:
        tie = u01(stream_key(seed, config, _S_TIE), 0, nrows) < tie_rate
        marg[tie] = np.float32(0.0)
    runner = np.empty(nrows, dtype=np.int32)
    gen.gen_plant_rows(code, vocab, nrows, _p(logits), _p(peak), _p(marg), _p(runner))

    # Draft roles: the planted peak, the runner-up, or a uniform token.
    role_u = u01(stream_key(seed, config, _S_ROLE), 0, nrows)
    uni = uniform_index(stream_key(seed, config, _S_UNIFORM), 0, nrows, vocab)
    p_peak, p_runner = mix
    draft = np.where(role_u < p_peak, peak,
                     np.where(role_u < p_peak + p_runner, runner.astype(np.int64), uni))
    # Bonus rows: a uniform token (the verifier must ignore it).
    ends = []
    start = 0
    for _ in range(blocks):
        for k in block_lens_per_call:
            ends.append(start + int(k))
            start += int(k) + 1
    assert start == nrows
    draft[np.asarray(ends, dtype=np.int64)] = uni[np.asarray(ends, dtype=np.int64)]
    return logits, draft.astype(np.int32), peak, runner


def make_config(index: int, seed: Optional[int] = None, *, batch: Optional[int] = None,
                vocab: Optional[int] = None, variant: str = "asd") -> Workload:
    """Build one of the five benchmark workloads.

    1: one request decoding 64 sequential blocks of K=8, V=32,000 fp32 N(0,1),
       peak +3.0, drafts 70% greedy / 20% runner-up / 10% uniform,
       g=1.5, M=1, B=4.0 carried across the blocks.  Seed 0.
    2: B=32 requests, K=16, V=151,936 bf16 N(0,2^2), peak +4.0,
       drafts 75/15/10, g=2.0, M=1, B=8.0.
    3: B=256 requests, K=16, V=151,936 bf16 N(0,2^2), peak +4.0,
       drafts 75/15/10, g=2.0, M=2, budgets U[0,16].  The headline shape.
    4: B=64 requests, K=32, V=151,936 fp32 N(0,2^2); the top two values
       differ by U[0,0.5] and by exactly 0 in 1% of rows; drafts take the
       runner-up w.p. 0.4, else the planted top.  variant "asd": M=4, g=1.0,
       B=1.0; "asd_b8": the same with B=8.0; "strict": B=0.
    5: B=512 requests with K_i uniform on 1..8 (packed rows), V=129,280 bf16
       N(0,2^2), peak +3.5, drafts 65/25/10, g_i ~ U[0.5,3.0],
       budgets U[0,10], M=1.
    ``batch`` and ``vocab`` shrink a workload for quick tests; ``seed``
    defaults to 0 for config 1 and to the config index otherwise.
    """
    if seed is None:
        seed = 0 if index == 1 else index
    if index == 1:
        V = vocab or 32000
        blocks = 64 if batch is None else batch
        K = 8
        lens = np.array([K], dtype=np.int32)
        nrows = blocks * (K + 1)
        logits, draft, peak, runner = _rows(seed, 1, "f32", V, nrows, 1.0, 3.0, (0.7, 0.2),
                                            [K], blocks)
        return Workload("seq64_b1_k8_v%d_f32" % V, "f32", V, logits, draft, lens,
                        np.array([1.5], np.float32), np.array([1], np.int32),
                        np.array([[4.0, 0.0]], np.float32), peak, runner, None, blocks)
    if index in (2, 3):
        V = vocab or 151936
        B = batch or (32 if index == 2 else 256)
        K = 16
        lens = np.full(B, K, dtype=np.int32)
        nrows = B * (K + 1)
        logits, draft, peak, runner = _rows(seed, index, "bf16", V, nrows, 2.0, 4.0,
                                            (0.75, 0.15), list(lens), 1)
        if index == 2:
            budget = np.tile(np.array([[8.0, 0.0]], np.float32), (B, 1))
            cap = 1
        else:
            budget = np.zeros((B, 2), np.float32)
            budget[:, 0] = (16.0 * u01(stream_key(seed, index, _S_BUDGET), 0, B)).astype(np.float32)
            cap = 2
        return Workload("b%d_k16_v%d_bf16" % (B, V), "bf16", V, logits, draft,
                        lens, np.full(B, 2.0, np.float32), np.full(B, cap, np.int32), budget,
                        peak, runner)
    if index == 4:
        V = vocab or 151936
        B = batch or 64
        K = 32
        lens = np.full(B, K, dtype=np.int32)
        nrows = B * (K + 1)
        logits, draft, peak, runner = _rows(seed, 4, "f32", V, nrows, 2.0, None, (0.6, 0.4),
                                            list(lens), 1, tie_rate=0.01,
                                            margin_uniform=(0.0, 0.5))
        total = {"asd": 1.0, "asd_b8": 8.0, "strict": 0.0}[variant]
        budget = np.tile(np.array([[total, 0.0]], np.float32), (B, 1))
        return Workload("b%d_k32_v%d_f32_%s" % (B, V, variant), "f32", V, logits, draft,
                        lens, np.full(B, 1.0, np.float32), np.full(B, 4, np.int32), budget,
                        peak, runner)
    if index == 5:
        V = vocab or 129280
        B = batch or 512
        lens = (1 + uniform_index(stream_key(seed, 5, _S_LENS), 0, B, 8)).astype(np.int32)
        nrows = int(np.sum(lens.astype(np.int64) + 1))
        logits, draft, peak, runner = _rows(seed, 5, "bf16", V, nrows, 2.0, 3.5, (0.65, 0.25),
                                            list(lens), 1)
        tau = (0.5 + 2.5 * u01(stream_key(seed, 5, _S_TAU), 0, B)).astype(np.float32)
        budget = np.zeros((B, 2), np.float32)
        budget[:, 0] = (10.0 * u01(stream_key(seed, 5, _S_BUDGET), 0, B)).astype(np.float32)
        return Workload("b%d_ragged1to8_v%d_bf16" % (B, V), "bf16", V, logits, draft,
                        lens, tau, np.ones(B, np.int32), budget, peak, runner)
    raise ValueError("unknown config %r" % index)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float32 (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 bit patterns, nearest-even (finite values)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)
