"""CPU oracle of the ASD verifier -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does, and it
shares no code with the HIP path.

The arithmetic lives in ``asd_oracle.c`` (plain sequential C); this module only
marshals numpy arrays to it.  Logits are numpy ``float32`` arrays, or ``uint16``
arrays holding bf16 bit patterns.
"""
import ctypes
import os

import numpy as np

from .build import LIBRARY, build_oracle

F32 = 0
BF16 = 1

RAW_GATE = 1            # flag: gate on r <= g instead of r / q <= g
ERR_NEGATIVE_K = 1      # error-word bit: some K < 0 (read as 0)
ERR_ROWS = 2            # error-word bit: some request's rows outside [0, total_rows)

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build_oracle()
        lib = ctypes.CDLL(LIBRARY)
        i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
        lib.oracle_ranks_above.argtypes = [f32, f32]
        lib.oracle_ranks_above.restype = ctypes.c_int
        lib.oracle_row_argmax.argtypes = [vp, ctypes.c_int, i64, i64]
        lib.oracle_row_argmax.restype = i64
        lib.oracle_argmax_rows.argtypes = [vp, ctypes.c_int, i64, i64, vp]
        lib.oracle_argmax_rows.restype = None
        lib.oracle_block.argtypes = [i32, vp, vp, vp, vp, vp, f32, vp, f32, i32, ctypes.c_int,
                                     vp, vp, vp]
        lib.oracle_block.restype = None
        lib.oracle_verify.argtypes = [vp, ctypes.c_int, i64, i32, i64, vp, vp, vp, vp, vp, vp,
                                      vp, vp, vp, vp]
        lib.oracle_verify.restype = ctypes.c_int
        lib.oracle_verify_ex.argtypes = lib.oracle_verify.argtypes + [ctypes.c_uint32, vp]
        lib.oracle_verify_ex.restype = ctypes.c_int
        lib.oracle_opportunity.argtypes = [vp, vp, vp, i64, i32, i64, vp, vp, vp, i32, vp, i32,
                                           vp, vp]
        lib.oracle_opportunity.restype = None
        lib.oracle_commit.argtypes = [vp, vp, vp, i32, i64, vp, vp, vp, i64, vp, vp]
        lib.oracle_commit.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(logits):
    if logits.dtype == np.float32:
        return F32
    if logits.dtype == np.uint16:
        return BF16
    raise TypeError("logits must be float32 or uint16 (bf16 bit patterns), got %s" % logits.dtype)


def ranks_above(a, b):
    """True if logit value ``a`` ranks strictly above ``b`` in the argmax order."""
    return bool(_load().oracle_ranks_above(float(np.float32(a)), float(np.float32(b))))


def argmax_rows(logits):
    """Eq. 1 on every row of a [R, V] array: lowest index of the greatest value."""
    logits = np.ascontiguousarray(logits)
    code = _dtype_code(logits)
    rows, vocab = logits.shape
    out = np.empty(rows, dtype=np.int32)
    _load().oracle_argmax_rows(_ptr(logits), code, vocab, rows, _ptr(out))
    return out


def block(x, x_valid, y, z_y, z_x, B, s, g, M, raw_gate=False):
    """Algorithm 1 for one draft block.

    ``x`` (K,), ``x_valid`` (K,), ``y`` (K+1,), ``z_y`` (K,), ``z_x`` (K,).
    ``raw_gate`` gates on r <= g instead of r / q <= g.
    Returns ``(a, next_token, s_new, r)``.
    """
    x = np.ascontiguousarray(x, dtype=np.int32)
    K = x.shape[0]
    x_valid = np.ascontiguousarray(x_valid, dtype=np.uint8)
    y = np.ascontiguousarray(y, dtype=np.int32)
    z_y = np.ascontiguousarray(z_y, dtype=np.float32)
    z_x = np.ascontiguousarray(z_x, dtype=np.float32)
    assert x_valid.shape == (K,) and y.shape == (K + 1,) and z_y.shape == (K,) and z_x.shape == (K,)
    s_box = np.array([s], dtype=np.float32)
    a = np.zeros(1, dtype=np.int32)
    nxt = np.zeros(1, dtype=np.int32)
    r = np.zeros(max(K, 1), dtype=np.float32)
    _load().oracle_block(K, _ptr(x), _ptr(x_valid), _ptr(y), _ptr(z_y), _ptr(z_x),
                         float(np.float32(B)), _ptr(s_box), float(np.float32(g)), int(M),
                         int(bool(raw_gate)), _ptr(a), _ptr(nxt), _ptr(r))
    return int(a[0]), int(nxt[0]), np.float32(s_box[0]), r[:K].copy()


def verify(logits, draft_tokens, block_lens, tau, exc_cap, budget, row_offsets=None,
           raw_gate=False):
    """The whole verifier call on host arrays.

    ``budget`` is a float32 [B, 2] array of (total, spent); a new array with the
    updated ledger is returned (the input is not modified).  ``raw_gate`` gates
    on r <= g instead of the paper's r / q <= g.
    Returns a dict with ``accept_len``, ``next_token``, ``budget``, ``argmax``,
    ``regret`` (rows outside verified requests hold NaN) and ``error`` (the
    ERR_* bits of the call's requests).
    """
    logits = np.ascontiguousarray(logits)
    code = _dtype_code(logits)
    rows, vocab = logits.shape
    draft = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    lens = np.ascontiguousarray(block_lens, dtype=np.int32)
    nreq = lens.shape[0]
    tau = np.ascontiguousarray(np.broadcast_to(np.asarray(tau, dtype=np.float32), (nreq,)))
    cap = np.ascontiguousarray(np.broadcast_to(np.asarray(exc_cap, dtype=np.int32), (nreq,)))
    bud = np.array(budget, dtype=np.float32, copy=True).reshape(nreq, 2)
    offs = None if row_offsets is None else np.ascontiguousarray(row_offsets, dtype=np.int64)
    assert draft.shape == (rows,)
    accept = np.zeros(nreq, dtype=np.int32)
    nxt = np.zeros(nreq, dtype=np.int32)
    amax = np.zeros(rows, dtype=np.int32)
    regret = np.full(rows, np.nan, dtype=np.float32)
    err = np.zeros(1, dtype=np.uint32)
    rc = _load().oracle_verify_ex(_ptr(logits), code, vocab, nreq, rows, _ptr(draft), _ptr(lens),
                                  _ptr(offs), _ptr(tau), _ptr(cap), _ptr(bud), _ptr(accept),
                                  _ptr(nxt), _ptr(amax), _ptr(regret),
                                  RAW_GATE if raw_gate else 0, _ptr(err))
    if rc != 0:
        raise ValueError("oracle_verify rejected its arguments (code %d)" % rc)
    return {"accept_len": accept, "next_token": nxt, "budget": bud, "argmax": amax,
            "regret": regret, "error": int(err[0])}


def opportunity(draft_tokens, row_argmax, row_regret, vocab, block_lens, taus, ps,
                row_offsets=None):
    """Eq. 4 counts over one batch: returns ``(counts[len(taus), len(ps)], |M|)``.

    ``row_argmax`` / ``row_regret`` are the per-row outputs of :func:`verify`.
    Omega(taus[a], ps[b]) = counts[a, b] / |M|.
    """
    draft = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    amax = np.ascontiguousarray(row_argmax, dtype=np.int32)
    reg = np.ascontiguousarray(row_regret, dtype=np.float32)
    lens = np.ascontiguousarray(block_lens, dtype=np.int32)
    taus = np.ascontiguousarray(taus, dtype=np.float32)
    ps = np.ascontiguousarray(ps, dtype=np.int32)
    offs = None if row_offsets is None else np.ascontiguousarray(row_offsets, dtype=np.int64)
    counts = np.zeros((taus.shape[0], ps.shape[0]), dtype=np.uint64)
    mism = np.zeros(1, dtype=np.uint64)
    _load().oracle_opportunity(_ptr(draft), _ptr(amax), _ptr(reg), int(vocab), lens.shape[0],
                               draft.shape[0], _ptr(lens), _ptr(offs), _ptr(taus),
                               taus.shape[0], _ptr(ps), ps.shape[0], _ptr(counts), _ptr(mism))
    return counts, int(mism[0])


def commit(draft_tokens, block_lens, accept_len, next_token, tokens, seq_len, row_offsets=None):
    """Commit the emitted tokens (Sec. 3.3).  Returns new ``(tokens, seq_len, committed)``;
    ``tokens`` is [num_requests, capacity] int32, ``seq_len`` int64 [num_requests]."""
    draft = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    lens = np.ascontiguousarray(block_lens, dtype=np.int32)
    acc = np.ascontiguousarray(accept_len, dtype=np.int32)
    nxt = np.ascontiguousarray(next_token, dtype=np.int32)
    tok = np.array(tokens, dtype=np.int32, copy=True)
    sl = np.array(seq_len, dtype=np.int64, copy=True)
    offs = None if row_offsets is None else np.ascontiguousarray(row_offsets, dtype=np.int64)
    done = np.zeros(lens.shape[0], dtype=np.int32)
    _load().oracle_commit(_ptr(draft), _ptr(lens), _ptr(offs), lens.shape[0], draft.shape[0],
                          _ptr(acc), _ptr(nxt), _ptr(tok), tok.shape[1], _ptr(sl), _ptr(done))
    return tok, sl, done


def lmhead_logits(hidden_bits, weight_bits):
    """Logit rows z = H W^T of bf16 hidden states [R, d] and output weights [V, d]
    (uint16 bit patterns): the sum of the bf16 products taken in binary64 (a
    library matmul), rounded to binary32; a zero sum is +0.  Exact whenever the
    sum and its partial sums are representable in binary32 (small dyadic inputs)."""
    def widen(bits):
        return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(
            np.float32).astype(np.float64)
    z = widen(hidden_bits) @ widen(weight_bits).T
    return z.astype(np.float32) + np.float32(0.0)


def lmhead_verify(hidden_bits, weight_bits, draft_tokens, block_lens, tau, exc_cap, budget,
                  row_offsets=None, raw_gate=False):
    """The verifier on the logit rows of :func:`lmhead_logits`."""
    return verify(lmhead_logits(hidden_bits, weight_bits), draft_tokens, block_lens, tau,
                  exc_cap, budget, row_offsets, raw_gate)
