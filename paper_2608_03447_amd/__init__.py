"""MI355X (gfx950) verifier of Approximate Speculative Decoding.

A thin ctypes binding over ``libasd.so`` (C ABI declared in ``include/asd.h``).
The functions here only marshal torch tensors (device memory) and the current
HIP stream into the C calls; every step of the verifier runs in the library's
HIP kernels.  There is no CPU fallback: if the library is missing or a call
fails, an exception is raised.
"""
import ctypes
import os

import torch

from .build import HASHED_SOURCES, LIBRARY, source_hash

__all__ = ["asd_verify", "asd_verify_static", "asd_verify_ws", "asd_verify_ex", "asd_shard_argmax",
           "asd_verify_partials", "asd_opportunity", "asd_commit", "asd_verify_commit",
           "asd_lmhead_verify", "asd_device_error", "asd_row_splits", "asd_row_pass", "asd_read_probe",
           "asd_mfma_probe", "asd_workspace_bytes",
           "asd_status_string", "asd_version", "asd_release", "AsdError", "ASD_F32", "ASD_BF16",
           "ASD_GATE_RAW", "ASD_DEVERR_NEGATIVE_K", "ASD_DEVERR_ROWS", "ASD_DEVERR_COMMIT",
           "library_path", "library_source_hash", "check_built_from_sources"]

ASD_F32 = 0
ASD_BF16 = 1
ASD_GATE_RAW = 1            # asd_verify_ex flag: gate on r <= g instead of r / q <= g
ASD_DEVERR_NEGATIVE_K = 1   # device error word bits (asd_device_error)
ASD_DEVERR_ROWS = 2
ASD_DEVERR_COMMIT = 4
ASD_ESCRATCH = 6            # status: the call needs more than asd_verify_static's scratch
ASD_STATIC_SCRATCH_BYTES = 4 << 20
_DTYPES = {torch.float32: ASD_F32, torch.bfloat16: ASD_BF16}

_lib = None


class AsdError(RuntimeError):
    def __init__(self, status, where):
        self.status = int(status)
        super().__init__("%s failed: %s" % (where, asd_status_string(status)))


def library_path() -> str:
    return LIBRARY


def library_source_hash(lib) -> str:
    """The source hash a loaded library was built with (last word of asd_version)."""
    return lib.asd_version().decode().split()[-1]


def check_built_from_sources(lib, path=LIBRARY):
    """Raise unless the library was built from the sources beside it (the hash
    embedded by the build equals the hash of the current sources)."""
    if not all(os.path.exists(p) for p in HASHED_SOURCES):
        raise RuntimeError("the sources of %s are missing; cannot check the build" % path)
    built, current = library_source_hash(lib), source_hash()
    if built != current:
        raise RuntimeError("%s was built from other sources (built %s, sources %s); run "
                           "__graft_entry__.build() again" % (path, built, current))


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise RuntimeError("libasd.so is not built (%s); run __graft_entry__.build() first"
                           % LIBRARY)
    lib = ctypes.CDLL(LIBRARY)
    lib.asd_version.argtypes = []
    lib.asd_version.restype = ctypes.c_char_p
    check_built_from_sources(lib, LIBRARY)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    common = [vp, ctypes.c_int, i64, i32, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.asd_verify.argtypes = common
    lib.asd_verify.restype = ctypes.c_int
    lib.asd_verify_static.argtypes = common
    lib.asd_verify_static.restype = ctypes.c_int
    lib.asd_verify_ws.argtypes = common + [vp, sz]
    lib.asd_verify_ws.restype = ctypes.c_int
    lib.asd_verify_ex.argtypes = common[:-1] + [ctypes.c_uint32, vp, vp, sz]
    lib.asd_verify_ex.restype = ctypes.c_int
    lib.asd_device_error.argtypes = [vp, i32, vp]
    lib.asd_device_error.restype = ctypes.c_int
    lib.asd_mfma_probe.argtypes = [vp, i64, i64, i64, vp, vp]
    lib.asd_mfma_probe.restype = ctypes.c_int
    lib.asd_row_splits.argtypes = [ctypes.c_int, i64, i64]
    lib.asd_row_splits.restype = i32
    lib.asd_row_pass.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, vp]
    lib.asd_row_pass.restype = ctypes.c_int
    lib.asd_read_probe.argtypes = [vp, i64, i64, vp, vp]
    lib.asd_read_probe.restype = ctypes.c_int
    lib.asd_shard_argmax.argtypes = [vp, ctypes.c_int, i64, i64, i64, i64, vp, vp, vp]
    lib.asd_shard_argmax.restype = ctypes.c_int
    lib.asd_verify_partials.argtypes = [vp, i32, i64, i64, i32, i64, vp, vp, vp, vp, vp, vp, vp,
                                         vp, vp, vp, vp]
    lib.asd_verify_partials.restype = ctypes.c_int
    lib.asd_opportunity.argtypes = [vp, vp, vp, i64, i32, i64, vp, vp, vp, i32, vp, i32, vp, vp,
                                     vp]
    lib.asd_opportunity.restype = ctypes.c_int
    lib.asd_lmhead_verify.argtypes = [vp, vp, i64, i64, i32, i64, vp, vp, vp, vp, vp, vp, vp, vp,
                                      vp, vp, vp]
    lib.asd_lmhead_verify.restype = ctypes.c_int
    lib.asd_commit.argtypes = [vp, vp, vp, i32, i64, vp, vp, vp, i64, vp, vp, vp]
    lib.asd_verify_commit.argtypes = common[:-1] + [vp, i64, vp, vp, vp, vp, sz]
    lib.asd_verify_commit.restype = ctypes.c_int
    lib.asd_commit.restype = ctypes.c_int
    lib.asd_workspace_bytes.argtypes = [ctypes.c_int, i64, i32, i64]
    lib.asd_workspace_bytes.restype = sz
    lib.asd_status_string.argtypes = [ctypes.c_int]
    lib.asd_status_string.restype = ctypes.c_char_p
    lib.asd_version.argtypes = []
    lib.asd_version.restype = ctypes.c_char_p
    lib.asd_release.argtypes = []
    lib.asd_release.restype = ctypes.c_int
    _lib = lib
    return lib


def asd_status_string(status) -> str:
    return _load().asd_status_string(int(status)).decode()


def asd_version() -> str:
    return _load().asd_version().decode()


def asd_release() -> None:
    st = _load().asd_release()
    if st != 0:
        raise AsdError(st, "asd_release")


def asd_workspace_bytes(dtype, vocab, num_requests, total_rows) -> int:
    code = _DTYPES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return int(_load().asd_workspace_bytes(code, int(vocab), int(num_requests), int(total_rows)))


def _per_request(value, n, dtype, device, name):
    if isinstance(value, torch.Tensor):
        if value.dtype != dtype or value.device != device or value.shape != (n,):
            raise ValueError("%s must be a %s tensor of shape (%d,) on %s" % (name, dtype, n, device))
        return value.contiguous()
    return torch.full((n,), value, dtype=dtype, device=device)


def _check_vector(t, n, dtype, device, name):
    """An optional vector argument: None, or a contiguous tensor of this dtype
    and shape (n,) on `device` (the library reads it through a plain pointer)."""
    if t is not None and (t.dtype != dtype or t.shape != (n,) or t.device != device
                          or not t.is_contiguous()):
        raise ValueError("%s must be a contiguous %s tensor of shape (%d,) on %s"
                         % (name, dtype, n, device))


def _check_logits(logits):
    if logits.dim() != 2 or logits.dtype not in _DTYPES or not logits.is_cuda:
        raise ValueError("logits must be a 2-D float32 or bfloat16 tensor on a GPU")
    if not logits.is_contiguous():
        raise ValueError("logits must be contiguous (row-major, dense)")


def _marshal(dev, rows, draft_tokens, block_lens, tau, exc_cap, budget, row_offsets,
             out_accept_len, out_next_token, out_argmax, out_regret):
    """Checks and pointers of the arguments shared by every verifying call:
    [num_requests, total_rows, draft, lens, offsets, tau, cap, budget, accept,
    next, argmax, regret, stream]."""
    if block_lens.dtype != torch.int32 or block_lens.dim() != 1 or block_lens.device != dev:
        raise ValueError("block_lens must be an int32 vector on the logits' device")
    n = block_lens.shape[0]
    if draft_tokens.dtype != torch.int32 or draft_tokens.shape != (rows,) or draft_tokens.device != dev:
        raise ValueError("draft_tokens must be int32 of shape (%d,) on %s" % (rows, dev))
    if budget.dtype != torch.float32 or budget.shape != (n, 2) or budget.device != dev \
            or not budget.is_contiguous():
        raise ValueError("budget must be a contiguous float32 (%d, 2) tensor on %s" % (n, dev))
    _check_vector(row_offsets, n, torch.int64, dev, "row_offsets")
    tau = _per_request(tau, n, torch.float32, dev, "tau")
    exc_cap = _per_request(exc_cap, n, torch.int32, dev, "exc_cap")
    block_lens = block_lens.contiguous()
    draft_tokens = draft_tokens.contiguous()
    if out_accept_len is None:
        out_accept_len = torch.empty(n, dtype=torch.int32, device=dev)
    if out_next_token is None:
        out_next_token = torch.empty(n, dtype=torch.int32, device=dev)
    for t, name, shape, dt in ((out_accept_len, "out_accept_len", (n,), torch.int32),
                               (out_next_token, "out_next_token", (n,), torch.int32),
                               (out_argmax, "out_argmax", (rows,), torch.int32),
                               (out_regret, "out_regret", (rows,), torch.float32)):
        if t is not None and (t.dtype != dt or t.shape != shape or t.device != dev
                              or not t.is_contiguous()):
            raise ValueError("%s must be a contiguous %s tensor of shape %s on %s"
                             % (name, dt, shape, dev))

    def p(t):
        return None if t is None else ctypes.c_void_p(t.data_ptr())

    stream = torch.cuda.current_stream(dev).cuda_stream
    args = [n, rows, p(draft_tokens), p(block_lens), p(row_offsets), p(tau), p(exc_cap),
            p(budget), p(out_accept_len), p(out_next_token), p(out_argmax), p(out_regret),
            ctypes.c_void_p(stream)]
    keep = (tau, exc_cap, block_lens, draft_tokens)
    return args, out_accept_len, out_next_token, keep


def asd_verify(logits, draft_tokens, block_lens, tau, exc_cap, budget, *, row_offsets=None,
               out_accept_len=None, out_next_token=None, out_argmax=None, out_regret=None):
    """Verify a batch of draft blocks on the GPU (``asd_verify`` of ``include/asd.h``).

    logits        [total_rows, V] float32 or bfloat16, contiguous, on a GPU
    draft_tokens  int32 [total_rows]
    block_lens    int32 [num_requests] (K_i)
    tau           float or float32 [num_requests]: local gate g of each request
    exc_cap       int or int32 [num_requests]: block cap M of each request
    budget        float32 [num_requests, 2] = (B, s); s is updated in place
    Returns ``(accept_len, next_token)`` int32 tensors; the work is enqueued on
    the current stream of the logits' device.
    """
    _check_logits(logits)
    with torch.cuda.device(logits.device):
        args, acc, nxt, keep = _marshal(logits.device, logits.shape[0], draft_tokens, block_lens,
                                        tau, exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        st = _load().asd_verify(ctypes.c_void_p(logits.data_ptr()), _DTYPES[logits.dtype],
                                logits.shape[1], *args)
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify")
    return acc, nxt


def asd_verify_static(logits, draft_tokens, block_lens, tau, exc_cap, budget, *,
                      row_offsets=None, out_accept_len=None, out_next_token=None,
                      out_argmax=None, out_regret=None):
    """``asd_verify`` with its workspace in the library's fixed per-device scratch
    (``asd_verify_static`` of ``include/asd.h``): the call allocates nothing.
    Calls that may overlap on one device race on that scratch."""
    _check_logits(logits)
    with torch.cuda.device(logits.device):
        args, acc, nxt, keep = _marshal(logits.device, logits.shape[0], draft_tokens, block_lens,
                                        tau, exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        st = _load().asd_verify_static(ctypes.c_void_p(logits.data_ptr()),
                                       _DTYPES[logits.dtype], logits.shape[1], *args)
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify_static")
    return acc, nxt


def asd_verify_ws(logits, draft_tokens, block_lens, tau, exc_cap, budget, workspace, *,
                  row_offsets=None, out_accept_len=None, out_next_token=None, out_argmax=None,
                  out_regret=None):
    """``asd_verify`` with a caller-provided workspace (a uint8 tensor, any content)."""
    if workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor")
    _check_logits(logits)
    with torch.cuda.device(logits.device):
        args, acc, nxt, keep = _marshal(logits.device, logits.shape[0], draft_tokens, block_lens,
                                        tau, exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        st = _load().asd_verify_ws(ctypes.c_void_p(logits.data_ptr()), _DTYPES[logits.dtype],
                                   logits.shape[1], *args,
                                   ctypes.c_void_p(workspace.data_ptr()), workspace.numel())
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify_ws")
    return acc, nxt


def asd_verify_ex(logits, draft_tokens, block_lens, tau, exc_cap, budget, *, flags=0,
                  workspace=None, row_offsets=None, out_accept_len=None, out_next_token=None,
                  out_argmax=None, out_regret=None):
    """``asd_verify`` with flags (``ASD_GATE_RAW``) and an optional workspace
    (``asd_verify_ex`` of ``include/asd.h``)."""
    if workspace is not None and (workspace.dtype != torch.uint8 or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor")
    _check_logits(logits)
    with torch.cuda.device(logits.device):
        args, acc, nxt, keep = _marshal(logits.device, logits.shape[0], draft_tokens, block_lens,
                                        tau, exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        ws = None if workspace is None else ctypes.c_void_p(workspace.data_ptr())
        ws_bytes = 0 if workspace is None else workspace.numel()
        st = _load().asd_verify_ex(ctypes.c_void_p(logits.data_ptr()), _DTYPES[logits.dtype],
                                   logits.shape[1], *args[:-1], int(flags), args[-1], ws,
                                   ws_bytes)
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify_ex")
    return acc, nxt


def asd_device_error(clear=False, device=None) -> int:
    """The sticky error word of a device (``asd_device_error``): ``ASD_DEVERR_*``
    bits, read once the current stream's work has completed; ``clear`` resets it."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None \
        else torch.device(device)
    word = ctypes.c_uint32(0)
    with torch.cuda.device(dev):
        stream = torch.cuda.current_stream(dev).cuda_stream
        st = _load().asd_device_error(ctypes.byref(word), 1 if clear else 0,
                                      ctypes.c_void_p(stream))
    if st != 0:
        raise AsdError(st, "asd_device_error")
    return int(word.value)


def asd_row_splits(dtype, vocab, total_rows):
    """Column tiles per row of asd_verify's row pass on the current device
    (``asd_row_splits``); ``dtype`` is torch.float32 or torch.bfloat16."""
    if dtype not in _DTYPES:
        raise ValueError("dtype must be torch.float32 or torch.bfloat16")
    return int(_load().asd_row_splits(_DTYPES[dtype], int(vocab), int(total_rows)))


def asd_row_pass(logits, draft_tokens, out_partials=None):
    """asd_verify's row pass alone, on the call's own tile grid (``asd_row_pass``).

    logits        [total_rows, V] float32 or bfloat16, contiguous, on a GPU
    draft_tokens  int32 [total_rows]
    Returns the partials, an int32 tensor [total_rows, S, 4] (16 opaque bytes
    per tile, S = asd_row_splits)."""
    if logits.dim() != 2 or logits.dtype not in _DTYPES or not logits.is_cuda:
        raise ValueError("logits must be a 2-D float32 or bfloat16 tensor on a GPU")
    if not logits.is_contiguous():
        raise ValueError("logits must be contiguous (row-major, dense)")
    dev = logits.device
    rows, vocab = logits.shape
    if draft_tokens.dtype != torch.int32 or draft_tokens.shape != (rows,) \
            or draft_tokens.device != dev:
        raise ValueError("draft_tokens must be int32 of shape (%d,) on %s" % (rows, dev))
    with torch.cuda.device(dev):
        splits = asd_row_splits(logits.dtype, vocab, rows)
        if splits < 1:
            raise ValueError("no row pass for %d rows of %d columns" % (rows, vocab))
        if out_partials is None:
            out_partials = torch.empty((rows, splits, 4), dtype=torch.int32, device=dev)
        if out_partials.dtype != torch.int32 or out_partials.shape != (rows, splits, 4) \
                or not out_partials.is_contiguous() or out_partials.device != dev:
            raise ValueError("out_partials must be a contiguous int32 (%d, %d, 4) tensor on %s"
                             % (rows, splits, dev))
        draft_tokens = draft_tokens.contiguous()
        stream = torch.cuda.current_stream(dev).cuda_stream
        st = _load().asd_row_pass(ctypes.c_void_p(logits.data_ptr()), _DTYPES[logits.dtype],
                                  vocab, rows, ctypes.c_void_p(draft_tokens.data_ptr()),
                                  ctypes.c_void_p(out_partials.data_ptr()), ctypes.c_void_p(stream))
    if st != 0:
        raise AsdError(st, "asd_row_pass")
    return out_partials


def asd_read_probe(buf, rows, row_bytes, out_word):
    """Stream ``rows`` x ``row_bytes`` of ``buf`` (a contiguous GPU tensor) with the
    row pass's access pattern (``asd_read_probe``); ``out_word`` is a uint32-sized
    int32 tensor on the same device."""
    if (not buf.is_cuda or not buf.is_contiguous()
            or buf.numel() * buf.element_size() < rows * row_bytes):
        raise ValueError("buf must be a contiguous GPU tensor of at least rows * row_bytes bytes")
    if out_word.dtype != torch.int32 or out_word.numel() < 1 or out_word.device != buf.device:
        raise ValueError("out_word must be an int32 tensor on the buffer's device")
    with torch.cuda.device(buf.device):
        stream = torch.cuda.current_stream(buf.device).cuda_stream
        st = _load().asd_read_probe(ctypes.c_void_p(buf.data_ptr()), int(rows), int(row_bytes),
                                    ctypes.c_void_p(out_word.data_ptr()), ctypes.c_void_p(stream))
    if st != 0:
        raise AsdError(st, "asd_read_probe")


def asd_mfma_probe(operands, workgroups, steps, out):
    """The LM-head kernel's matrix-core work without memory traffic
    (``asd_mfma_probe``): ``operands`` a contiguous bfloat16 GPU tensor of at
    least 48 values, ``out`` an int32 tensor of ``workgroups`` entries on the
    same device (binary32 bits of each workgroup's thread-0 accumulator sum)."""
    if operands.dtype != torch.bfloat16 or not operands.is_cuda or not operands.is_contiguous():
        raise ValueError("operands must be a contiguous bfloat16 GPU tensor")
    if out.dtype != torch.int32 or out.numel() < workgroups or out.device != operands.device:
        raise ValueError("out must be an int32 tensor of at least `workgroups` entries")
    with torch.cuda.device(operands.device):
        stream = torch.cuda.current_stream(operands.device).cuda_stream
        st = _load().asd_mfma_probe(ctypes.c_void_p(operands.data_ptr()), operands.numel() // 8,
                                    int(workgroups), int(steps), ctypes.c_void_p(out.data_ptr()),
                                    ctypes.c_void_p(stream))
    if st != 0:
        raise AsdError(st, "asd_mfma_probe")


def asd_shard_argmax(shard_logits, vocab_offset, vocab, draft_tokens, out_partials=None):
    """Row pass of one vocabulary shard (``asd_shard_argmax`` of ``include/asd.h``).

    shard_logits  [total_rows, W] float32 or bfloat16: columns
                  [vocab_offset, vocab_offset + W) of the full vocabulary
    draft_tokens  int32 [total_rows] (global ids)
    Returns the partials, an int32 tensor [total_rows, 4] (16 opaque bytes per row).
    """
    if shard_logits.dim() != 2 or shard_logits.dtype not in _DTYPES or not shard_logits.is_cuda:
        raise ValueError("shard_logits must be a 2-D float32 or bfloat16 tensor on a GPU")
    if not shard_logits.is_contiguous():
        raise ValueError("shard_logits must be contiguous (row-major, dense)")
    dev = shard_logits.device
    rows, width = shard_logits.shape
    if draft_tokens.dtype != torch.int32 or draft_tokens.shape != (rows,) \
            or draft_tokens.device != dev:
        raise ValueError("draft_tokens must be int32 of shape (%d,) on %s" % (rows, dev))
    if out_partials is None:
        out_partials = torch.empty((rows, 4), dtype=torch.int32, device=dev)
    if out_partials.dtype != torch.int32 or out_partials.shape != (rows, 4) \
            or not out_partials.is_contiguous() or out_partials.device != dev:
        raise ValueError("out_partials must be a contiguous int32 (%d, 4) tensor on %s" % (rows, dev))
    draft_tokens = draft_tokens.contiguous()
    with torch.cuda.device(dev):
        stream = torch.cuda.current_stream(dev).cuda_stream
        st = _load().asd_shard_argmax(ctypes.c_void_p(shard_logits.data_ptr()),
                                      _DTYPES[shard_logits.dtype], width, int(vocab_offset),
                                      int(vocab), rows, ctypes.c_void_p(draft_tokens.data_ptr()),
                                      ctypes.c_void_p(out_partials.data_ptr()),
                                      ctypes.c_void_p(stream))
    if st != 0:
        raise AsdError(st, "asd_shard_argmax")
    return out_partials


def asd_verify_partials(partials, shard_vocab, vocab, draft_tokens, block_lens, tau, exc_cap,
                        budget, *, row_offsets=None, out_accept_len=None, out_next_token=None,
                        out_argmax=None, out_regret=None):
    """Finish the verification from the partials of all shards
    (``asd_verify_partials`` of ``include/asd.h``).

    partials  int32 [num_shards, total_rows, 4]; shard k holds columns
              [k * shard_vocab, min((k + 1) * shard_vocab, vocab))
    Other arguments as for :func:`asd_verify`.  Returns ``(accept_len, next_token)``.
    """
    if partials.dtype != torch.int32 or partials.dim() != 3 or partials.shape[2] != 4 \
            or not partials.is_contiguous() or not partials.is_cuda:
        raise ValueError("partials must be a contiguous int32 (num_shards, total_rows, 4) GPU tensor")
    dev = partials.device
    shards, rows = partials.shape[0], partials.shape[1]
    with torch.cuda.device(dev):
        args, acc, nxt, keep = _marshal(dev, rows, draft_tokens, block_lens, tau, exc_cap, budget,
                                        row_offsets, out_accept_len, out_next_token,
                                        out_argmax, out_regret)
        st = _load().asd_verify_partials(ctypes.c_void_p(partials.data_ptr()), shards,
                                         int(shard_vocab), int(vocab), *args)
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify_partials")
    return acc, nxt


def asd_opportunity(draft_tokens, row_argmax, row_regret, vocab, block_lens, taus, ps, counts,
                    mismatches, *, row_offsets=None):
    """Accumulate the opportunity statistic of Eq. 4 (``asd_opportunity`` of ``include/asd.h``).

    row_argmax / row_regret  the out_argmax / out_regret of asd_verify on the batch
    taus   float32 [A]; ps int32 [P]
    counts int64 [A, P] and mismatches int64 [1]: uint64 accumulators, added to in place
    """
    dev = draft_tokens.device
    rows = draft_tokens.shape[0]
    for t, name, dt, shape in ((draft_tokens, "draft_tokens", torch.int32, (rows,)),
                               (row_argmax, "row_argmax", torch.int32, (rows,)),
                               (row_regret, "row_regret", torch.float32, (rows,)),
                               (taus, "taus", torch.float32, None),
                               (ps, "ps", torch.int32, None),
                               (mismatches, "mismatches", torch.int64, (1,))):
        if t.dtype != dt or t.device != dev or not t.is_contiguous() or \
                (shape is not None and t.shape != shape):
            raise ValueError("%s must be a contiguous %s tensor%s on %s" % (
                name, dt, "" if shape is None else " of shape %s" % (shape,), dev))
    if block_lens.dtype != torch.int32 or block_lens.device != dev:
        raise ValueError("block_lens must be an int32 tensor on %s" % dev)
    n = block_lens.shape[0]
    if counts.dtype != torch.int64 or counts.shape != (taus.shape[0], ps.shape[0]) \
            or not counts.is_contiguous() or counts.device != dev:
        raise ValueError("counts must be a contiguous int64 (%d, %d) tensor on %s"
                         % (taus.shape[0], ps.shape[0], dev))
    _check_vector(row_offsets, n, torch.int64, dev, "row_offsets")
    block_lens = block_lens.contiguous()

    def p(t):
        return None if t is None else ctypes.c_void_p(t.data_ptr())

    with torch.cuda.device(dev):
        st = _load().asd_opportunity(p(draft_tokens), p(row_argmax), p(row_regret), int(vocab), n,
                                     rows, p(block_lens), p(row_offsets), p(taus),
                                     taus.shape[0], p(ps), ps.shape[0], p(counts),
                                     p(mismatches),
                                     ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    if st != 0:
        raise AsdError(st, "asd_opportunity")


def asd_commit(draft_tokens, block_lens, accept_len, next_token, tokens, seq_len, *,
               row_offsets=None, out_committed=None):
    """Commit the emitted tokens (``asd_commit`` of ``include/asd.h``).

    tokens   int32 [num_requests, capacity]; seq_len int64 [num_requests], both updated in place
    """
    dev = draft_tokens.device
    n = block_lens.shape[0]
    for t, name, dt, shape in ((draft_tokens, "draft_tokens", torch.int32, None),
                               (block_lens, "block_lens", torch.int32, (n,)),
                               (accept_len, "accept_len", torch.int32, (n,)),
                               (next_token, "next_token", torch.int32, (n,)),
                               (seq_len, "seq_len", torch.int64, (n,))):
        if t.dtype != dt or t.device != dev or not t.is_contiguous() or \
                (shape is not None and t.shape != shape):
            raise ValueError("%s must be a contiguous %s tensor%s on %s" % (
                name, dt, "" if shape is None else " of shape %s" % (shape,), dev))
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or tokens.shape[0] != n \
            or not tokens.is_contiguous() or tokens.device != dev:
        raise ValueError("tokens must be a contiguous int32 (%d, capacity) tensor on %s" % (n, dev))
    _check_vector(out_committed, n, torch.int32, dev, "out_committed")
    _check_vector(row_offsets, n, torch.int64, dev, "row_offsets")

    def p(t):
        return None if t is None else ctypes.c_void_p(t.data_ptr())

    with torch.cuda.device(dev):
        st = _load().asd_commit(p(draft_tokens), p(block_lens), p(row_offsets), n,
                                draft_tokens.shape[0], p(accept_len), p(next_token), p(tokens),
                                tokens.shape[1], p(seq_len), p(out_committed),
                                ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    if st != 0:
        raise AsdError(st, "asd_commit")


def asd_verify_commit(logits, draft_tokens, block_lens, tau, exc_cap, budget, tokens, seq_len, *,
                      row_offsets=None, out_accept_len=None, out_next_token=None,
                      out_argmax=None, out_regret=None, out_committed=None, workspace=None):
    """Verification and commit in one pass (``asd_verify_commit`` of ``include/asd.h``).

    tokens   int32 [num_requests, capacity]; seq_len int64 [num_requests], both updated in
             place as by :func:`asd_commit`.  workspace: None (library workspace) or a uint8
             tensor as for :func:`asd_verify_ws`.  Returns (accept_len, next_token).
    """
    _check_logits(logits)
    dev = logits.device
    n = block_lens.shape[0]
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or tokens.shape[0] != n \
            or not tokens.is_contiguous() or tokens.device != dev:
        raise ValueError("tokens must be a contiguous int32 (%d, capacity) tensor on %s" % (n, dev))
    if seq_len.dtype != torch.int64 or seq_len.shape != (n,) or not seq_len.is_contiguous() \
            or seq_len.device != dev:
        raise ValueError("seq_len must be a contiguous int64 tensor of shape (%d,) on %s" % (n, dev))
    _check_vector(out_committed, n, torch.int32, dev, "out_committed")
    if workspace is not None and (workspace.dtype != torch.uint8 or not workspace.is_contiguous()
                                  or workspace.device != dev):
        raise ValueError("workspace must be a contiguous uint8 tensor on %s" % dev)
    with torch.cuda.device(dev):
        args, acc, nxt, keep = _marshal(dev, logits.shape[0], draft_tokens, block_lens, tau,
                                        exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        p = (lambda t: None if t is None else ctypes.c_void_p(t.data_ptr()))
        st = _load().asd_verify_commit(
            ctypes.c_void_p(logits.data_ptr()), _DTYPES[logits.dtype], logits.shape[1],
            *args[:-1], p(tokens), tokens.shape[1], p(seq_len), p(out_committed), args[-1],
            p(workspace), 0 if workspace is None else workspace.numel())
    del keep
    if st != 0:
        raise AsdError(st, "asd_verify_commit")
    return acc, nxt


def asd_lmhead_verify(hidden, weight, draft_tokens, block_lens, tau, exc_cap, budget, *,
                      row_offsets=None, out_accept_len=None, out_next_token=None,
                      out_argmax=None, out_regret=None):
    """LM-head-fused verification (``asd_lmhead_verify`` of ``include/asd.h``).

    hidden  bf16 [total_rows, d]; weight bf16 [V, d]; other arguments as for :func:`asd_verify`.
    """
    for t, name in ((hidden, "hidden"), (weight, "weight")):
        if t.dim() != 2 or t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("%s must be a contiguous 2-D bfloat16 GPU tensor" % name)
    if hidden.shape[1] != weight.shape[1] or hidden.device != weight.device:
        raise ValueError("hidden and weight must share d and device")
    dev = hidden.device
    with torch.cuda.device(dev):
        args, acc, nxt, keep = _marshal(dev, hidden.shape[0], draft_tokens, block_lens, tau,
                                        exc_cap, budget, row_offsets, out_accept_len,
                                        out_next_token, out_argmax, out_regret)
        st = _load().asd_lmhead_verify(ctypes.c_void_p(hidden.data_ptr()),
                                       ctypes.c_void_p(weight.data_ptr()), hidden.shape[1],
                                       weight.shape[0], *args)
    del keep
    if st != 0:
        raise AsdError(st, "asd_lmhead_verify")
    return acc, nxt
