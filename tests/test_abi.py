"""The C-ABI library: it loads, exports every function include/asd.h declares,
and rejects invalid host-checkable arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import paper_2608_03447_amd as asd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "asd.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(asd_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("asd_verify", "asd_verify_ws", "asd_workspace_bytes", "asd_status_string",
              "asd_version", "asd_release"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(asd.library_path())
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    assert asd.asd_status_string(0) == "ASD_OK"
    assert "EINVAL" in asd.asd_status_string(1)
    assert "unknown" in asd.asd_status_string(99)
    assert "gfx950" in asd.asd_version()


def _call(entry="asd_verify", **kw):
    lib = asd._load()
    a = dict(logits=0x1000, dtype=1, vocab=100, nreq=1, rows=2, draft=0x2000, lens=0x3000,
             offs=None, tau=0x4000, cap=0x5000, budget=0x6000, acc=0x7000, nxt=0x8000,
             amax=None, regret=None, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return getattr(lib, entry)(vp(a["logits"]), a["dtype"], a["vocab"], a["nreq"], a["rows"],
                          vp(a["draft"]), vp(a["lens"]), vp(a["offs"]), vp(a["tau"]),
                          vp(a["cap"]), vp(a["budget"]), vp(a["acc"]), vp(a["nxt"]),
                          vp(a["amax"]), vp(a["regret"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 2),
    (dict(vocab=0), 1),
    (dict(vocab=1 << 30), 1),
    (dict(nreq=-1), 1),
    (dict(nreq=3, rows=2), 1),
    (dict(rows=1 << 31), 1),
    (dict(logits=None), 1),
    (dict(draft=None), 1),
    (dict(lens=None), 1),
    (dict(tau=None), 1),
    (dict(cap=None), 1),
    (dict(budget=None), 1),
    (dict(acc=None), 1),
    (dict(nxt=None), 1),
    (dict(logits=0x1001), 1),                  # not a multiple of the bf16 size
    (dict(dtype=0, logits=0x1002), 1),         # not a multiple of the f32 size
])
@pytest.mark.parametrize("entry", ["asd_verify", "asd_verify_static"])
def test_invalid_arguments_are_rejected_without_launch(kw, status, entry):
    assert _call(entry, **kw) == status


@pytest.mark.parametrize("entry", ["asd_verify", "asd_verify_static"])
def test_empty_batch_is_a_no_op(entry):
    assert _call(entry, nreq=0, rows=0, logits=None, draft=None) == 0


def test_static_scratch_size_and_status_string():
    assert asd.ASD_STATIC_SCRATCH_BYTES == 4 << 20
    assert "ESCRATCH" in asd.asd_status_string(asd.ASD_ESCRATCH)


def test_workspace_bytes_rejects_invalid_shapes():
    lib = asd._load()
    assert lib.asd_workspace_bytes(9, 100, 1, 2) == 0
    assert lib.asd_workspace_bytes(1, 0, 1, 2) == 0
    assert lib.asd_workspace_bytes(1, 100, 3, 2) == 0


def test_package_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(asd, "_lib", None)
    monkeypatch.setattr(asd, "LIBRARY", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        asd._load()


def _shard(**kw):
    lib = asd._load()
    a = dict(logits=0x1000, dtype=1, width=100, offset=0, vocab=100, rows=2, draft=0x2000,
             out=0x3000, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_shard_argmax(vp(a["logits"]), a["dtype"], a["width"], a["offset"], a["vocab"],
                                a["rows"], vp(a["draft"]), vp(a["out"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2),
    (dict(width=0), 1),
    (dict(offset=-1), 1),
    (dict(offset=1), 1),                      # offset + width > vocab
    (dict(vocab=1 << 30, width=10), 1),
    (dict(rows=0), 1),
    (dict(rows=1 << 31), 1),
    (dict(logits=None), 1),
    (dict(draft=None), 1),
    (dict(out=None), 1),
    (dict(out=0x3008), 1),                    # partials must be 16-byte aligned
    (dict(logits=0x1001), 1),
])
def test_shard_argmax_rejects_invalid_arguments(kw, status):
    assert _shard(**kw) == status


def _vp(**kw):
    lib = asd._load()
    a = dict(parts=0x1000, shards=2, width=50, vocab=100, nreq=1, rows=2, draft=0x2000,
             lens=0x3000, offs=None, tau=0x4000, cap=0x5000, budget=0x6000, acc=0x7000,
             nxt=0x8000, amax=None, regret=None, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_verify_partials(vp(a["parts"]), a["shards"], a["width"], a["vocab"], a["nreq"],
                                   a["rows"], vp(a["draft"]), vp(a["lens"]), vp(a["offs"]),
                                   vp(a["tau"]), vp(a["cap"]), vp(a["budget"]), vp(a["acc"]),
                                   vp(a["nxt"]), vp(a["amax"]), vp(a["regret"]),
                                   vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(shards=0), 1),
    (dict(shards=4097), 1),
    (dict(width=0), 1),
    (dict(width=30), 1),                      # 2 x 30 < 100: columns left over
    (dict(width=100), 1),                     # shard 2 would be empty
    (dict(parts=None), 1),
    (dict(parts=0x1004), 1),
    (dict(lens=None), 1),
    (dict(nreq=3, rows=2), 1),
])
def test_verify_partials_rejects_invalid_arguments(kw, status):
    assert _vp(**kw) == status


def test_verify_partials_empty_batch_is_a_no_op():
    assert _vp(nreq=0, rows=0, parts=None, draft=None) == 0


def _opp(**kw):
    lib = asd._load()
    a = dict(draft=0x1000, amax=0x2000, reg=0x3000, vocab=100, nreq=1, rows=2, lens=0x4000,
             offs=None, taus=0x5000, ntau=2, ps=0x6000, nps=3, counts=0x7000, mism=0x8000,
             stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_opportunity(vp(a["draft"]), vp(a["amax"]), vp(a["reg"]), a["vocab"], a["nreq"],
                               a["rows"], vp(a["lens"]), vp(a["offs"]), vp(a["taus"]), a["ntau"],
                               vp(a["ps"]), a["nps"], vp(a["counts"]), vp(a["mism"]),
                               vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(vocab=0), 1), (dict(ntau=0), 1), (dict(nps=0), 1), (dict(ntau=33, nps=32), 1),
    (dict(nreq=3, rows=2), 1), (dict(draft=None), 1), (dict(amax=None), 1), (dict(reg=None), 1),
    (dict(counts=None), 1), (dict(mism=None), 1), (dict(taus=None), 1), (dict(ps=None), 1),
])
def test_opportunity_rejects_invalid_arguments(kw, status):
    assert _opp(**kw) == status


def test_opportunity_empty_batch_is_a_no_op():
    assert _opp(nreq=0, rows=0, draft=None) == 0


def _commit(**kw):
    lib = asd._load()
    a = dict(draft=0x1000, lens=0x2000, offs=None, nreq=1, rows=2, acc=0x3000, nxt=0x4000,
             tok=0x5000, cap=8, sl=0x6000, done=None, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_commit(vp(a["draft"]), vp(a["lens"]), vp(a["offs"]), a["nreq"], a["rows"],
                          vp(a["acc"]), vp(a["nxt"]), vp(a["tok"]), a["cap"], vp(a["sl"]),
                          vp(a["done"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(cap=0), 1), (dict(nreq=-1), 1), (dict(nreq=3, rows=2), 1), (dict(draft=None), 1),
    (dict(lens=None), 1), (dict(acc=None), 1), (dict(nxt=None), 1), (dict(tok=None), 1),
    (dict(sl=None), 1), (dict(cap=1 << 62, nreq=4, rows=4), 1),
])
def test_commit_rejects_invalid_arguments(kw, status):
    assert _commit(**kw) == status


def _lmhead(**kw):
    lib = asd._load()
    a = dict(hidden=0x1000, weight=0x2000, d=256, vocab=100, nreq=1, rows=2, draft=0x3000,
             lens=0x4000, offs=None, tau=0x5000, cap=0x6000, budget=0x7000, acc=0x8000,
             nxt=0x9000, amax=None, reg=None, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_lmhead_verify(vp(a["hidden"]), vp(a["weight"]), a["d"], a["vocab"], a["nreq"],
                                 a["rows"], vp(a["draft"]), vp(a["lens"]), vp(a["offs"]),
                                 vp(a["tau"]), vp(a["cap"]), vp(a["budget"]), vp(a["acc"]),
                                 vp(a["nxt"]), vp(a["amax"]), vp(a["reg"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(d=64), 1), (dict(d=192), 1), (dict(d=0), 1), (dict(d=(1 << 20) + 128), 1),
    (dict(weight=None), 1), (dict(hidden=None), 1), (dict(hidden=0x1008), 1),
    (dict(weight=0x2008), 1), (dict(vocab=0), 1), (dict(nreq=3, rows=2), 1),
    (dict(draft=None), 1), (dict(budget=None), 1),
])
def test_lmhead_rejects_invalid_arguments(kw, status):
    assert _lmhead(**kw) == status


def test_lmhead_empty_batch_is_a_no_op():
    assert _lmhead(nreq=0, rows=0) == 0


def _verify_commit(**kw):
    lib = asd._load()
    a = dict(logits=0x1000, dtype=1, vocab=100, nreq=1, rows=2, draft=0x3000, lens=0x4000,
             offs=None, tau=0x5000, cap=0x6000, budget=0x7000, acc=0x8000, nxt=0x9000,
             amax=None, reg=None, tok=0xa000, capacity=8, sl=0xb000, done=None, stream=None,
             ws=None, ws_bytes=0)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_verify_commit(vp(a["logits"]), a["dtype"], a["vocab"], a["nreq"], a["rows"],
                                 vp(a["draft"]), vp(a["lens"]), vp(a["offs"]), vp(a["tau"]),
                                 vp(a["cap"]), vp(a["budget"]), vp(a["acc"]), vp(a["nxt"]),
                                 vp(a["amax"]), vp(a["reg"]), vp(a["tok"]), a["capacity"],
                                 vp(a["sl"]), vp(a["done"]), vp(a["stream"]), vp(a["ws"]),
                                 a["ws_bytes"])


@pytest.mark.parametrize("kw,status", [
    (dict(capacity=0), 1), (dict(tok=None), 1), (dict(sl=None), 1),
    (dict(capacity=1 << 62, nreq=4, rows=4), 1), (dict(ws=0xc010, ws_bytes=1 << 20), 1),
    (dict(logits=None), 1), (dict(dtype=5), 2), (dict(vocab=0), 1), (dict(nreq=3, rows=2), 1),
    (dict(draft=None), 1), (dict(budget=None), 1), (dict(logits=0x1001), 1),
])
def test_verify_commit_rejects_invalid_arguments(kw, status):
    assert _verify_commit(**kw) == status


def test_verify_commit_empty_batch_is_a_no_op():
    assert _verify_commit(nreq=0, rows=0) == 0


@pytest.mark.parametrize("lang", ["c", "c++"])
def test_header_compiles_cleanly_as_c_and_cpp(tmp_path, lang):
    """include/asd.h is a plain C header: it compiles as C99 and C++17 with
    every warning an error, and a call through it type-checks."""
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    src = tmp_path / ("use.c" if lang == "c" else "use.cpp")
    src.write_text(
        '#include "asd.h"\n'
        "asd_status use(const void *l, const int32_t *d, const int32_t *k, const float *t,\n"
        "               const int32_t *m, asd_budget *b, int32_t *a, int32_t *x, void *s) {\n"
        "    return asd_verify(l, ASD_BF16, 100, 1, 2, d, k, 0, t, m, b, a, x, 0, 0, s);\n"
        "}\n")
    std = "-std=c99" if lang == "c" else "-std=c++17"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    r = subprocess.run([cc, std, "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", inc, "-c",
                        str(src), "-o", str(tmp_path / "use.o")], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _call_ex(flags, ws=None, ws_bytes=0, **kw):
    lib = asd._load()
    a = dict(logits=0x1000, dtype=1, vocab=100, nreq=1, rows=2, draft=0x2000, lens=0x3000,
             offs=None, tau=0x4000, cap=0x5000, budget=0x6000, acc=0x7000, nxt=0x8000,
             amax=None, regret=None, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_verify_ex(vp(a["logits"]), a["dtype"], a["vocab"], a["nreq"], a["rows"],
                             vp(a["draft"]), vp(a["lens"]), vp(a["offs"]), vp(a["tau"]),
                             vp(a["cap"]), vp(a["budget"]), vp(a["acc"]), vp(a["nxt"]),
                             vp(a["amax"]), vp(a["regret"]), flags, vp(a["stream"]), vp(ws),
                             ws_bytes)


@pytest.mark.parametrize("flags", [2, 4, 0x80000000, 0xFFFFFFFF, 3])
def test_verify_ex_rejects_unknown_flags(flags):
    assert _call_ex(flags) == 1


def test_verify_ex_checks_arguments_like_verify():
    assert _call_ex(0, logits=None) == 1
    assert _call_ex(1, dtype=5) == 2
    assert _call_ex(1, nreq=0, rows=0, logits=None, draft=None) == 0     # empty: no-op
    assert _call_ex(0, ws=0x10010, ws_bytes=1 << 20) == 1                # misaligned workspace


def test_device_error_needs_an_output():
    lib = asd._load()
    assert lib.asd_device_error(None, 0, None) == 1
    assert asd.ASD_GATE_RAW == 1
    assert (asd.ASD_DEVERR_NEGATIVE_K, asd.ASD_DEVERR_ROWS, asd.ASD_DEVERR_COMMIT) == (1, 2, 4)


@pytest.mark.parametrize("args", [
    (None, 1, 16, 0x2000), (0x1008, 1, 16, 0x2000), (0x1000, 0, 16, 0x2000),
    (0x1000, 1 << 31, 16, 0x2000), (0x1000, 1, 8, 0x2000), (0x1000, 1, 24, 0x2000),
    (0x1000, 1, 16, None), (0x1000, 1 << 30, 1 << 62, 0x2000),
])
def test_read_probe_rejects_invalid_arguments(args):
    lib = asd._load()
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    buf, rows, row_bytes, out = args
    assert lib.asd_read_probe(vp(buf), rows, row_bytes, vp(out), None) == 1


def test_binding_rejects_strided_or_misplaced_vectors():
    """The binding passes plain pointers, so an optional vector must be a dense
    tensor of the right dtype and shape on the call's device; a strided view
    is refused before any call (host tensors here, so nothing reaches a GPU)."""
    import torch
    cpu = torch.device("cpu")
    n = 4
    draft = torch.zeros(3 * n, dtype=torch.int32)
    lens = torch.full((n,), 2, dtype=torch.int32)
    budget = torch.zeros(n, 2)
    strided64 = torch.zeros(2 * n, dtype=torch.int64)[::2]
    strided32 = torch.zeros(2 * n, dtype=torch.int32)[::2]
    assert strided64.shape == (n,) and not strided64.is_contiguous()
    with pytest.raises(ValueError, match="row_offsets"):
        asd._marshal(cpu, 3 * n, draft, lens, 1.0, 1, budget, strided64, None, None, None, None)
    with pytest.raises(ValueError, match="row_offsets"):
        asd._marshal(cpu, 3 * n, draft, lens, 1.0, 1, budget,
                     torch.zeros(n, dtype=torch.int32), None, None, None, None)
    acc = torch.zeros(n, dtype=torch.int32)
    nxt = torch.zeros(n, dtype=torch.int32)
    tokens = torch.zeros(n, 8, dtype=torch.int32)
    seq = torch.zeros(n, dtype=torch.int64)
    with pytest.raises(ValueError, match="row_offsets"):
        asd.asd_commit(draft, lens, acc, nxt, tokens, seq, row_offsets=strided64)
    with pytest.raises(ValueError, match="out_committed"):
        asd.asd_commit(draft, lens, acc, nxt, tokens, seq, out_committed=strided32)
    amax = torch.zeros(3 * n, dtype=torch.int32)
    regret = torch.zeros(3 * n)
    taus = torch.zeros(2)
    ps = torch.ones(2, dtype=torch.int32)
    counts = torch.zeros(2, 2, dtype=torch.int64)
    mism = torch.zeros(1, dtype=torch.int64)
    with pytest.raises(ValueError, match="row_offsets"):
        asd.asd_opportunity(draft, amax, regret, 100, lens, taus, ps, counts, mism,
                            row_offsets=strided64)


@pytest.mark.parametrize("args", [
    (None, 24, 1, 1), (0x1008, 24, 1, 1), (0x1000, 5, 1, 1), (0x1000, 24, 0, 1),
    (0x1000, 24, 1 << 31, 1), (0x1000, 24, 1, 0)])
def test_mfma_probe_rejects_invalid_arguments(args):
    lib = asd._load()
    ops, vectors, wgs, steps = args
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    assert lib.asd_mfma_probe(vp(ops), vectors, wgs, steps, vp(0x2000), None) == 1


def _row_pass(**kw):
    lib = asd._load()
    a = dict(logits=0x1000, dtype=1, vocab=100, rows=2, draft=0x2000, out=0x3000, stream=None)
    a.update(kw)
    vp = lambda v: None if v is None else ctypes.c_void_p(v)
    return lib.asd_row_pass(vp(a["logits"]), a["dtype"], a["vocab"], a["rows"], vp(a["draft"]),
                            vp(a["out"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2),
    (dict(vocab=0), 1),
    (dict(vocab=1 << 30), 1),
    (dict(rows=0), 1),
    (dict(rows=1 << 31), 1),
    (dict(logits=None), 1),
    (dict(draft=None), 1),
    (dict(out=None), 1),
    (dict(out=0x3008), 1),                    # partials must be 16-byte aligned
    (dict(logits=0x1001), 1),
    (dict(logits=0x1002, dtype=0), 1),        # f32 rows must be 4-byte aligned
])
def test_row_pass_rejects_invalid_arguments(kw, status):
    assert _row_pass(**kw) == status


@pytest.mark.parametrize("args", [(5, 100, 2), (1, 0, 2), (1, 1 << 30, 2), (1, 100, 0),
                                  (0, 100, 1 << 31)])
def test_row_splits_is_zero_for_invalid_shapes(args):
    assert asd._load().asd_row_splits(*args) == 0
