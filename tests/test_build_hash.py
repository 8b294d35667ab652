"""The library is tied to the sources it was built from: the build embeds a
hash of the sources in asd_version(), and loading a library whose hash differs
from the sources beside it fails (so a stale build is never tested, benchmarked
or smoke-checked)."""
import ctypes
import os
import subprocess

import pytest

import paper_2608_03447_amd as asd
from paper_2608_03447_amd.build import HASHED_SOURCES, LIBRARY, source_hash


def _stub_library(tmp_path, word):
    src = tmp_path / "stub.c"
    src.write_text('const char *asd_version(void) { return "asd-mi355x 0.4.0 gfx950 src %s"; }\n'
                   % word)
    out = tmp_path / "libasd_stub.so"
    subprocess.run(["gcc", "-shared", "-fPIC", str(src), "-o", str(out)], check=True)
    lib = ctypes.CDLL(str(out))
    lib.asd_version.restype = ctypes.c_char_p
    return out, lib


def test_built_library_carries_the_hash_of_its_sources():
    if not os.path.exists(LIBRARY):
        pytest.skip("library not built")
    lib = asd._load()
    assert asd.library_source_hash(lib) == source_hash()


def test_hash_ignores_comments_and_whitespace_but_not_code(tmp_path):
    a = tmp_path / "a.cpp"
    b = tmp_path / "b.cpp"
    c = tmp_path / "c.cpp"
    a.write_text("int f(int x) { return x + 1; }  // one\n")
    b.write_text("/* other comment */ int f(int x)\n{\n    return x + 1;\n}\n")
    c.write_text("int f(int x) { return x + 2; }\n")
    assert source_hash([str(a)]) == source_hash([str(b)])
    assert source_hash([str(a)]) != source_hash([str(c)])
    assert len(HASHED_SOURCES) == 4


def test_stale_library_is_refused(tmp_path):
    path, lib = _stub_library(tmp_path, "0000000000000000")
    with pytest.raises(RuntimeError, match="built from other sources"):
        asd.check_built_from_sources(lib, str(path))
    (tmp_path / "good").mkdir()
    _, good = _stub_library(tmp_path / "good", source_hash())
    asd.check_built_from_sources(good, "stub")


def test_smoke_refuses_a_stale_library(tmp_path, monkeypatch):
    import __graft_entry__
    path, _ = _stub_library(tmp_path, "0123456789abcdef")
    monkeypatch.setattr(asd, "LIBRARY", str(path))
    monkeypatch.setattr(asd, "_lib", None)
    with pytest.raises(RuntimeError, match="built from other sources"):
        __graft_entry__.smoke()
