"""The C ABI: the library loads and exports every symbol include/massive.h
declares (no compute calls; runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "massive.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(massive_[a-z_]+)\s*\(", text)))


def test_header_declares_the_three_calls():
    names = declared_functions()
    for n in ("massive_init", "massive_sample", "massive_evict_step"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2410_22697_amd import massive
    if not os.path.exists(massive.LIB_PATH):
        pytest.skip("libmassive.so not built")
    lib = ctypes.CDLL(massive.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(massive.EXPORTS)


def test_init_error_path_without_gpu():
    """An invalid argument is rejected before any device call."""
    from paper_2410_22697_amd import massive
    if not os.path.exists(massive.LIB_PATH):
        pytest.skip("libmassive.so not built")
    lib = massive.load()
    a = massive.InitArgs()
    a.L, a.H, a.K = 4, 0, 0   # K = 0 is invalid
    h = ctypes.c_void_p()
    rc = lib.massive_init(ctypes.byref(a), ctypes.byref(h))
    assert rc == massive.EINVAL
    assert b"NULL" in lib.massive_last_error(None) or b"K" in lib.massive_last_error(None)
    assert not h.value


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    from paper_2410_22697_amd import massive
    monkeypatch.setattr(massive, "LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(massive, "_lib", None)
    with pytest.raises(ImportError):
        massive.load()
