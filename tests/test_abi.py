"""The C-ABI library loads and exports every entry point its header declares
(CPU: no compute calls)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fst_compose.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"FST_API\s+[\w\s\*]+?\b(fst_\w+)\s*\(", text)))


def test_header_declares_entry_points():
    names = declared_functions()
    assert "fst_compose_run" in names and "fst_compose_fill" in names
    assert len(names) >= 8


def test_library_exports_every_declared_symbol():
    from paper_2110_02848_amd import gpu
    if not os.path.exists(gpu.LIB_PATH):
        pytest.skip("library not built")
    lib = ctypes.CDLL(gpu.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", gpu.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(\w+)$", out, flags=re.M))
    assert exported == set(declared_functions())


def test_strerror_without_gpu():
    from paper_2110_02848_amd import gpu
    if not os.path.exists(gpu.LIB_PATH):
        pytest.skip("library not built")
    lib = gpu.load()
    assert lib.fst_strerror(0) == b"ok"
    assert b"invalid graph" == lib.fst_strerror(2)
    assert lib.fst_strerror(99) == b"unknown error"


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2110_02848_amd import gpu
    monkeypatch.setattr(gpu, "_lib", None)
    monkeypatch.setattr(gpu, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        gpu.load()
