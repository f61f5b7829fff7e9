"""The C-ABI library loads without a GPU and exports every symbol that
include/fate.h declares (no compute calls)."""

import os
import re

from paper_2605_07238_amd import fate

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "fate.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fate_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_symbols() == sorted(fate.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = fate.load()
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_version_and_strerror():
    assert "gfx950" in fate.version()
    lib = fate.load()
    for code in range(-7, 1):
        assert lib.fate_strerror(code).decode()
    assert lib.fate_strerror(-99).decode() == "unknown status"
