"""The C-ABI library loads and exports every function include/das.h declares
(no compute calls)."""

import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

lib_mod = pytest.importorskip("paper_2609_34538_amd._lib")
LIB = lib_mod.LIB


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "das.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(das_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = _declared_functions()
    assert "das_attn_draft_maturev" in names and "das_kv_append" in names
    for n in names:
        assert hasattr(LIB, n), f"libdas.so does not export {n}"
    assert set(names) >= set(lib_mod.EXPORTED)


def test_status_strings_and_version():
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8, 12345):
        assert LIB.das_status_string(code)
    assert LIB.das_version() >= 100
