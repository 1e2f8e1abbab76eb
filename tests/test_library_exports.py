"""The C-ABI library loads on the CPU host and exports every declared entry point."""

import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ravel.h")
LIB = os.path.join(ROOT, "paper_2609_34170_amd", "libravel.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ravel_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ["ravel_create", "ravel_set_context", "ravel_step", "ravel_buffer_create",
                 "ravel_context_acquire", "ravel_fop_encode", "ravel_last_error"]:
        assert must in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libravel.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (ravel_\w+)", out))
    assert set(declared_functions()) <= exported


@pytest.mark.skipif(not os.path.exists(LIB), reason="libravel.so not built")
def test_binding_symbol_table_matches_header():
    from paper_2609_34170_amd import ravel
    assert sorted(ravel.SYMBOLS) == declared_functions()
    lib = ravel.load_library()
    assert lib.ravel_last_error() == b""


@pytest.mark.skipif(not os.path.exists(LIB), reason="libravel.so not built")
def test_argument_errors_are_reported_without_a_gpu():
    from paper_2609_34170_amd import ravel
    lib = ravel.load_library()
    st = lib.ravel_create(None, None, 0, None)
    assert st == -1
    assert b"null" in lib.ravel_last_error()
    assert lib.ravel_step(None, None, None, None) == -1
