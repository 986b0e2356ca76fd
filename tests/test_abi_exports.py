"""The C-ABI library builds for gfx950, loads without a GPU and exports every symbol the header declares.
No compute call is made here."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fold.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(fold_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def lib_path():
    from paper_1702_02181_amd import build_lib
    if not os.path.exists(build_lib.LIB):
        build_lib.build()
    return build_lib.LIB


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("fold_schedule", "fold_forward", "fold_backward", "fold_last_error", "fold_workspace_size"):
        assert n in names


def test_library_exports_every_declared_symbol(lib_path):
    out = subprocess.run(["nm", "-D", "--defined-only", lib_path], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (\w+)$", out, flags=re.M))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing


def test_library_loads_and_binding_matches(lib_path):
    from paper_1702_02181_amd import fold as F
    L = F.lib()
    for n in declared_functions():
        assert hasattr(L, n)
    assert sorted(F.EXPORTS) == declared_functions()
    # pure host helpers, no device work
    assert F.fold_row_ld(300) == 320 and F.fold_row_ld(256) == 256 and F.fold_row_ld(1) == 64
    assert F.fold_last_error() == ""
