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


def test_argument_checks_before_any_device_work(lib_path):
    """Host-side validation that returns before any HIP call: argument errors of fold_pack_params (including a
    set whose packed matrix would reach 2^32 entries), fold_adam_step and fold_loss_workspace_size."""
    from ctypes import c_void_p
    from paper_1702_02181_amd import fold as F
    fake = c_void_p(256)  # never dereferenced: validation fails first
    bias = c_void_p(512)
    null_stream = type("Stream", (), {"cuda_stream": 0})()  # the calls fail before using it
    ft = type("FakeTensor", (), {"data_ptr": lambda self: 256})()  # binding marshals tensors by data_ptr()

    def pack(kind, in_dim, arity, hidden, dtype=F.FOLD_F32):
        sets = (F.fold_param_set * 1)()
        sets[0] = F.fold_param_set(kind, in_dim, arity, fake, fake, bias)
        return F.fold_pack_params(F.fold_params(dtype, hidden, 1, sets), null_stream)

    for args in ((F.FOLD_TREELSTM, 1_000_000, 2, 4096), (F.FOLD_TREELSTM, 64, 2, 4097),
                 (F.FOLD_TREELSTM, 64, 1, 64), (F.FOLD_LSTM, -1, 1, 64)):
        with pytest.raises(F.FoldError) as e:
            pack(*args)
        assert e.value.code == F.FOLD_E_INVALID, args
    with pytest.raises(F.FoldError) as e:
        pack(F.FOLD_TREELSTM, 1_000_000, 2, 4096)
    assert "2^32" in str(e.value)
    # attention sets: in_dim 0, the kind's child slots, hidden >= 2 (c holds m and s), a scorer with w and b
    for args in ((F.FOLD_ATTN_SCORE, 0, 1, 1), (F.FOLD_ATTN_SUM, 0, 2, 1), (F.FOLD_ATTN_SCORE, 8, 1, 64),
                 (F.FOLD_ATTN_SCORE, 0, 2, 64), (F.FOLD_ATTN_SUM, 0, 1, 64), (F.FOLD_ATTN_OUT, 0, 2, 64),
                 (8, 0, 1, 64)):
        with pytest.raises(F.FoldError) as e:
            pack(*args)
        assert e.value.code == F.FOLD_E_INVALID, args
    sets = (F.fold_param_set * 1)()
    sets[0] = F.fold_param_set(F.FOLD_ATTN_SCORE, 0, 1, None, None, bias)
    with pytest.raises(F.FoldError) as e:
        F.fold_pack_params(F.fold_params(F.FOLD_F32, 64, 1, sets), null_stream)
    assert e.value.code == F.FOLD_E_INVALID and "scorer" in str(e.value)
    for args in ((16, ft, None, ft, ft, ft, 1e-3, 0.9, 0.999, 1e-8, 0),
                 (16, ft, None, ft, ft, ft, 1e-3, 0.9, 1.0, 1e-8, 1),
                 (16, ft, None, ft, ft, ft, float("inf"), 0.9, 0.999, 1e-8, 1),
                 (16, ft, None, ft, ft, ft, 1e-3, 0.9, 0.999, -1.0, 1)):
        with pytest.raises(F.FoldError) as e:
            F.fold_adam_step(*args, stream=null_stream)
        assert e.value.code == F.FOLD_E_INVALID, args
    with pytest.raises(F.FoldError) as e:
        F.fold_loss_workspace_size(None, 5)
    assert e.value.code == F.FOLD_E_INVALID
