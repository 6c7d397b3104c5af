"""The C-ABI library loads and exports every entry point its headers declare;
argument validation rejects bad calls before any device work (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2309_16743_amd", "libonline_train.so")


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if not fn.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", fn)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(", text, re.M):
            names.add(m.group(1))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2309_16743_amd.build import build
        build()
    from paper_2309_16743_amd import _abi
    return _abi.load(LIB)


def test_headers_declare_the_four_paper_calls():
    names = declared_functions()
    for n in ("reservoir_put", "reservoir_sample_batch", "surrogate_train_step", "surrogate_predict"):
        assert n in names
    assert len(names) >= 19


def test_every_declared_symbol_is_exported(lib):
    from paper_2309_16743_amd import _abi
    names = declared_functions()
    for n in names:
        assert hasattr(lib, n), n
    assert names == set(_abi.SIGNATURES), names ^ set(_abi.SIGNATURES)


def test_version_and_error_string(lib):
    assert b"gfx950" in lib.ot_version()
    assert lib.ot_last_error() == b""


def test_validation_errors_before_device_work(lib):
    from paper_2309_16743_amd import _abi
    h = C.c_void_p()
    assert lib.reservoir_create(C.byref(h), 0, 0, 6, 10, 0, 0, None) == _abi.OT_E_INVAL
    assert b"capacity" in lib.ot_last_error()
    assert lib.reservoir_create(C.byref(h), 10, -1, 6, 10, 0, 0, None) == _abi.OT_E_INVAL
    assert lib.reservoir_create(C.byref(h), 10, 1, 6, 10, 0, 3, None) == _abi.OT_E_INVAL
    assert b"policy" in lib.ot_last_error()
    assert lib.reservoir_put(None, None, 0, None, 0, 1, None, None, None) == _abi.OT_E_INVAL
    assert lib.reservoir_sample_batch(None, 4, None, None, None, 0, None, 0, None, None) == _abi.OT_E_INVAL
    w = (C.c_int64 * 3)(6, 0, 4)
    assert lib.surrogate_create(C.byref(h), w, 3, 0, 1e-3, 0.9, 0.999, 1e-8, 0, 16, 0) == _abi.OT_E_INVAL
    w = (C.c_int64 * 3)(6, 8, 4)
    assert lib.surrogate_create(C.byref(h), w, 3, 0, 1e-3, 0.9, 0.999, 1e-8, 0, 16, 7) == _abi.OT_E_INVAL
    assert lib.surrogate_train_step(None, None, 0, None, 0, 1, None, None) == _abi.OT_E_INVAL
    assert lib.surrogate_train_step_rows(None, None, 0, None, 0, None, 1, 1, None, None, None) == _abi.OT_E_INVAL
    assert b"NULL surrogate" in lib.ot_last_error()
    assert lib.surrogate_eval_loss(None, None, 0, None, 0, 1, None, None) == _abi.OT_E_INVAL
    assert lib.surrogate_set_lr(None, C.c_float(1e-3)) == _abi.OT_E_INVAL
    assert lib.surrogate_set_device_step(None, 1) == _abi.OT_E_INVAL
    assert lib.reservoir_slab(None, None, None, None, None) == _abi.OT_E_INVAL
    assert b"NULL reservoir" in lib.ot_last_error()
    assert lib.reservoir_destroy(None) == _abi.OT_OK
