"""CPU-side checks of the C-ABI boundary: the library loads, exports every
function include/nmt.h declares, and rejects bad host arguments without
touching a device.  Also checks that the product path never reaches the
oracle."""
import ctypes
import os
import re

import pytest

from paper_1605_04809_amd import binding as nb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def declared_functions():
    names = set()
    for f in sorted(os.listdir(INCLUDE)):
        if f.endswith(".h"):
            src = re.sub(r"/\*.*?\*/", "", open(os.path.join(INCLUDE, f)).read(), flags=re.S)
            names.update(re.findall(r"\b(nmt_[a-z_0-9]+)\s*\(", src))
    return sorted(names)


def test_header_and_binding_agree():
    assert declared_functions() == sorted(nb.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = nb.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_host_argument_errors_need_no_device():
    lib = nb.load_library()
    out = ctypes.c_void_p()
    assert lib.nmt_model_create(None, None, ctypes.byref(out)) == nb.NMT_EINVAL
    assert "NULL" in nb.last_error()
    dims = nb.Dims(10, 10, 6, 8, 8, nb.NMT_F32)  # E not a multiple of 4
    w = nb.Weights()
    assert lib.nmt_model_create(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(out)) == nb.NMT_EINVAL
    assert "multiples of 4" in nb.last_error()
    dims = nb.Dims(10, 10, 8, 8, 8, nb.NMT_F32)  # all weight pointers NULL
    assert lib.nmt_model_create(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(out)) == nb.NMT_EINVAL
    assert lib.nmt_score_batch(None, None, 4, *([None] * 8), 0, None) == nb.NMT_EINVAL
    assert lib.nmt_score_workspace_bytes(None, 5) == 0
    assert lib.nmt_stream_status(None, None) == nb.NMT_EINVAL
    lib.nmt_model_destroy(None)
    lib.nmt_source_destroy(None)


def test_product_path_does_not_touch_the_oracle():
    pkg = os.path.join(ROOT, "paper_1605_04809_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), f
                assert "liboracle" not in text and "oracle.h" not in text, f


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="missing"):
        nb.load_library.__wrapped__(str(tmp_path / "libnmt.so")) if hasattr(nb.load_library, "__wrapped__") \
            else _fresh_load(str(tmp_path / "libnmt.so"))


def _fresh_load(path):
    saved = nb._lib
    nb._lib = None
    try:
        nb.load_library(path)
    finally:
        nb._lib = saved


def test_noalloc_scratch_size_and_host_errors():
    """The binding's copy of the allocation-free scratch size matches the
    header, and the entry point rejects host arguments without a device."""
    hdr = open(os.path.join(INCLUDE, "nmt.h")).read()
    m = re.search(r"#define\s+NMT_NOALLOC_SCRATCH_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == nb.NOALLOC_SCRATCH_BYTES
    lib = nb.load_library()
    assert lib.nmt_score_batch_noalloc(None, None, 4, *([None] * 7), None) == nb.NMT_EINVAL
    assert "NULL" in nb.last_error()


def test_gemm_form_switch_needs_no_device():
    """The test switch between the bf16 products' kernel forms (nmt_debug.h)
    returns the previous form and refuses forms outside 0..4."""
    prev = nb.debug_gemm_form(0)
    try:
        assert nb.debug_gemm_form(5) == -1
        assert nb.debug_gemm_form(-1) == -1
        assert nb.debug_gemm_form(2) == 0
        assert nb.debug_gemm_form(4) == 2
        assert nb.debug_gemm_form(1) == 4
        assert nb.debug_gemm_form(0) == 1
    finally:
        nb.debug_gemm_form(prev)
