"""CPU checks of the C-ABI library: it loads and exports every function that
include/fa.h declares, and the Python binding declares the same set.  No
compute call is made (no GPU here)."""
import ctypes
import os
import re
import shutil

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fa.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fa_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2608_21131_amd import build, fa
    if not os.path.exists(fa.LIB_PATH):
        if not shutil.which(os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")):
            pytest.skip("libfa.so not built and hipcc unavailable")
        build.build()
    return ctypes.CDLL(fa.LIB_PATH)


def test_header_declares_the_path():
    names = declared_functions()
    for required in ("fa_keygen", "fa_encrypt", "fa_decrypt", "fa_encode_db_block", "fa_project_ct",
                     "fa_score_block", "fa_rotate_sum"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_matches_header(lib):
    from paper_2608_21131_amd import fa
    assert sorted(fa.SIGNATURES) == declared_functions()
    fa.load_library()  # declares argtypes for every symbol


def test_last_error_is_callable_without_gpu(lib):
    lib.fa_last_error.restype = ctypes.c_char_p
    assert isinstance(lib.fa_last_error(), bytes)
