"""CPU checks of the C-ABI library: it loads and exports every function that
include/fa.h declares, and the Python binding declares the same set.  No
compute call is made (no GPU here)."""
import ctypes
import os
import re
import shutil

import numpy as np
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


def test_chebyshev_square_root_fit_matches_numpy(lib):
    """fa_cheb_fit_sqrt (host only) is Chebyshev interpolation at the first-kind points:
    numpy's chebinterpolate of the same function agrees to rounding."""
    from paper_2608_21131_amd import fa
    for tau, lo, hi, deg in [(0.6, 0.5, 2.5, 7), (1.0, 0.1, 1.0, 12), (0.3, 1.0, 9.0, 3)]:
        got = fa.cheb_fit_sqrt(tau, lo, hi, deg)
        half, mid = (hi - lo) / 2, (hi + lo) / 2
        ref = np.polynomial.chebyshev.chebinterpolate(lambda u: tau * np.sqrt(mid + half * u), deg)
        assert np.max(np.abs(got - ref)) < 1e-14
    with pytest.raises(fa.FaError):
        fa.cheb_fit_sqrt(0.6, 0.0, 2.5, 7)


def test_context_parameters_rejected_before_the_device(lib):
    """fa_ctx_create refuses, before touching the device, more key-switch digits than the
    kernels are built for and explicit primes the arithmetic cannot use: outside (2^49, 2^50),
    not 1 mod 2N, composite, or listed twice."""
    from oracle import ckks
    from paper_2608_21131_amd import fa
    fa.load_library()
    h = ctypes.c_void_p()

    def create(logn, L, K, primes=None):
        arr = None if primes is None else np.ascontiguousarray(primes, dtype=np.uint64)
        prm = fa._Params(logn, L, K, 40, None if arr is None else arr.ctypes.data_as(fa._u64p))
        rc = fa._LIB.fa_ctx_create(ctypes.byref(prm), ctypes.byref(h))
        return rc, fa._LIB.fa_last_error().decode()

    rc, msg = create(16, 12, 1)          # twelve digits
    assert rc == fa.FA_E_INVAL and "digits" in msg
    rc, msg = create(12, 16, 1)          # sixteen digits
    assert rc == fa.FA_E_INVAL and "digits" in msg
    logn = 12
    m = 2 << logn
    good = ckks.find_primes(logn, 4)
    composite = next(c for c in range(good[0] - m, good[0] - 200 * m, -m) if not ckks.is_probable_prime(c))
    for bad, what in [([good[0], good[1], 1 << 50, good[3]], "not in"),
                      ([good[0], good[1], good[2] + 2, good[3]], "1 mod 2N"),
                      ([good[0], composite, good[2], good[3]], "not prime"),
                      ([good[0], good[1], good[0], good[3]], "twice")]:
        rc, msg = create(logn, 3, 1, bad)
        assert rc == fa.FA_E_INVAL and what in msg, (bad, msg)
