"""Thin Python binding of libfa (the C ABI in include/fa.h).

Argument marshalling only: every step of the encrypted scoring path runs in
the library's HIP kernels.  PyTorch provides device memory (8-byte-word
tensors) and the current HIP stream.  There is no fallback: if libfa.so is
missing or no GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

import torch  # noqa: F401  (load torch's HIP runtime before libfa so both share it)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfa.so")

FA_OK, FA_E_INVAL, FA_E_SHAPE, FA_E_NOKEY, FA_E_NOMEM, FA_E_HIP = 0, -1, -2, -3, -4, -5
LAYOUT_ROW, LAYOUT_DIAG, LAYOUT_DIAG_ENC = 0, 1, 2
(OP_SCORE, OP_PROJECT, OP_ROTATE_SUM, OP_ROTATE, OP_PREPARE, OP_SCORE_PREPARED, OP_SCORE_ENC,
 OP_PROJECT_ENC) = 0, 1, 2, 3, 4, 5, 6, 7

_ERR_NAMES = {FA_E_INVAL: "FA_E_INVAL", FA_E_SHAPE: "FA_E_SHAPE", FA_E_NOKEY: "FA_E_NOKEY",
              FA_E_NOMEM: "FA_E_NOMEM", FA_E_HIP: "FA_E_HIP"}


class FaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class _Params(ctypes.Structure):
    _fields_ = [("log_n", ctypes.c_uint32), ("L", ctypes.c_uint32), ("K", ctypes.c_uint32),
                ("log_scale", ctypes.c_uint32), ("primes", ctypes.POINTER(ctypes.c_uint64))]


class _FaBuf(ctypes.Structure):
    _fields_ = [("dev", ctypes.c_void_p), ("bytes", ctypes.c_size_t), ("n_polys", ctypes.c_uint32),
                ("count", ctypes.c_uint32), ("limbs", ctypes.c_uint32), ("log_scale", ctypes.c_int32)]


_vp = ctypes.c_void_p
_bp = ctypes.POINTER(_FaBuf)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)
_f32p = ctypes.POINTER(ctypes.c_float)

# name -> (restype, argtypes); mirrors include/fa.h
SIGNATURES = {
    "fa_ctx_create": (ctypes.c_int, [ctypes.POINTER(_Params), ctypes.POINTER(_vp)]),
    "fa_ctx_destroy": (None, [_vp]),
    "fa_ctx_create_level": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.POINTER(_vp)]),
    "fa_drop_level": (ctypes.c_int, [_vp, _vp, _bp, _bp, _vp]),
    "fa_ctx_primes": (ctypes.c_int, [_vp, _u64p]),
    "fa_ct_bytes": (ctypes.c_size_t, [_vp]),
    "fa_pt_bytes": (ctypes.c_size_t, [_vp]),
    "fa_key_bytes": (ctypes.c_size_t, [_vp]),
    "fa_last_error": (ctypes.c_char_p, []),
    "fa_keygen": (ctypes.c_int, [_vp, _i64p, _i32p, ctypes.c_int, _u64p, _i64p]),
    "fa_has_key": (ctypes.c_int, [_vp, ctypes.c_int]),
    "fa_set_secret": (ctypes.c_int, [_vp, _i64p]),
    "fa_encrypt": (ctypes.c_int, [_vp, _i64p, ctypes.c_int32, _u64p, _i64p, _bp, _vp]),
    "fa_decrypt": (ctypes.c_int, [_vp, _bp, _u64p, _vp]),
    "fa_export_coeffs": (ctypes.c_int, [_vp, _bp, _u64p, _vp]),
    "fa_import_coeffs": (ctypes.c_int, [_vp, _u64p, _bp, _vp]),
    "fa_encode": (ctypes.c_int, [_vp, _f64p, ctypes.c_int, ctypes.c_int, _i64p]),
    "fa_decode": (ctypes.c_int, [_vp, _u64p, ctypes.c_int, _f64p, ctypes.c_int]),
    "fa_encode_db_block": (ctypes.c_int, [_vp, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp]),
    "fa_encode_db_block_int": (ctypes.c_int, [_vp, _i64p, ctypes.c_int, ctypes.c_int32, _bp, _vp]),
    "fa_encode_projection": (ctypes.c_int, [_vp, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp]),
    "fa_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "fa_score_block": (ctypes.c_int, [_vp, _bp, _bp, ctypes.c_int, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_project_ct": (ctypes.c_int, [_vp, _bp, _bp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_project_ct_enc": (ctypes.c_int, [_vp, _bp, _bp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_rotate_sum": (ctypes.c_int, [_vp, _bp, ctypes.c_int, ctypes.c_int, _vp, ctypes.c_size_t, _vp]),
    "fa_rotate": (ctypes.c_int, [_vp, _bp, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_prepared_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int]),
    "fa_prepare_query": (ctypes.c_int, [_vp, _bp, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_score_prepared": (ctypes.c_int, [_vp, _bp, _bp, _bp, ctypes.c_int, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_keygen_relin": (ctypes.c_int, [_vp, _i64p, _u64p, _i64p]),
    "fa_has_relin_key": (ctypes.c_int, [_vp]),
    "fa_encrypt_pts": (ctypes.c_int, [_vp, _bp, _u64p, _i64p, _bp, _vp]),
    "fa_rescale": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_mul_ct": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_ct_add": (ctypes.c_int, [_vp, _vp, _vp, _vp, ctypes.c_int, _vp]),
    "fa_ct_mul_const": (ctypes.c_int, [_vp, _vp, ctypes.c_int64, _vp, _vp]),
    "fa_ct_add_const": (ctypes.c_int, [_vp, _vp, ctypes.c_double, _vp, _vp]),
    "fa_chain_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int]),
    "fa_cheb_eval": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.c_int, _vp, ctypes.c_int, ctypes.c_double, _f64p,
                                    ctypes.c_int, _vp, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double),
                                    _vp, ctypes.c_size_t, _vp]),
    "fa_sign_iter": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.c_int, _vp, ctypes.c_int, ctypes.c_double,
                                    ctypes.c_int64, ctypes.c_int, _vp, ctypes.POINTER(ctypes.c_int),
                                    ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), _vp,
                                    ctypes.c_size_t, _vp]),
    "fa_cheb_fit_sqrt": (ctypes.c_int, [ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int, _f64p]),
    "fa_membership_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                        ctypes.c_int]),
    "fa_membership": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.c_int, _vp, ctypes.c_int, ctypes.c_double,
                                     ctypes.POINTER(_vp), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_double, ctypes.c_double, _f64p, ctypes.c_int, ctypes.c_int64,
                                     ctypes.c_int, _vp, ctypes.POINTER(ctypes.c_int),
                                     ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), _vp,
                                     ctypes.c_size_t, _vp]),
    "fa_prepare_batch_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int]),
    "fa_prepare_batch": (ctypes.c_int, [_vp, _bp, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_batch_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "fa_score_batch": (ctypes.c_int, [_vp, _bp, _bp, ctypes.c_int, _bp, ctypes.c_int, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _bp, _vp, ctypes.c_size_t, _vp]),
    "fa_rotate_static": (ctypes.c_int, [_vp, _bp, ctypes.c_int, _bp, _vp]),
    "fa_profile": (ctypes.c_int, [_vp, ctypes.c_int]),
    "fa_profile_read": (ctypes.c_int, [_vp, _f64p]),
}

_LIB = None


def load_library(path: str | None = None):
    """Load libfa.so (the in-tree build, or the file FA_LIBRARY names) and declare its
    signatures; raises if it was never built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = path or os.environ.get("FA_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"libfa.so not built ({path}); run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def _check(rc: int):
    if rc != FA_OK:
        raise FaError(rc, _LIB.fa_last_error().decode())


def _np(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a: np.ndarray, kind):
    return a.ctypes.data_as(kind)


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t):
    t = t.t if isinstance(t, Buf) else t
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8
    return ctypes.c_void_p(t.data_ptr())


CT, PT, CT3 = 2, 1, 3  # polynomials per object: ciphertext, plaintext, product before relinearisation


class Buf:
    """A device tensor (8-byte words) with the descriptor the library checks: polynomials per
    object (2 ciphertext, 1 plaintext), objects held, primes per polynomial (the level) and the
    scale exponent.  Calls that write a Buf set its descriptor; calls that read one check it.
    Slicing by words is allowed on whole objects and gives a Buf of those objects."""

    __slots__ = ("t", "n_polys", "count", "limbs", "log_scale", "n")

    def __init__(self, t: torch.Tensor, n_polys: int, count: int, limbs: int, log_scale: int, n: int):
        self.t, self.n_polys, self.count, self.limbs, self.log_scale, self.n = t, n_polys, count, limbs, log_scale, n

    @property
    def obj_words(self) -> int:
        return self.n_polys * self.limbs * self.n

    def items(self, i: int, k: int = 1) -> "Buf":
        """Objects i .. i+k-1 as a Buf over the same memory."""
        if i < 0 or k < 0 or i + k > self.count:
            raise IndexError(f"objects {i}..{i + k - 1} of {self.count}")
        w = self.obj_words
        return Buf(self.t[i * w:(i + k) * w], self.n_polys, k, self.limbs, self.log_scale, self.n)

    def item(self, i: int) -> "Buf":
        return self.items(i, 1)

    def __getitem__(self, sl):
        if not isinstance(sl, slice) or sl.step not in (None, 1):
            raise TypeError("a Buf is sliced by a contiguous range of words")
        w = self.obj_words
        a = 0 if sl.start is None else sl.start
        b = self.count * w if sl.stop is None else min(sl.stop, self.count * w)
        if a % w or b % w:
            raise ValueError(f"slice [{a}:{b}] does not fall on whole objects of {w} words")
        return self.items(a // w, (b - a) // w)

    def numel(self) -> int:
        return self.t.numel()

    def zero_(self) -> "Buf":
        self.t.zero_()
        return self

    def c(self) -> _FaBuf:
        assert self.t.is_cuda and self.t.is_contiguous() and self.t.element_size() == 8
        return _FaBuf(ctypes.c_void_p(self.t.data_ptr()), self.t.numel() * 8, self.n_polys, self.count, self.limbs,
                      self.log_scale)

    def take(self, fb: _FaBuf) -> "Buf":
        """Adopt the descriptor the library wrote into fb."""
        self.n_polys, self.count, self.limbs, self.log_scale = fb.n_polys, fb.count, fb.limbs, fb.log_scale
        return self

    def __repr__(self):
        return (f"Buf({self.count} x {self.n_polys} polys, {self.limbs} primes, 2^{self.log_scale}, "
                f"{self.t.numel()} words)")


def _bufs(bs):
    bs = list(bs)
    arr = (_FaBuf * max(1, len(bs)))(*[b.c() for b in bs])
    return arr, len(bs)


def _ids(ids):
    if ids is None:
        return None, None
    a = _np(ids, np.int32)
    return a, _ptr(a, _i32p)


class Context:
    """One parameter set (ring degree, primes, tables, rotation keys) on the current GPU."""

    def __init__(self, log_n: int, L: int, K: int, log_scale: int = 40, _parent: "Context | None" = None,
                 primes=None):
        if not torch.cuda.is_available():
            raise RuntimeError("libfa needs a HIP GPU; none is visible")
        self.lib = load_library()
        self.log_n, self.L, self.K, self.log_scale = log_n, L, K, log_scale
        self.n = 1 << log_n
        self.slots = self.n // 2
        self.dnum = -(-L // K)
        h = _vp()
        if _parent is None:
            pa = None if primes is None else _np(primes, np.uint64)
            prm = _Params(log_n, L, K, log_scale, None if pa is None else _ptr(pa, _u64p))
            _check(self.lib.fa_ctx_create(ctypes.byref(prm), ctypes.byref(h)))
        else:
            _check(self.lib.fa_ctx_create_level(_parent.h, L, ctypes.byref(h)))
        self.h = h
        self.parent = _parent
        pr = np.zeros(L + K, dtype=np.uint64)
        _check(self.lib.fa_ctx_primes(self.h, _ptr(pr, _u64p)))
        self.primes = [int(x) for x in pr]
        self.ct_bytes = int(self.lib.fa_ct_bytes(self.h))
        self.pt_bytes = int(self.lib.fa_pt_bytes(self.h))
        self.ct_words = self.ct_bytes // 8
        self.pt_words = self.pt_bytes // 8

    def at_level(self, L_low: int) -> "Context":
        """Lower-level context: first L_low ciphertext primes, same special primes,
        restricted secret and rotation keys."""
        return Context(self.log_n, L_low, self.K, self.log_scale, _parent=self)

    def drop_level(self, child: "Context", ct: Buf, out: Buf | None = None, stream=None) -> Buf:
        out = child.new_ct(ct.count) if out is None else out
        fo = out.c()
        _check(self.lib.fa_drop_level(self.h, child.h, ctypes.byref(ct.c()), ctypes.byref(fo), _stream(stream)))
        return out.take(fo)

    def close(self):
        if getattr(self, "h", None):
            self.lib.fa_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- buffers ----
    def new_ct(self, count: int = 1, log_scale: int = 0) -> Buf:
        t = torch.empty(count * self.ct_words, dtype=torch.float64, device="cuda")
        return Buf(t, CT, count, self.L, log_scale, self.n)

    def new_pt(self, count: int = 1, log_scale: int = 0) -> Buf:
        t = torch.empty(count * self.pt_words, dtype=torch.float64, device="cuda")
        return Buf(t, PT, count, self.L, log_scale, self.n)

    def wrap(self, t: torch.Tensor, n_polys: int, count: int, log_scale: int) -> Buf:
        """Describe an existing device tensor as count objects of n_polys polynomials at this level."""
        return Buf(t, n_polys, count, self.L, log_scale, self.n)

    def workspace(self, op: int, n_blocks: int = 1, d: int = 1, baby_step: int = 1) -> torch.Tensor:
        nbytes = int(self.lib.fa_workspace_bytes(self.h, op, n_blocks, d, baby_step))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def workspace_bytes(self, op: int, n_blocks: int = 1, d: int = 1, baby_step: int = 1) -> int:
        return int(self.lib.fa_workspace_bytes(self.h, op, n_blocks, d, baby_step))

    # ---- keys / client ----
    def keygen(self, s, steps, a, e):
        s = _np(s, np.int64)
        steps = _np(steps, np.int32)
        a = _np(a, np.uint64)
        e = _np(e, np.int64)
        assert a.size == len(steps) * self.dnum * (self.L + self.K) * self.n
        assert e.size == len(steps) * self.dnum * self.n
        _check(self.lib.fa_keygen(self.h, _ptr(s, _i64p), _ptr(steps, _i32p), len(steps), _ptr(a, _u64p),
                                  _ptr(e, _i64p)))

    def has_key(self, step: int) -> bool:
        return bool(self.lib.fa_has_key(self.h, step))

    def keygen_relin(self, s, a, e):
        """Relinearisation key (s^2 -> s) from host randomness a [dnum][L+K][N], e [dnum][N]."""
        s = _np(s, np.int64)
        a = _np(a, np.uint64)
        e = _np(e, np.int64)
        assert a.size == self.dnum * (self.L + self.K) * self.n and e.size == self.dnum * self.n
        _check(self.lib.fa_keygen_relin(self.h, _ptr(s, _i64p), _ptr(a, _u64p), _ptr(e, _i64p)))

    def has_relin_key(self) -> bool:
        return bool(self.lib.fa_has_relin_key(self.h))

    def encrypt_pts(self, pts: Buf, n_pts: int | None = None, a=None, e=None, out: Buf | None = None,
                    stream=None) -> Buf:
        """Encrypt the device plaintexts of pts with host randomness a [count][L][N], e [count][N];
        returns that many ciphertexts (an encrypted diagonal block)."""
        if n_pts is not None and n_pts != pts.count:
            pts = pts.items(0, n_pts)
        a = _np(a, np.uint64)
        e = _np(e, np.int64)
        assert a.size == pts.count * self.L * self.n and e.size == pts.count * self.n
        out = self.new_ct(pts.count) if out is None else out
        fo = out.c()
        _check(self.lib.fa_encrypt_pts(self.h, ctypes.byref(pts.c()), _ptr(a, _u64p), _ptr(e, _i64p),
                                       ctypes.byref(fo), _stream(stream)))
        return out.take(fo)

    def set_secret(self, s):
        s = _np(s, np.int64)
        _check(self.lib.fa_set_secret(self.h, _ptr(s, _i64p)))

    def encrypt(self, m, a, e, out: Buf | None = None, stream=None, log_scale: int | None = None) -> Buf:
        out = self.new_ct() if out is None else out
        m, a, e = _np(m, np.int64), _np(a, np.uint64), _np(e, np.int64)
        ls = self.log_scale if log_scale is None else log_scale
        fo = out.c()
        _check(self.lib.fa_encrypt(self.h, _ptr(m, _i64p), ls, _ptr(a, _u64p), _ptr(e, _i64p), ctypes.byref(fo),
                                   _stream(stream)))
        return out.take(fo)

    def decrypt(self, ct: Buf, stream=None) -> np.ndarray:
        out = np.empty((self.L, self.n), dtype=np.uint64)
        _check(self.lib.fa_decrypt(self.h, ctypes.byref(ct.c()), _ptr(out, _u64p), _stream(stream)))
        return out

    def export(self, buf: Buf, n_polys: int | None = None, stream=None) -> np.ndarray:
        """Canonical coefficient form of every polynomial of buf: [count * n_polys][L][N]."""
        total = buf.count * buf.n_polys
        if n_polys is not None and n_polys != total:
            raise ValueError(f"buffer holds {total} polynomials, not {n_polys}")
        out = np.empty((total, self.L, self.n), dtype=np.uint64)
        _check(self.lib.fa_export_coeffs(self.h, ctypes.byref(buf.c()), _ptr(out, _u64p), _stream(stream)))
        return out

    def import_coeffs(self, coeffs, n_polys: int = 1, log_scale: int = 0, out: Buf | None = None,
                      stream=None) -> Buf:
        """The inverse of export: canonical [count * n_polys][L][N] residues into a device buffer of
        count objects of n_polys polynomials at scale 2^log_scale."""
        c = _np(coeffs, np.uint64)
        if c.ndim != 3 or c.shape[1:] != (self.L, self.n) or c.shape[0] % n_polys:
            raise ValueError(f"coefficients must be [count * {n_polys}][{self.L}][{self.n}]")
        count = c.shape[0] // n_polys
        if out is None:
            out = Buf(torch.empty(c.size, dtype=torch.float64, device="cuda"), n_polys, count, self.L, log_scale,
                      self.n)
        else:
            out.n_polys, out.count, out.limbs, out.log_scale = n_polys, count, self.L, log_scale
        _check(self.lib.fa_import_coeffs(self.h, _ptr(c, _u64p), ctypes.byref(out.c()), _stream(stream)))
        return out

    def save_buffers(self, path: str, buffers: dict) -> None:
        """Save device buffers {name: Buf} (enrolled blocks, ciphertexts) in canonical coefficient
        form with a header naming this context's ring, primes and each buffer's descriptor."""
        import json
        header = {"format": "fa-coeffs-2", "log_n": self.log_n, "L": self.L, "K": self.K,
                  "primes": [int(p) for p in self.primes],
                  "buffers": {k: [int(v.n_polys), int(v.count), int(v.log_scale)] for k, v in buffers.items()}}
        arrays = {"header": np.frombuffer(json.dumps(header).encode(), dtype=np.uint8)}
        for name, buf in buffers.items():
            arrays["buf_" + name] = self.export(buf)
        np.savez(path, **arrays)

    def load_buffers(self, path: str) -> dict:
        """Load what save_buffers wrote into new device buffers {name: Buf}; the file must come
        from a context with the same ring degree and primes."""
        import json
        with np.load(path, allow_pickle=False) as z:
            header = json.loads(bytes(z["header"]).decode())
            mine = {"log_n": self.log_n, "L": self.L, "K": self.K, "primes": [int(p) for p in self.primes]}
            if header.get("format") != "fa-coeffs-2" or any(header.get(k) != v for k, v in mine.items()):
                raise ValueError(f"{path}: saved for another context ({header.get('log_n')}, {header.get('L')}, "
                                 f"{header.get('K')})")
            return {name: self.import_coeffs(z["buf_" + name], n_polys=d[0], log_scale=d[2])
                    for name, d in header["buffers"].items()}

    def encode(self, slots, log_scale: int | None = None) -> np.ndarray:
        v = _np(slots, np.float64)
        out = np.empty(self.n, dtype=np.int64)
        ls = self.log_scale if log_scale is None else log_scale
        _check(self.lib.fa_encode(self.h, _ptr(v, _f64p), v.size, ls, _ptr(out, _i64p)))
        return out

    def decode(self, res, log_scale: int, n_slots: int | None = None) -> np.ndarray:
        r = _np(res, np.uint64)
        k = self.slots if n_slots is None else n_slots
        out = np.empty(k, dtype=np.float64)
        _check(self.lib.fa_decode(self.h, _ptr(r, _u64p), log_scale, _ptr(out, _f64p), k))
        return out

    # ---- enrollment ----
    def encode_db_block(self, rows, d: int, layout: int, baby_step: int = 1,
                        out: Buf | None = None, stream=None) -> Buf:
        rows = _np(rows, np.float32)
        n_rows, dim = rows.shape
        n_pts = d if layout == LAYOUT_DIAG else max(1, -(-n_rows // (self.slots // d)))
        out = self.new_pt(n_pts) if out is None else out
        fo = out.c()
        _check(self.lib.fa_encode_db_block(self.h, _ptr(rows, _f32p), n_rows, dim, d, layout, baby_step,
                                           ctypes.byref(fo), _stream(stream)))
        return out.take(fo)

    def encode_projection(self, W, baby_step: int, out: Buf | None = None, stream=None) -> Buf:
        W = _np(W, np.float32)
        d_in, r = W.shape
        out = self.new_pt(r) if out is None else out
        fo = out.c()
        _check(self.lib.fa_encode_projection(self.h, _ptr(W, _f32p), d_in, r, baby_step, ctypes.byref(fo),
                                             _stream(stream)))
        return out.take(fo)

    def encode_db_block_int(self, coeffs, out: Buf | None = None, stream=None, log_scale: int | None = None) -> Buf:
        c = _np(coeffs, np.int64).reshape(-1, self.n)
        out = self.new_pt(c.shape[0]) if out is None else out
        ls = self.log_scale if log_scale is None else log_scale
        fo = out.c()
        _check(self.lib.fa_encode_db_block_int(self.h, _ptr(c, _i64p), c.shape[0], ls, ctypes.byref(fo),
                                               _stream(stream)))
        return out.take(fo)

    # ---- scoring ----
    def score_block(self, q: Buf, blocks, d: int, layout: int, baby_step: int = 1, out: Buf | None = None,
                    ws: torch.Tensor | None = None, stream=None, block_ids=None) -> Buf:
        """Score q against the blocks named by block_ids among `blocks` (all of them, in order,
        when block_ids is None): one output ciphertext per scored block."""
        barr, nres = _bufs(blocks)
        ida, idp = _ids(block_ids)
        nb = nres if ida is None else len(ida)
        out = self.new_ct(max(1, nb)) if out is None else out
        if ws is None and layout == LAYOUT_DIAG:
            ws = self.workspace(OP_SCORE, nb, d, baby_step)
        elif ws is None and layout == LAYOUT_DIAG_ENC:
            ws = self.workspace(OP_SCORE_ENC, nb, d, baby_step)
        ws_p, ws_b = (_dev(ws), ws.numel() * 8) if ws is not None else (ctypes.c_void_p(0), 0)
        fo = out.c()
        _check(self.lib.fa_score_block(self.h, ctypes.byref(q.c()), barr, nres, idp, nb, d, layout, baby_step,
                                       ctypes.byref(fo), ws_p, ws_b, _stream(stream)))
        return out.take(fo)

    def new_prep(self, baby_step: int) -> Buf:
        words = int(self.lib.fa_prepared_bytes(self.h, baby_step)) // 8
        t = torch.empty(words, dtype=torch.float64, device="cuda")
        return Buf(t, CT, max(0, baby_step - 1), self.L, 0, self.n)

    def prepare_query(self, q: Buf, baby_step: int, out: Buf | None = None, ws: torch.Tensor | None = None,
                      stream=None) -> Buf:
        out = self.new_prep(baby_step) if out is None else out
        ws = self.workspace(OP_PREPARE, 1, baby_step, baby_step) if ws is None else ws
        fo = out.c()
        _check(self.lib.fa_prepare_query(self.h, ctypes.byref(q.c()), baby_step, ctypes.byref(fo), _dev(ws),
                                         ws.numel() * 8, _stream(stream)))
        return out.take(fo)

    def prepare_batch_workspace(self, n_q: int, baby_step: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_prepare_batch_workspace_bytes(self.h, n_q, baby_step))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def prepare_batch(self, qs, baby_step: int, outs=None, ws: torch.Tensor | None = None, stream=None) -> list:
        """Prepare several queries together; outs[j] equals prepare_query(qs[j], baby_step)."""
        qs = list(qs)
        nq = len(qs)
        outs = [self.new_prep(baby_step) for _ in range(nq)] if outs is None else list(outs)
        if len(outs) != nq:
            raise ValueError("one prepared buffer per query")
        ws = self.prepare_batch_workspace(nq, baby_step) if ws is None else ws
        qa, _ = _bufs(qs)
        oa, _ = _bufs(outs)
        _check(self.lib.fa_prepare_batch(self.h, qa, nq, baby_step, oa, _dev(ws), ws.numel() * 8, _stream(stream)))
        for j in range(nq):
            outs[j].take(oa[j])
        return outs

    def score_prepared(self, q: Buf, prep: Buf, blocks, d: int, baby_step: int, out: Buf | None = None,
                       ws: torch.Tensor | None = None, stream=None, block_ids=None) -> Buf:
        barr, nres = _bufs(blocks)
        ida, idp = _ids(block_ids)
        nb = nres if ida is None else len(ida)
        out = self.new_ct(max(1, nb)) if out is None else out
        ws = self.workspace(OP_SCORE_PREPARED, nb, d, baby_step) if ws is None else ws
        fo = out.c()
        _check(self.lib.fa_score_prepared(self.h, ctypes.byref(q.c()), ctypes.byref(prep.c()), barr, nres, idp, nb,
                                          d, baby_step, ctypes.byref(fo), _dev(ws), ws.numel() * 8,
                                          _stream(stream)))
        return out.take(fo)

    def batch_workspace(self, n_q: int, n_blocks: int, d: int, baby_step: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_batch_workspace_bytes(self.h, n_q, n_blocks, d, baby_step))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def score_batch(self, qs, preps, blocks, d: int, baby_step: int, outs=None, ws: torch.Tensor | None = None,
                    stream=None, block_ids=None) -> list:
        """Score several prepared queries against the same blocks, one plaintext pass per
        group of up to four queries; outs[j] equals score_prepared(qs[j], preps[j], ...)."""
        qs, preps = list(qs), list(preps)
        nq = len(qs)
        if len(preps) != nq:
            raise ValueError("one prepared rotation set per query")
        barr, nres = _bufs(blocks)
        ida, idp = _ids(block_ids)
        nb = nres if ida is None else len(ida)
        outs = [self.new_ct(max(1, nb)) for _ in range(nq)] if outs is None else list(outs)
        ws = self.batch_workspace(nq, nb, d, baby_step) if ws is None else ws
        qa, _ = _bufs(qs)
        pa, _ = _bufs(preps)
        oa, _ = _bufs(outs)
        _check(self.lib.fa_score_batch(self.h, qa, pa, nq, barr, nres, idp, nb, d, baby_step, oa, _dev(ws),
                                       ws.numel() * 8, _stream(stream)))
        for j in range(nq):
            outs[j].take(oa[j])
        return outs

    # ---- the membership path (plain device pointers: level and scale are explicit) ----
    def chain_workspace(self, degree: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_chain_workspace_bytes(self.h, degree))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def rescale(self, lo: "Context", ct, n_polys: int = 2, out: Buf | None = None,
                ws: torch.Tensor | None = None, stream=None) -> Buf:
        """round(ct / last prime) at the next level down (lo = this context minus that prime)."""
        if out is None:
            # the membership path tracks its (non power-of-two) scales itself: log_scale 0
            out = Buf(torch.empty(n_polys * lo.L * lo.n, dtype=torch.float64, device="cuda"), n_polys, 1, lo.L, 0,
                      lo.n)
        if ws is None:
            ws = torch.empty(n_polys * self.L * self.n + 32, dtype=torch.float64, device="cuda")
        _check(self.lib.fa_rescale(self.h, lo.h, _dev(ct), n_polys, _dev(out), _dev(ws), ws.numel() * 8,
                                   _stream(stream)))
        return out

    def mul_ct(self, x, y, out: Buf | None = None, stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        ws = self.chain_workspace(1)
        _check(self.lib.fa_mul_ct(self.h, _dev(x), _dev(y), _dev(out), _dev(ws), ws.numel() * 8, _stream(stream)))
        return out

    def ct_add(self, x, y, out=None, subtract: bool = False, stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_add(self.h, _dev(x), _dev(y), _dev(out), 1 if subtract else 0, _stream(stream)))
        return out

    def ct_mul_const(self, x, k: int, out=None, stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_mul_const(self.h, _dev(x), int(k), _dev(out), _stream(stream)))
        return out

    def ct_add_const(self, x, k: int, out=None, stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_add_const(self.h, _dev(x), float(k), _dev(out), _stream(stream)))
        return out

    def project_ct(self, q: Buf, w_pts: Buf, d_in: int, r: int, baby_step: int, out: Buf | None = None,
                   ws: torch.Tensor | None = None, stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_PROJECT, 1, r, baby_step) if ws is None else ws
        fo = out.c()
        _check(self.lib.fa_project_ct(self.h, ctypes.byref(q.c()), ctypes.byref(w_pts.c()), d_in, r, baby_step,
                                      ctypes.byref(fo), _dev(ws), ws.numel() * 8, _stream(stream)))
        return out.take(fo)

    def project_ct_enc(self, q: Buf, w_cts: Buf, d_in: int, r: int, baby_step: int, out: Buf | None = None,
                       ws: torch.Tensor | None = None, stream=None) -> Buf:
        """The projection with W's r diagonals encrypted (fa_encrypt_pts of project_ct's plaintexts)."""
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_PROJECT_ENC, 1, r, baby_step) if ws is None else ws
        fo = out.c()
        _check(self.lib.fa_project_ct_enc(self.h, ctypes.byref(q.c()), ctypes.byref(w_cts.c()), d_in, r, baby_step,
                                          ctypes.byref(fo), _dev(ws), ws.numel() * 8, _stream(stream)))
        return out.take(fo)

    def rotate_sum(self, cts: Buf, n_cts: int | None, first_shift: int, n_steps: int,
                   ws: torch.Tensor | None = None, stream=None) -> Buf:
        """In place on the first n_cts ciphertexts of cts (all of them when n_cts is None)."""
        sub = cts if n_cts is None or n_cts == cts.count else cts.items(0, n_cts)
        ws = self.workspace(OP_ROTATE_SUM, sub.count) if ws is None else ws
        _check(self.lib.fa_rotate_sum(self.h, ctypes.byref(sub.c()), first_shift, n_steps, _dev(ws),
                                      ws.numel() * 8, _stream(stream)))
        return cts

    def profile(self, enable: bool = True):
        _check(self.lib.fa_profile(self.h, 1 if enable else 0))

    def profile_read(self) -> dict:
        ms = np.zeros(4, dtype=np.float64)
        _check(self.lib.fa_profile_read(self.h, _ptr(ms, _f64p)))
        return {"baby_ms": ms[0], "mac_ms": ms[1], "giant_ms": ms[2], "total_ms": ms[3]}

    def rotate_static(self, ct: Buf, step: int, out: Buf | None = None, stream=None) -> Buf:
        """fa_rotate with the library's fixed scratch array: no workspace, no allocation in the call."""
        out = self.new_ct() if out is None else out
        fo = out.c()
        _check(self.lib.fa_rotate_static(self.h, ctypes.byref(ct.c()), step, ctypes.byref(fo), _stream(stream)))
        return out.take(fo)

    def rotate(self, ct: Buf, step: int, out: Buf | None = None, ws: torch.Tensor | None = None,
               stream=None) -> Buf:
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_ROTATE, 1) if ws is None else ws
        fo = out.c()
        _check(self.lib.fa_rotate(self.h, ctypes.byref(ct.c()), step, ctypes.byref(fo), _dev(ws), ws.numel() * 8,
                                  _stream(stream)))
        return out.take(fo)


def _levels_arg(levels):
    levels = list(levels)
    return (_vp * len(levels))(*[c.h for c in levels]), len(levels)


def cheb_eval(levels, u: torch.Tensor, L_u: int, s_u: float, coeffs, out: torch.Tensor | None = None,
              ws: torch.Tensor | None = None, stream=None):
    """sum_k coeffs[k] T_k(u) on a chain of contexts (levels[0] the top); returns
    (out, level, scale) with out[:2*level*N] the result."""
    top = levels[0]
    arr, nl = _levels_arg(levels)
    c = _np(coeffs, np.float64)
    out = top.new_ct() if out is None else out
    ws = top.chain_workspace(len(c) - 1) if ws is None else ws
    L_out, s_out = ctypes.c_int(0), ctypes.c_double(0.0)
    _check(top.lib.fa_cheb_eval(arr, nl, _dev(u), L_u, s_u, _ptr(c, _f64p), len(c) - 1, _dev(out),
                                ctypes.byref(L_out), ctypes.byref(s_out), _dev(ws), ws.numel() * 8,
                                _stream(stream)))
    return out, L_out.value, s_out.value


def sign_iter(levels, v: torch.Tensor, L_v: int, s_v: float, m: int, iters: int, out: torch.Tensor | None = None,
              ws: torch.Tensor | None = None, stream=None):
    """iters steps of f(x) = (3x - x^3)/2 on x = v/m; returns (out, level, scale, multiplier)."""
    top = levels[0]
    arr, nl = _levels_arg(levels)
    out = top.new_ct() if out is None else out
    ws = top.chain_workspace(3) if ws is None else ws
    L_out, s_out, m_out = ctypes.c_int(0), ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(top.lib.fa_sign_iter(arr, nl, _dev(v), L_v, s_v, int(m), iters, _dev(out), ctypes.byref(L_out),
                                ctypes.byref(s_out), ctypes.byref(m_out), _dev(ws), ws.numel() * 8,
                                _stream(stream)))
    return out, L_out.value, s_out.value, m_out.value


def cheb_fit_sqrt(tau: float, y_lo: float, y_hi: float, degree: int) -> np.ndarray:
    """Chebyshev coefficients of tau * sqrt(y) for y in [y_lo, y_hi] mapped onto [-1, 1]."""
    lib = load_library()
    out = np.zeros(degree + 1, dtype=np.float64)
    _check(lib.fa_cheb_fit_sqrt(float(tau), float(y_lo), float(y_hi), int(degree), _ptr(out, _f64p)))
    return out


def membership_workspace(ctx_q, n_blocks: int, d: int, baby_step: int, degree: int) -> torch.Tensor:
    nbytes = int(ctx_q.lib.fa_membership_workspace_bytes(ctx_q.h, n_blocks, d, baby_step, degree))
    return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")


def membership(levels, q_r: torch.Tensor, L_q: int, s_q: float, blocks, d: int, baby_step: int, y_lo: float,
               y_hi: float, coeffs, m: int, iters: int, out: torch.Tensor | None = None,
               ws: torch.Tensor | None = None, stream=None):
    """Membership scan of a projected query against diagonal blocks encoded at level L_q;
    returns (out, level, scale, multiplier): out holds one ciphertext per block at a
    stride of the level-L_q ciphertext size."""
    top = levels[0]
    arr, nl = _levels_arg(levels)
    cq = levels[top.L - L_q]
    blocks = list(blocks)
    nb = len(blocks)
    c = _np(coeffs, np.float64)
    out = cq.new_ct(nb) if out is None else out
    ws = membership_workspace(cq, nb, d, baby_step, len(c) - 1) if ws is None else ws
    barr = (_vp * nb)(*[_dev(b) for b in blocks])
    L_out, s_out, m_out = ctypes.c_int(0), ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(top.lib.fa_membership(arr, nl, _dev(q_r), L_q, s_q, barr, nb, d, baby_step, float(y_lo), float(y_hi),
                                 _ptr(c, _f64p), len(c) - 1, int(m), iters, _dev(out), ctypes.byref(L_out),
                                 ctypes.byref(s_out), ctypes.byref(m_out), _dev(ws), ws.numel() * 8,
                                 _stream(stream)))
    return out, L_out.value, s_out.value, m_out.value
