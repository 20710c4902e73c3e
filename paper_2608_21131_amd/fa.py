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
                ("log_scale", ctypes.c_uint32)]


_vp = ctypes.c_void_p
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
    "fa_drop_level": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp]),
    "fa_ctx_primes": (ctypes.c_int, [_vp, _u64p]),
    "fa_ct_words": (ctypes.c_size_t, [_vp]),
    "fa_pt_words": (ctypes.c_size_t, [_vp]),
    "fa_key_bytes": (ctypes.c_size_t, [_vp]),
    "fa_last_error": (ctypes.c_char_p, []),
    "fa_keygen": (ctypes.c_int, [_vp, _i64p, _i32p, ctypes.c_int, _u64p, _i64p]),
    "fa_has_key": (ctypes.c_int, [_vp, ctypes.c_int]),
    "fa_set_secret": (ctypes.c_int, [_vp, _i64p]),
    "fa_encrypt": (ctypes.c_int, [_vp, _i64p, _u64p, _i64p, _vp, _vp]),
    "fa_decrypt": (ctypes.c_int, [_vp, _vp, _u64p, _vp]),
    "fa_export_coeffs": (ctypes.c_int, [_vp, _vp, ctypes.c_int, _u64p, _vp]),
    "fa_import_coeffs": (ctypes.c_int, [_vp, _u64p, ctypes.c_int, _vp, _vp]),
    "fa_encode": (ctypes.c_int, [_vp, _f64p, ctypes.c_int, ctypes.c_int, _i64p]),
    "fa_decode": (ctypes.c_int, [_vp, _u64p, ctypes.c_int, _f64p, ctypes.c_int]),
    "fa_encode_db_block": (ctypes.c_int, [_vp, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, _vp, _vp]),
    "fa_encode_db_block_int": (ctypes.c_int, [_vp, _i64p, ctypes.c_int, _vp, _vp]),
    "fa_encode_projection": (ctypes.c_int, [_vp, _f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp]),
    "fa_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "fa_score_block": (ctypes.c_int, [_vp, _vp, ctypes.POINTER(_vp), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_project_ct": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp,
                                     ctypes.c_size_t, _vp]),
    "fa_project_ct_enc": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp,
                                         ctypes.c_size_t, _vp]),
    "fa_rotate_sum": (ctypes.c_int, [_vp, _vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, ctypes.c_size_t,
                                     _vp]),
    "fa_rotate": (ctypes.c_int, [_vp, _vp, ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_prepared_words": (ctypes.c_size_t, [_vp, ctypes.c_int]),
    "fa_prepare_query": (ctypes.c_int, [_vp, _vp, ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_score_prepared": (ctypes.c_int, [_vp, _vp, _vp, ctypes.POINTER(_vp), ctypes.c_int, ctypes.c_int,
                                         ctypes.c_int, _vp, _vp, ctypes.c_size_t, _vp]),
    "fa_keygen_relin": (ctypes.c_int, [_vp, _i64p, _u64p, _i64p]),
    "fa_has_relin_key": (ctypes.c_int, [_vp]),
    "fa_encrypt_pts": (ctypes.c_int, [_vp, _vp, ctypes.c_int, _u64p, _i64p, _vp, _vp]),
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
    "fa_prepare_batch": (ctypes.c_int, [_vp, ctypes.POINTER(_vp), ctypes.c_int, ctypes.c_int, ctypes.POINTER(_vp),
                                        _vp, ctypes.c_size_t, _vp]),
    "fa_batch_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "fa_score_batch": (ctypes.c_int, [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.c_int,
                                      ctypes.POINTER(_vp), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.POINTER(_vp), _vp, ctypes.c_size_t, _vp]),
    "fa_profile": (ctypes.c_int, [_vp, ctypes.c_int]),
    "fa_profile_read": (ctypes.c_int, [_vp, _f64p]),
}

_LIB = None


def load_library(path: str = LIB_PATH):
    """Load libfa.so and declare its signatures (raises if it was never built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
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


def _dev(t: torch.Tensor):
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8
    return ctypes.c_void_p(t.data_ptr())


class Context:
    """One parameter set (ring degree, primes, tables, rotation keys) on the current GPU."""

    def __init__(self, log_n: int, L: int, K: int, log_scale: int = 40, _parent: "Context | None" = None):
        if not torch.cuda.is_available():
            raise RuntimeError("libfa needs a HIP GPU; none is visible")
        self.lib = load_library()
        self.log_n, self.L, self.K, self.log_scale = log_n, L, K, log_scale
        self.n = 1 << log_n
        self.slots = self.n // 2
        self.dnum = -(-L // K)
        h = _vp()
        if _parent is None:
            prm = _Params(log_n, L, K, log_scale)
            _check(self.lib.fa_ctx_create(ctypes.byref(prm), ctypes.byref(h)))
        else:
            _check(self.lib.fa_ctx_create_level(_parent.h, L, ctypes.byref(h)))
        self.h = h
        self.parent = _parent
        pr = np.zeros(L + K, dtype=np.uint64)
        _check(self.lib.fa_ctx_primes(self.h, _ptr(pr, _u64p)))
        self.primes = [int(x) for x in pr]
        self.ct_words = int(self.lib.fa_ct_words(self.h))
        self.pt_words = int(self.lib.fa_pt_words(self.h))

    def at_level(self, L_low: int) -> "Context":
        """Lower-level context: first L_low ciphertext primes, same special primes,
        restricted secret and rotation keys."""
        return Context(self.log_n, L_low, self.K, self.log_scale, _parent=self)

    def drop_level(self, child: "Context", ct: torch.Tensor, out: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
        out = child.new_ct() if out is None else out
        _check(self.lib.fa_drop_level(self.h, child.h, _dev(ct), _dev(out), _stream(stream)))
        return out

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
    def new_ct(self, count: int = 1) -> torch.Tensor:
        return torch.empty(count * self.ct_words, dtype=torch.float64, device="cuda")

    def new_pt(self, count: int = 1) -> torch.Tensor:
        return torch.empty(count * self.pt_words, dtype=torch.float64, device="cuda")

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

    def encrypt_pts(self, pts: torch.Tensor, n_pts: int, a, e, out: torch.Tensor | None = None,
                    stream=None) -> torch.Tensor:
        """Encrypt n_pts device plaintexts with host randomness a [n_pts][L][N], e [n_pts][N];
        returns [n_pts][2][L][N] ciphertexts (an encrypted diagonal block)."""
        a = _np(a, np.uint64)
        e = _np(e, np.int64)
        assert a.size == n_pts * self.L * self.n and e.size == n_pts * self.n
        out = self.new_ct(n_pts) if out is None else out
        _check(self.lib.fa_encrypt_pts(self.h, _dev(pts), n_pts, _ptr(a, _u64p), _ptr(e, _i64p), _dev(out),
                                       _stream(stream)))
        return out

    def set_secret(self, s):
        s = _np(s, np.int64)
        _check(self.lib.fa_set_secret(self.h, _ptr(s, _i64p)))

    def encrypt(self, m, a, e, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        out = self.new_ct() if out is None else out
        m, a, e = _np(m, np.int64), _np(a, np.uint64), _np(e, np.int64)
        _check(self.lib.fa_encrypt(self.h, _ptr(m, _i64p), _ptr(a, _u64p), _ptr(e, _i64p), _dev(out),
                                   _stream(stream)))
        return out

    def decrypt(self, ct: torch.Tensor, stream=None) -> np.ndarray:
        out = np.empty((self.L, self.n), dtype=np.uint64)
        _check(self.lib.fa_decrypt(self.h, _dev(ct), _ptr(out, _u64p), _stream(stream)))
        return out

    def export(self, buf: torch.Tensor, n_polys: int, stream=None) -> np.ndarray:
        out = np.empty((n_polys, self.L, self.n), dtype=np.uint64)
        _check(self.lib.fa_export_coeffs(self.h, _dev(buf), n_polys, _ptr(out, _u64p), _stream(stream)))
        return out

    def import_coeffs(self, coeffs, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """The inverse of export: canonical [n_polys][L][N] residues into a device buffer."""
        c = _np(coeffs, np.uint64)
        if c.ndim != 3 or c.shape[1:] != (self.L, self.n):
            raise ValueError(f"coefficients must be [n_polys][{self.L}][{self.n}]")
        out = torch.empty(c.size, dtype=torch.float64, device="cuda") if out is None else out
        _check(self.lib.fa_import_coeffs(self.h, _ptr(c, _u64p), c.shape[0], _dev(out), _stream(stream)))
        return out

    def save_buffers(self, path: str, buffers: dict) -> None:
        """Save device buffers {name: (tensor, n_polys)} (enrolled blocks, ciphertexts) in canonical
        coefficient form with a header naming this context's ring, primes and each buffer's size."""
        import json
        header = {"format": "fa-coeffs-1", "log_n": self.log_n, "L": self.L, "K": self.K,
                  "primes": [int(p) for p in self.primes], "buffers": {k: int(v[1]) for k, v in buffers.items()}}
        arrays = {"header": np.frombuffer(json.dumps(header).encode(), dtype=np.uint8)}
        for name, (buf, n_polys) in buffers.items():
            arrays["buf_" + name] = self.export(buf, n_polys)
        np.savez(path, **arrays)

    def load_buffers(self, path: str) -> dict:
        """Load what save_buffers wrote into new device buffers {name: tensor}; the file must come
        from a context with the same ring degree and primes."""
        import json
        with np.load(path, allow_pickle=False) as z:
            header = json.loads(bytes(z["header"]).decode())
            mine = {"log_n": self.log_n, "L": self.L, "K": self.K, "primes": [int(p) for p in self.primes]}
            if header.get("format") != "fa-coeffs-1" or any(header.get(k) != v for k, v in mine.items()):
                raise ValueError(f"{path}: saved for another context ({header.get('log_n')}, {header.get('L')}, "
                                 f"{header.get('K')})")
            return {name: self.import_coeffs(z["buf_" + name]) for name in header["buffers"]}

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
                        out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        rows = _np(rows, np.float32)
        n_rows, dim = rows.shape
        n_pts = d if layout == LAYOUT_DIAG else -(-n_rows // (self.slots // d))
        out = self.new_pt(n_pts) if out is None else out
        _check(self.lib.fa_encode_db_block(self.h, _ptr(rows, _f32p), n_rows, dim, d, layout, baby_step,
                                           _dev(out), _stream(stream)))
        return out

    def encode_projection(self, W, baby_step: int, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        W = _np(W, np.float32)
        d_in, r = W.shape
        out = self.new_pt(r) if out is None else out
        _check(self.lib.fa_encode_projection(self.h, _ptr(W, _f32p), d_in, r, baby_step, _dev(out), _stream(stream)))
        return out

    def encode_db_block_int(self, coeffs, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        c = _np(coeffs, np.int64).reshape(-1, self.n)
        out = self.new_pt(c.shape[0]) if out is None else out
        _check(self.lib.fa_encode_db_block_int(self.h, _ptr(c, _i64p), c.shape[0], _dev(out), _stream(stream)))
        return out

    # ---- scoring ----
    def score_block(self, q: torch.Tensor, blocks, d: int, layout: int, baby_step: int = 1,
                    out: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        blocks = list(blocks)
        nb = len(blocks)
        out = self.new_ct(nb) if out is None else out
        if ws is None and layout == LAYOUT_DIAG:
            ws = self.workspace(OP_SCORE, nb, d, baby_step)
        elif ws is None and layout == LAYOUT_DIAG_ENC:
            ws = self.workspace(OP_SCORE_ENC, nb, d, baby_step)
        arr = (_vp * nb)(*[ctypes.c_void_p(b.data_ptr()) for b in blocks])
        ws_p, ws_b = (_dev(ws), ws.numel() * 8) if ws is not None else (ctypes.c_void_p(0), 0)
        _check(self.lib.fa_score_block(self.h, _dev(q), arr, nb, d, layout, baby_step, _dev(out), ws_p, ws_b,
                                       _stream(stream)))
        return out

    def prepare_query(self, q: torch.Tensor, baby_step: int, out: torch.Tensor | None = None,
                      ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        words = int(self.lib.fa_prepared_words(self.h, baby_step))
        out = torch.empty(words, dtype=torch.float64, device="cuda") if out is None else out
        ws = self.workspace(OP_PREPARE, 1, baby_step, baby_step) if ws is None else ws
        _check(self.lib.fa_prepare_query(self.h, _dev(q), baby_step, _dev(out), _dev(ws), ws.numel() * 8,
                                         _stream(stream)))
        return out

    def prepare_batch_workspace(self, n_q: int, baby_step: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_prepare_batch_workspace_bytes(self.h, n_q, baby_step))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def prepare_batch(self, qs, baby_step: int, outs=None, ws: torch.Tensor | None = None, stream=None) -> list:
        """Prepare several queries together; outs[j] equals prepare_query(qs[j], baby_step)."""
        qs = list(qs)
        nq = len(qs)
        words = int(self.lib.fa_prepared_words(self.h, baby_step))
        outs = [torch.empty(words, dtype=torch.float64, device="cuda") for _ in range(nq)] if outs is None \
            else list(outs)
        if len(outs) != nq:
            raise ValueError("one prepared buffer per query")
        ws = self.prepare_batch_workspace(nq, baby_step) if ws is None else ws
        qa = (_vp * nq)(*[ctypes.c_void_p(x.data_ptr()) for x in qs])
        oa = (_vp * nq)(*[ctypes.c_void_p(x.data_ptr()) for x in outs])
        _check(self.lib.fa_prepare_batch(self.h, qa, nq, baby_step, oa, _dev(ws), ws.numel() * 8, _stream(stream)))
        return outs

    def score_prepared(self, q: torch.Tensor, prep: torch.Tensor, blocks, d: int, baby_step: int,
                       out: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        blocks = list(blocks)
        nb = len(blocks)
        out = self.new_ct(nb) if out is None else out
        ws = self.workspace(OP_SCORE_PREPARED, nb, d, baby_step) if ws is None else ws
        arr = (_vp * nb)(*[ctypes.c_void_p(b.data_ptr()) for b in blocks])
        _check(self.lib.fa_score_prepared(self.h, _dev(q), _dev(prep), arr, nb, d, baby_step, _dev(out), _dev(ws),
                                          ws.numel() * 8, _stream(stream)))
        return out

    def batch_workspace(self, n_q: int, n_blocks: int, d: int, baby_step: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_batch_workspace_bytes(self.h, n_q, n_blocks, d, baby_step))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def score_batch(self, qs, preps, blocks, d: int, baby_step: int, outs=None, ws: torch.Tensor | None = None,
                    stream=None) -> list:
        """Score several prepared queries against the same blocks, one plaintext pass per
        group of up to four queries; outs[j] equals score_prepared(qs[j], preps[j], ...)."""
        qs, preps, blocks = list(qs), list(preps), list(blocks)
        nq, nb = len(qs), len(blocks)
        if len(preps) != nq:
            raise ValueError("one prepared rotation set per query")
        outs = [self.new_ct(nb) for _ in range(nq)] if outs is None else list(outs)
        ws = self.batch_workspace(nq, nb, d, baby_step) if ws is None else ws
        qa = (_vp * nq)(*[ctypes.c_void_p(x.data_ptr()) for x in qs])
        pa = (_vp * nq)(*[ctypes.c_void_p(x.data_ptr()) for x in preps])
        oa = (_vp * nq)(*[ctypes.c_void_p(x.data_ptr()) for x in outs])
        ba = (_vp * nb)(*[ctypes.c_void_p(b.data_ptr()) for b in blocks])
        _check(self.lib.fa_score_batch(self.h, qa, pa, nq, ba, nb, d, baby_step, oa, _dev(ws), ws.numel() * 8,
                                       _stream(stream)))
        return outs

    # ---- the membership path ----
    def chain_workspace(self, degree: int) -> torch.Tensor:
        nbytes = int(self.lib.fa_chain_workspace_bytes(self.h, degree))
        return torch.empty(max(1, nbytes // 8 + 32), dtype=torch.float64, device="cuda")

    def rescale(self, lo: "Context", ct: torch.Tensor, n_polys: int = 2, out: torch.Tensor | None = None,
                ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """round(ct / last prime) at the next level down (lo = this context minus that prime)."""
        out = torch.empty(n_polys * lo.L * lo.n, dtype=torch.float64, device="cuda") if out is None else out
        if ws is None:
            ws = torch.empty(n_polys * self.L * self.n + 32, dtype=torch.float64, device="cuda")
        _check(self.lib.fa_rescale(self.h, lo.h, _dev(ct), n_polys, _dev(out), _dev(ws), ws.numel() * 8,
                                   _stream(stream)))
        return out

    def mul_ct(self, x: torch.Tensor, y: torch.Tensor, out: torch.Tensor | None = None, stream=None):
        out = self.new_ct() if out is None else out
        ws = self.chain_workspace(1)
        _check(self.lib.fa_mul_ct(self.h, _dev(x), _dev(y), _dev(out), _dev(ws), ws.numel() * 8, _stream(stream)))
        return out

    def ct_add(self, x, y, out=None, subtract: bool = False, stream=None):
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_add(self.h, _dev(x), _dev(y), _dev(out), 1 if subtract else 0, _stream(stream)))
        return out

    def ct_mul_const(self, x, k: int, out=None, stream=None):
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_mul_const(self.h, _dev(x), int(k), _dev(out), _stream(stream)))
        return out

    def ct_add_const(self, x, k: int, out=None, stream=None):
        out = self.new_ct() if out is None else out
        _check(self.lib.fa_ct_add_const(self.h, _dev(x), float(k), _dev(out), _stream(stream)))
        return out

    def project_ct(self, q: torch.Tensor, w_pts: torch.Tensor, d_in: int, r: int, baby_step: int,
                   out: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_PROJECT, 1, r, baby_step) if ws is None else ws
        _check(self.lib.fa_project_ct(self.h, _dev(q), _dev(w_pts), d_in, r, baby_step, _dev(out), _dev(ws),
                                      ws.numel() * 8, _stream(stream)))
        return out

    def project_ct_enc(self, q: torch.Tensor, w_cts: torch.Tensor, d_in: int, r: int, baby_step: int,
                       out: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """The projection with W's r diagonals encrypted (fa_encrypt_pts of project_ct's plaintexts)."""
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_PROJECT_ENC, 1, r, baby_step) if ws is None else ws
        _check(self.lib.fa_project_ct_enc(self.h, _dev(q), _dev(w_cts), d_in, r, baby_step, _dev(out), _dev(ws),
                                          ws.numel() * 8, _stream(stream)))
        return out

    def rotate_sum(self, cts: torch.Tensor, n_cts: int, first_shift: int, n_steps: int,
                   ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        ws = self.workspace(OP_ROTATE_SUM, n_cts) if ws is None else ws
        _check(self.lib.fa_rotate_sum(self.h, _dev(cts), n_cts, first_shift, n_steps, _dev(ws), ws.numel() * 8,
                                      _stream(stream)))
        return cts

    def profile(self, enable: bool = True):
        _check(self.lib.fa_profile(self.h, 1 if enable else 0))

    def profile_read(self) -> dict:
        ms = np.zeros(4, dtype=np.float64)
        _check(self.lib.fa_profile_read(self.h, _ptr(ms, _f64p)))
        return {"baby_ms": ms[0], "mac_ms": ms[1], "giant_ms": ms[2], "total_ms": ms[3]}

    def rotate(self, ct: torch.Tensor, step: int, out: torch.Tensor | None = None,
               ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        out = self.new_ct() if out is None else out
        ws = self.workspace(OP_ROTATE, 1) if ws is None else ws
        _check(self.lib.fa_rotate(self.h, _dev(ct), step, _dev(out), _dev(ws), ws.numel() * 8, _stream(stream)))
        return out


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
    barr = (_vp * nb)(*[ctypes.c_void_p(b.data_ptr()) for b in blocks])
    L_out, s_out, m_out = ctypes.c_int(0), ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(top.lib.fa_membership(arr, nl, _dev(q_r), L_q, s_q, barr, nb, d, baby_step, float(y_lo), float(y_hi),
                                 _ptr(c, _f64p), len(c) - 1, int(m), iters, _dev(out), ctypes.byref(L_out),
                                 ctypes.byref(s_out), ctypes.byref(m_out), _dev(ws), ws.numel() * 8,
                                 _stream(stream)))
    return out, L_out.value, s_out.value, m_out.value
