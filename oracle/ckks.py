"""CPU oracle for the encrypted scoring path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It shares no code with the GPU library.

What it computes, and the passage of the paper each step follows:

* Scheme: RNS-CKKS with a secret-key (single-key, client-owned) setting, slot
  packing, plaintext-ciphertext products and slot rotations through Galois
  automorphisms (paper, Section 2, paragraphs "Security parameters" and
  "What CKKS gives us").
* A block of up to n/2 candidate rows stored as d diagonals (Section 2,
  "Measured prototype vs. deployment"), scored against one slot-packed query
  ciphertext with the diagonal matrix-vector method and baby-step/giant-step
  rotations; database diagonals are pre-rotated in plaintext by their giant
  step (Section 3.1, "Detail" paragraph).
* Rank reduction Enc(W^T q) with the same diagonal method and one final fold
  (Section 3.1, "How" and "Detail").
* Client finish: decrypt, decode, divide by the plaintext norm of the
  projected query (Section 3.1, "The norm problem").

Integer steps run in ``ckks_oracle.c`` (u64 residues, ``unsigned __int128``
products reduced with ``%``).  Floating-point steps (encode / decode) and all
constants derived from products of primes run here in float64 / Python big
integers.  Where the paper is silent the readings are:

* primes: the L+K largest primes below 2^50 congruent to 1 mod 2N, descending;
  the first L are the ciphertext primes, the last K the special primes;
* slot j <-> root zeta^(5^j mod 2N), zeta = exp(i pi / N); Rotate(ct, r) is a
  left roll of the slots by r and uses the automorphism X -> X^(5^r);
* encode rounds half to even in float64; integers are the parity boundary;
* hybrid key switching with alpha = K primes per digit, digit i holding primes
  i*alpha .. (i+1)*alpha-1, gadget P * Qhat_i * [Qhat_i^-1]_{Q_i}; the fast
  basis conversion has no correction term; a rotation decomposes c1 first and
  permutes second, and divides by P after every rotation except the giant
  steps of one block, which share one division (see ``bsgs_block``);
* no rescale anywhere: scales multiply.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# FA_ORACLE_LIB names another build of the same C core (the sanitizer test
# loads one built with AddressSanitizer and UndefinedBehaviorSanitizer)
LIB_PATH = os.environ.get("FA_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

PRIME_BITS = 50


# ----------------------------------------------------------------------------
# primes and parameters
# ----------------------------------------------------------------------------
def is_probable_prime(n: int) -> bool:
    """Deterministic Miller-Rabin for n < 3.3e24 (bases = first 13 primes)."""
    if n < 2:
        return False
    small = [2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37, 41]
    for p in small:
        if n % p == 0:
            return n == p
    d, s = n - 1, 0
    while d % 2 == 0:
        d //= 2
        s += 1
    for a in small:
        x = pow(a, d, n)
        if x in (1, n - 1):
            continue
        for _ in range(s - 1):
            x = x * x % n
            if x == n - 1:
                break
        else:
            return False
    return True


def find_primes(logn: int, count: int, bits: int = PRIME_BITS) -> list[int]:
    """The ``count`` largest primes below 2^bits that are 1 mod 2N, descending."""
    m = 2 << logn
    c = ((1 << bits) - 2) // m * m + 1
    out = []
    while len(out) < count:
        if is_probable_prime(c):
            out.append(c)
        c -= m
    return out


@dataclass
class Params:
    logn: int
    L: int
    K: int
    log_scale: int = 40
    primes: list = field(default_factory=list)

    def __post_init__(self):
        if not self.primes:
            self.primes = find_primes(self.logn, self.L + self.K)
        self.n = 1 << self.logn
        self.slots = self.n // 2
        self.alpha = self.K
        self.dnum = -(-self.L // self.K)
        self.q = self.primes[: self.L]
        self.p = self.primes[self.L:]

    def digit(self, i: int) -> list[int]:
        lo = i * self.alpha
        return list(range(lo, min(lo + self.alpha, self.L)))

    @property
    def P(self) -> int:
        r = 1
        for x in self.p:
            r *= x
        return r

    @property
    def Q(self) -> int:
        r = 1
        for x in self.q:
            r *= x
        return r


def _prod(xs):
    r = 1
    for x in xs:
        r *= int(x)
    return r


def ks_tables(par: Params):
    """Fast-basis-conversion constants from their definitions (big integers)."""
    np_ = par.L + par.K
    modup_inv = np.zeros((par.dnum, par.alpha), dtype=np.uint64)
    modup_hat = np.zeros((par.dnum, par.alpha, np_), dtype=np.uint64)
    for i in range(par.dnum):
        src = [par.primes[t] for t in par.digit(i)]
        D = _prod(src)
        for j, qj in enumerate(src):
            hat = D // qj
            modup_inv[i, j] = pow(hat % qj, -1, qj)
            for t in range(np_):
                modup_hat[i, j, t] = hat % par.primes[t]
    P = par.P
    down_inv = np.zeros(par.K, dtype=np.uint64)
    down_hat = np.zeros((par.K, par.L), dtype=np.uint64)
    for k, pk in enumerate(par.p):
        hat = P // pk
        down_inv[k] = pow(hat % pk, -1, pk)
        for t in range(par.L):
            down_hat[k, t] = hat % par.q[t]
    p_inv = np.array([pow(P % qt, -1, qt) for qt in par.q], dtype=np.uint64)
    return modup_inv, modup_hat, down_inv, down_hat, p_inv


def gadget_table(par: Params) -> np.ndarray:
    """[dnum][L+K]: (P * Qhat_i * [Qhat_i^-1]_{Q_i}) mod every prime of Q u P."""
    Q, P = par.Q, par.P
    out = np.zeros((par.dnum, par.L + par.K), dtype=np.uint64)
    for i in range(par.dnum):
        Qi = _prod(par.primes[t] for t in par.digit(i))
        Qhat = Q // Qi
        v = P * Qhat * pow(Qhat % Qi, -1, Qi)
        for t, m in enumerate(par.primes):
            out[i, t] = v % m
    return out


def galois_element(n: int, r: int) -> int:
    """Galois element of a left slot rotation by r: 5^r mod 2N (r taken mod N/2)."""
    return pow(5, r % (n // 2), 2 * n)


# ----------------------------------------------------------------------------
# encoding / decoding (float64)
# ----------------------------------------------------------------------------
def slot_exponents(n: int) -> np.ndarray:
    """e_j = 5^j mod 2N for j < N/2 (slot j <-> zeta^{e_j})."""
    s = n // 2
    e = np.empty(s, dtype=np.int64)
    x = 1
    for j in range(s):
        e[j] = x
        x = x * 5 % (2 * n)
    return e


def encode_real_direct(v: np.ndarray, n: int, scale: float) -> np.ndarray:
    """Unrounded coefficients by the defining sum (O(N * N/2); small N only):
    m_k = scale * (2/N) * sum_j v_j cos(pi k e_j / N)."""
    v = np.asarray(v, dtype=np.float64)
    e = slot_exponents(n)
    k = np.arange(n, dtype=np.int64)
    ang = (np.outer(k, e) % (2 * n)).astype(np.float64) * (np.pi / n)
    return scale * (2.0 / n) * (np.cos(ang) @ v)


def encode_real(v: np.ndarray, n: int, scale: float) -> np.ndarray:
    """Same values as ``encode_real_direct`` via one length-N FFT.

    With omega = exp(i pi/N): sum_j v_j (omega^{-k e_j} + omega^{k e_j}) =
    omega^{-k} sum_t Z_t exp(-2 pi i k t / N), where Z_t = v_j at t = (e_j-1)/2
    and at t = (2N-e_j-1)/2, zero nowhere else (the e_j and 2N-e_j cover every
    odd residue once)."""
    v = np.asarray(v, dtype=np.float64)
    e = slot_exponents(n)
    z = np.zeros(n, dtype=np.complex128)
    z[(e - 1) // 2] = v
    z[(2 * n - e - 1) // 2] = v
    k = np.arange(n)
    f = np.fft.fft(z) * np.exp(-1j * np.pi * k / n)
    return scale * f.real / n


def encode(v: np.ndarray, n: int, log_scale: int) -> np.ndarray:
    """Integer coefficients m = rint(2^log_scale * encode_real(v)), ties to even."""
    m = np.rint(encode_real(v, n, float(2 ** log_scale)))
    return m.astype(np.int64)


def decode_coeffs(m: np.ndarray, n: int) -> np.ndarray:
    """Slots z_j = sum_k m_k zeta^{k e_j} (complex) from real coefficients m."""
    m = np.asarray(m, dtype=np.float64)
    k = np.arange(n)
    w = np.fft.ifft(m * np.exp(1j * np.pi * k / n)) * n  # index t <-> exponent 2t+1
    e = slot_exponents(n)
    return w[(e - 1) // 2]


def crt_centered(res: np.ndarray, moduli) -> list:
    """Centred integers x with x = res[t] mod moduli[t] (big ints), per coefficient."""
    moduli = [int(m) for m in moduli]
    M = _prod(moduli)
    terms = []
    for t, m in enumerate(moduli):
        hat = M // m
        c = hat * pow(hat % m, -1, m)
        terms.append((np.asarray(res[t]).astype(object), c))
    acc = np.zeros(len(res[0]), dtype=object)
    for r, c in terms:
        acc = acc + r * c
    acc = acc % M
    half = M // 2
    return [int(x) - M if x > half else int(x) for x in acc]


def decode_residues(res: np.ndarray, par: Params, log_scale: int, nlimbs: int | None = None) -> np.ndarray:
    """Real slot values of a decrypted [L][N] residue array at scale 2^log_scale."""
    L = par.L if nlimbs is None else nlimbs
    xs = crt_centered(res[:L], par.q[:L])
    m = np.array([float(x) for x in xs]) / float(2 ** log_scale)
    # x / 2^log_scale as exact big-int division then float is not needed: the
    # float conversion of x is correctly rounded and the scale is a power of 2.
    return decode_coeffs(m, par.n).real


def to_residues(m: np.ndarray, moduli) -> np.ndarray:
    """int64 coefficients -> [len(moduli)][N] uint64 residues in [0, q)."""
    m = np.asarray(m, dtype=np.int64)
    return np.stack([np.mod(m, np.int64(q)).astype(np.uint64) for q in moduli])


# ----------------------------------------------------------------------------
# slot packings
# ----------------------------------------------------------------------------
def replicate(q: np.ndarray, slots: int) -> np.ndarray:
    """Slot s = q[s mod d]  (d must divide the slot count)."""
    d = len(q)
    assert slots % d == 0
    return np.tile(np.asarray(q, dtype=np.float64), slots // d)


def pack_rows(X: np.ndarray, slots: int, d: int) -> np.ndarray:
    """Row packing: pt_w[t*d + u] = X[w*(S/d) + t][u]; rows beyond X are zero."""
    X = np.asarray(X, dtype=np.float64)
    per = slots // d
    n_pts = -(-X.shape[0] // per)
    out = np.zeros((n_pts, slots))
    Xp = np.zeros((n_pts * per, d))
    Xp[: X.shape[0], : X.shape[1]] = X
    for w in range(n_pts):
        out[w] = Xp[w * per:(w + 1) * per].reshape(-1)
    return out


def diagonals(X: np.ndarray, slots: int, d: int) -> np.ndarray:
    """diag_j[i] = X[i][(i+j) mod d] for i < rows, 0 beyond;  [d][slots]."""
    X = np.asarray(X, dtype=np.float64)
    n = X.shape[0]
    assert n <= slots
    Xp = np.zeros((n, d))
    Xp[:, : X.shape[1]] = X
    i = np.arange(n)
    out = np.zeros((d, slots))
    for j in range(d):
        out[j, :n] = Xp[i, (i + j) % d]
    return out


def prerotate(diags: np.ndarray, B: int) -> np.ndarray:
    """pt[g][b] = roll_right(diag_{gB+b}, gB), i.e. rotation by -gB in plaintext."""
    d = diags.shape[0]
    G = d // B
    out = np.zeros((G, B, diags.shape[1]))
    for g in range(G):
        for b in range(B):
            out[g, b] = np.roll(diags[g * B + b], g * B)
    return out


def projection_diagonals(W: np.ndarray, slots: int) -> np.ndarray:
    """Hybrid diagonals of W (d_in x R, d_in = c R): e_j[s] = W[(s+j) mod d_in][s mod R], j < R."""
    d_in, R = W.shape
    s = np.arange(slots)
    return np.stack([W[(s + j) % d_in, s % R] for j in range(R)])


# ----------------------------------------------------------------------------
# integer core (C)
# ----------------------------------------------------------------------------
_u64p = ctypes.POINTER(ctypes.c_uint64)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _p(a: np.ndarray, kind=_u64p):
    return a.ctypes.data_as(kind)


def _lib():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"oracle library missing: build it with oracle/build.py ({LIB_PATH})")
    lib = ctypes.CDLL(LIB_PATH)
    lib.or_create.restype = ctypes.c_void_p
    lib.or_create.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _u64p]
    lib.or_destroy.argtypes = [ctypes.c_void_p]
    lib.or_set_ks_tables.argtypes = [ctypes.c_void_p] + [_u64p] * 5
    for name in ("or_ntt", "or_intt"):
        getattr(lib, name).argtypes = [ctypes.c_void_p, ctypes.c_int, _u64p]
    lib.or_polymul.argtypes = [ctypes.c_void_p, ctypes.c_int, _u64p, _u64p, _u64p]
    lib.or_automorph.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int,
                                 ctypes.POINTER(ctypes.c_int), _u64p, _u64p]
    lib.or_modup_digit.argtypes = [ctypes.c_void_p, ctypes.c_int, _u64p, _u64p]
    lib.or_moddown.argtypes = [ctypes.c_void_p, _u64p, _u64p]
    lib.or_keygen.argtypes = [ctypes.c_void_p, _i64p, ctypes.c_uint64, _u64p, _i64p, _u64p, _u64p]
    lib.or_encrypt.argtypes = [ctypes.c_void_p, _i64p, _u64p, _i64p, _i64p, _u64p]
    lib.or_decrypt.argtypes = [ctypes.c_void_p, _u64p, _i64p, _u64p]
    lib.or_ks_inner.argtypes = [ctypes.c_void_p, _u64p, ctypes.c_uint64, _u64p, _u64p, _u64p]
    lib.or_rotate.argtypes = [ctypes.c_void_p, _u64p, ctypes.c_uint64, _u64p, _u64p, _u64p]
    lib.or_rotate_sum.argtypes = [ctypes.c_void_p, _u64p, ctypes.c_int, _u64p,
                                  ctypes.POINTER(_u64p), ctypes.POINTER(_u64p)]
    lib.or_mul_plain.argtypes = [ctypes.c_void_p, _u64p, _u64p, _u64p]
    lib.or_bsgs_block.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, _u64p, _u64p, _u64p,
                                  ctypes.POINTER(_u64p), ctypes.POINTER(_u64p), _u64p]
    lib.or_rescale.argtypes = [ctypes.c_void_p, _u64p, ctypes.c_int, _u64p]
    lib.or_mul_const.argtypes = [ctypes.c_void_p, _u64p, ctypes.c_int, _u64p, _u64p]
    lib.or_keygen_relin.argtypes = [ctypes.c_void_p, _i64p, _u64p, _i64p, _u64p, _u64p]
    lib.or_tensor.argtypes = [ctypes.c_void_p, _u64p, _u64p, _u64p]
    lib.or_relin.argtypes = [ctypes.c_void_p, _u64p, _u64p, _u64p, _u64p]
    lib.or_bsgs_block_ct.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, _u64p, _u64p, _u64p,
                                     ctypes.POINTER(_u64p), ctypes.POINTER(_u64p), _u64p, _u64p, _u64p]
    return lib


def _c(a, dtype=np.uint64):
    return np.ascontiguousarray(a, dtype=dtype)


class Oracle:
    """The oracle's integer core for one parameter set."""

    def __init__(self, par: Params):
        self.par = par
        self.lib = _lib()
        pr = _c(par.primes)
        self.ctx = self.lib.or_create(par.logn, par.L, par.K, _p(pr))
        self._tables = [_c(t) for t in ks_tables(par)]
        self.lib.or_set_ks_tables(self.ctx, *[_p(t) for t in self._tables])
        self.gadget = _c(gadget_table(par))

    def __del__(self):
        try:
            self.lib.or_destroy(self.ctx)
        except Exception:
            pass

    # ---- ring ----
    def ntt(self, limb: int, a: np.ndarray) -> np.ndarray:
        x = _c(a).copy()
        self.lib.or_ntt(self.ctx, limb, _p(x))
        return x

    def intt(self, limb: int, a: np.ndarray) -> np.ndarray:
        x = _c(a).copy()
        self.lib.or_intt(self.ctx, limb, _p(x))
        return x

    def polymul(self, limb: int, a: np.ndarray, b: np.ndarray) -> np.ndarray:
        out = np.empty(self.par.n, dtype=np.uint64)
        self.lib.or_polymul(self.ctx, limb, _p(_c(a)), _p(_c(b)), _p(out))
        return out

    def automorph(self, g: int, x: np.ndarray, limbs) -> np.ndarray:
        x = _c(x)
        ids = np.ascontiguousarray(limbs, dtype=np.int32)
        out = np.empty_like(x)
        self.lib.or_automorph(self.ctx, g, len(ids), ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                              _p(x), _p(out))
        return out

    def modup_digit(self, i: int, c1: np.ndarray) -> np.ndarray:
        out = np.empty((self.par.L + self.par.K, self.par.n), dtype=np.uint64)
        self.lib.or_modup_digit(self.ctx, i, _p(_c(c1)), _p(out))
        return out

    def moddown(self, x: np.ndarray) -> np.ndarray:
        out = np.empty((self.par.L, self.par.n), dtype=np.uint64)
        self.lib.or_moddown(self.ctx, _p(_c(x)), _p(out))
        return out

    # ---- keys / encryption ----
    def keygen(self, s: np.ndarray, r: int, a: np.ndarray, e: np.ndarray):
        """Rotation key for a left roll by r: (b, a), each [dnum][L+K][N]."""
        par = self.par
        a = _c(a)
        assert a.shape == (par.dnum, par.L + par.K, par.n)
        b = np.empty_like(a)
        g = galois_element(par.n, r)
        self.lib.or_keygen(self.ctx, _p(_c(s, np.int64), _i64p), g, _p(a), _p(_c(e, np.int64), _i64p),
                           _p(self.gadget), _p(b))
        return b, a

    def encrypt(self, m: np.ndarray, a: np.ndarray, e: np.ndarray, s: np.ndarray) -> np.ndarray:
        par = self.par
        ct = np.empty((2, par.L, par.n), dtype=np.uint64)
        self.lib.or_encrypt(self.ctx, _p(_c(m, np.int64), _i64p), _p(_c(a)), _p(_c(e, np.int64), _i64p),
                            _p(_c(s, np.int64), _i64p), _p(ct))
        return ct

    def decrypt(self, ct: np.ndarray, s: np.ndarray) -> np.ndarray:
        out = np.empty((self.par.L, self.par.n), dtype=np.uint64)
        self.lib.or_decrypt(self.ctx, _p(_c(ct)), _p(_c(s, np.int64), _i64p), _p(out))
        return out

    # ---- homomorphic operations ----
    def ks_inner(self, c1: np.ndarray, r: int, key) -> np.ndarray:
        par = self.par
        u = np.empty((2, par.L + par.K, par.n), dtype=np.uint64)
        kb, ka = key
        self.lib.or_ks_inner(self.ctx, _p(_c(c1)), galois_element(par.n, r), _p(_c(kb)), _p(_c(ka)), _p(u))
        return u

    def rotate(self, ct: np.ndarray, r: int, key) -> np.ndarray:
        out = np.empty_like(_c(ct))
        kb, ka = key
        self.lib.or_rotate(self.ctx, _p(_c(ct)), galois_element(self.par.n, r), _p(_c(kb)), _p(_c(ka)), _p(out))
        return out

    def rotate_sum(self, ct: np.ndarray, first_shift: int, steps: int, keys: dict) -> np.ndarray:
        """ct <- ct + Rotate(ct, first_shift * 2^k) for k < steps."""
        out = _c(ct).copy()
        shifts = [first_shift << k for k in range(steps)]
        gs = _c([galois_element(self.par.n, r) for r in shifts])
        kb = [_c(keys[r][0]) for r in shifts]
        ka = [_c(keys[r][1]) for r in shifts]
        kbp = (_u64p * steps)(*[_p(x) for x in kb])
        kap = (_u64p * steps)(*[_p(x) for x in ka])
        self.lib.or_rotate_sum(self.ctx, _p(out), steps, _p(gs), kbp, kap)
        return out

    def mul_plain(self, ct: np.ndarray, pt: np.ndarray) -> np.ndarray:
        out = np.empty_like(_c(ct))
        self.lib.or_mul_plain(self.ctx, _p(_c(ct)), _p(_c(pt)), _p(out))
        return out

    # ---- encrypted database (ct x ct) ----
    def keygen_relin(self, s: np.ndarray, a: np.ndarray, e: np.ndarray):
        """Relinearisation key switching s^2 to s: (b, a), each [dnum][L+K][N],
        b_i = -a_i s + e_i + gadget_i * s^2 (the rotation keys' form with s^2 in
        place of sigma(s))."""
        par = self.par
        a = _c(a)
        assert a.shape == (par.dnum, par.L + par.K, par.n)
        b = np.empty_like(a)
        self.lib.or_keygen_relin(self.ctx, _p(_c(s, np.int64), _i64p), _p(a), _p(_c(e, np.int64), _i64p),
                                 _p(self.gadget), _p(b))
        return b, a

    def tensor(self, x: np.ndarray, y: np.ndarray) -> np.ndarray:
        """(x0, x1) x (y0, y1) = (x0 y0, x0 y1 + x1 y0, x1 y1): [3][L][N], decrypts under (1, s, s^2)."""
        out = np.empty((3, self.par.L, self.par.n), dtype=np.uint64)
        self.lib.or_tensor(self.ctx, _p(_c(x)), _p(_c(y)), _p(out))
        return out

    def relin(self, d: np.ndarray, rlk) -> np.ndarray:
        """(d0 + ModDown(u0), d1 + ModDown(u1)), (u0, u1) the key-switch inner product of d2."""
        out = np.empty((2, self.par.L, self.par.n), dtype=np.uint64)
        kb, ka = rlk
        self.lib.or_relin(self.ctx, _p(_c(d)), _p(_c(kb)), _p(_c(ka)), _p(out))
        return out

    def decrypt3(self, d: np.ndarray, s: np.ndarray) -> np.ndarray:
        """d0 + d1 s + d2 s^2 per ciphertext prime (coefficient form)."""
        par = self.par
        out = np.empty((par.L, par.n), dtype=np.uint64)
        for t, q in enumerate(par.q):
            st = to_residues(s, [q])[0]
            s2 = self.polymul(t, st, st)
            v = (d[0, t].astype(object) + self.polymul(t, d[1, t], st).astype(object)
                 + self.polymul(t, d[2, t], s2).astype(object)) % q
            out[t] = v.astype(np.uint64)
        return out

    def bsgs_block_ct(self, qrot: np.ndarray, cts: np.ndarray, B: int, G: int, keys: dict, rlk) -> np.ndarray:
        """One block against encrypted pre-rotated diagonals cts [G][B][2][L][N]: per giant
        index, the tensor sum over b, one relinearisation, then the giant sum of bsgs_block."""
        par = self.par
        cts = _c(cts)
        assert cts.shape == (G, B, 2, par.L, par.n)
        qrot = _c(qrot)
        gs = _c([0] + [galois_element(par.n, g * B) for g in range(1, G)])
        dummy = np.zeros(1, dtype=np.uint64)
        kb = [dummy] + [_c(keys[g * B][0]) for g in range(1, G)]
        ka = [dummy] + [_c(keys[g * B][1]) for g in range(1, G)]
        kbp = (_u64p * G)(*[_p(x) for x in kb])
        kap = (_u64p * G)(*[_p(x) for x in ka])
        rkb, rka = _c(rlk[0]), _c(rlk[1])
        out = np.empty((2, par.L, par.n), dtype=np.uint64)
        self.lib.or_bsgs_block_ct(self.ctx, B, G, _p(qrot), _p(cts), _p(gs), kbp, kap, _p(rkb), _p(rka), _p(out))
        return out

    # ---- rescaling and constants (the membership path) ----
    def rescale(self, ct: np.ndarray) -> np.ndarray:
        """Divide by the last ciphertext prime with rounding and drop it: [h][L][N] -> [h][L-1][N]."""
        ct = _c(ct)
        h = ct.shape[0]
        assert ct.shape[1:] == (self.par.L, self.par.n)
        out = np.empty((h, self.par.L - 1, self.par.n), dtype=np.uint64)
        self.lib.or_rescale(self.ctx, _p(ct), h, _p(out))
        return out

    def mul_const(self, ct: np.ndarray, c: int) -> np.ndarray:
        """Every polynomial times the integer c (mod each ciphertext prime)."""
        ct = _c(ct)
        cres = _c([int(c) % q for q in self.par.q])
        out = np.empty_like(ct)
        self.lib.or_mul_const(self.ctx, _p(ct), ct.shape[0], _p(cres), _p(out))
        return out

    def add_const(self, ct: np.ndarray, c: int) -> np.ndarray:
        """c0 + c (the integer c, mod each ciphertext prime, on the constant coefficient);
        the constant polynomial c encodes the value c / scale in every slot."""
        out = _c(ct).copy()
        for t, q in enumerate(self.par.q):
            out[0, t, 0] = np.uint64((int(out[0, t, 0]) + int(c)) % q)
        return out

    def add(self, x: np.ndarray, y: np.ndarray, sub: bool = False) -> np.ndarray:
        out = np.empty_like(_c(x))
        for t, q in enumerate(self.par.q):
            a, b = x[:, t].astype(object), y[:, t].astype(object)
            out[:, t] = ((a - b if sub else a + b) % q).astype(np.uint64)
        return out

    def mul(self, x: np.ndarray, y: np.ndarray, rlk) -> np.ndarray:
        """ct x ct product relinearised (no rescale): Relin(x (x) y)."""
        return self.relin(self.tensor(x, y), rlk)

    def baby_rotations(self, ct: np.ndarray, B: int, keys: dict) -> np.ndarray:
        """[B][2][L][N]: qrot[0] = ct, qrot[b] = Rotate(ct, b)."""
        out = np.empty((B,) + ct.shape, dtype=np.uint64)
        out[0] = ct
        for b in range(1, B):
            out[b] = self.rotate(ct, b, keys[b])
        return out

    def bsgs_block(self, qrot: np.ndarray, pts: np.ndarray, B: int, G: int, keys: dict) -> np.ndarray:
        """One block of the diagonal product from the baby rotations and the
        pre-rotated plaintexts pts [G][B][L][N]; giant keys at steps g*B."""
        par = self.par
        pts = _c(pts)
        assert pts.shape == (G, B, par.L, par.n)
        qrot = _c(qrot)
        gs = _c([0] + [galois_element(par.n, g * B) for g in range(1, G)])
        dummy = np.zeros(1, dtype=np.uint64)
        kb = [dummy] + [_c(keys[g * B][0]) for g in range(1, G)]
        ka = [dummy] + [_c(keys[g * B][1]) for g in range(1, G)]
        kbp = (_u64p * G)(*[_p(x) for x in kb])
        kap = (_u64p * G)(*[_p(x) for x in ka])
        out = np.empty((2, par.L, par.n), dtype=np.uint64)
        self.lib.or_bsgs_block(self.ctx, B, G, _p(qrot), _p(pts), _p(gs), kbp, kap, _p(out))
        return out


# ----------------------------------------------------------------------------
# end-to-end flows used by the tests
# ----------------------------------------------------------------------------
def encode_residues(v: np.ndarray, par: Params, log_scale: int | None = None) -> np.ndarray:
    """Slot vector -> [L][N] residues of its integer encoding."""
    ls = par.log_scale if log_scale is None else log_scale
    return to_residues(encode(v, par.n, ls), par.q)


def layout_b_pts(X: np.ndarray, par: Params, d: int, B: int) -> np.ndarray:
    """Integer plaintexts of one block (<= N/2 rows): [G][B][L][N] residues."""
    pre = prerotate(diagonals(X, par.slots, d), B)
    G = d // B
    out = np.empty((G, B, par.L, par.n), dtype=np.uint64)
    for g in range(G):
        for b in range(B):
            out[g, b] = encode_residues(pre[g, b], par)
    return out


def layout_b_coeffs(X: np.ndarray, par: Params, d: int, B: int) -> np.ndarray:
    """Integer coefficients of one block's plaintexts: [G*B][N] int64 (g-major)."""
    pre = prerotate(diagonals(X, par.slots, d), B)
    return np.stack([encode(pre[g, b], par.n, par.log_scale)
                     for g in range(pre.shape[0]) for b in range(pre.shape[1])])


def steps_for_bsgs(d: int, B: int) -> list[int]:
    return list(range(1, B)) + [g * B for g in range(1, d // B)]


# ----------------------------------------------------------------------------
# The membership (threshold) path: a chain of levels with rescaling, a
# Chebyshev series by the direct (product-formula) evaluator, and an odd
# polynomial iteration approximating the sign (the paper's face path:
# sqrt(tau^2 |q_R|^2) by a low-degree Chebyshev polynomial, then the sign of
# score - tau |q_R| after pre-scaling into [-1, 1]).
#
# A ciphertext travels with its level (number of ciphertext primes) and its
# scale (a float); a product is relinearised and then rescaled by the last
# prime of its level, so a scale s_a * s_b / q follows it.  Constants enter
# only as integers: an added constant c at scale s is round(c * s) on the
# constant coefficient, a real factor c costs a rescale as round(c * q).
# ----------------------------------------------------------------------------
class LevelChain:
    """Oracles for every level L_top..2 of one prime chain, with the secret's keys
    restricted to each level (the same restriction as the level drop)."""

    def __init__(self, top: Params, s: np.ndarray, rlk_rand, rot_rand: dict, rot_levels=None):
        self.top = top
        self.s = s
        self.orc, self.rlk, self.keys = {}, {}, {}
        a_r, e_r = rlk_rand
        for L in range(top.L, 1, -1):
            par = top if L == top.L else Params(logn=top.logn, L=L, K=top.K, log_scale=top.log_scale,
                                                 primes=top.q[:L] + top.p)
            idx = list(range(L)) + list(range(top.L, top.L + top.K))
            orc = Oracle(par)
            self.orc[L] = orc
            self.rlk[L] = orc.keygen_relin(s, a_r[:par.dnum][:, idx], e_r[:par.dnum])
            self.keys[L] = {}
            if rot_levels is None or L in rot_levels:
                for r, (a, e) in rot_rand.items():
                    self.keys[L][r] = orc.keygen(s, r, a[:par.dnum][:, idx], e[:par.dnum])

    def q(self, L: int) -> int:
        return self.top.q[L - 1]

    @staticmethod
    def drop(ct: np.ndarray, L: int) -> np.ndarray:
        return np.ascontiguousarray(ct[:, :L])

    def mul_rescale(self, x, Lx, sx, y, Ly, sy):
        """Relinearised product of two ciphertexts at the lower of their levels, then rescaled."""
        L = min(Lx, Ly)
        p = self.orc[L].mul(self.drop(x, L), self.drop(y, L), self.rlk[L])
        return self.orc[L].rescale(p), L - 1, sx * sy / float(self.q(L))


def cheb_eval(ch: LevelChain, u: np.ndarray, Lu: int, su: float, coeffs) -> tuple:
    """sum_k c_k T_k(u) for a ciphertext u (slots in [-1, 1]) by the direct evaluator:
    T_{a+b} = 2 T_a T_b - T_{a-b} with a = b = k/2 (then T_0 = 1) for even k and
    a = b + 1 for odd k (then T_1), T_2..T_d in order.  Ciphertexts are added at a common
    scale, so T_{a-b} is brought to the product's scale s_a s_b before the rescale: T_0 as
    the constant round(s_a s_b), T_1 times the integer round(s_a s_b / s_1) (no level spent).
    Then every T_k is brought to the lowest level and multiplied by round(c_k q s_u / s_k)
    -- q the prime the final rescale divides out, s_k the scale T_k carries -- so that every
    term sits at the one scale s_u q, summed with round(c_0 s_u q) and rescaled.
    Returns (ct, level, scale s_u)."""
    d = len(coeffs) - 1
    assert d >= 1
    T = {1: (u, Lu, su)}
    for k in range(2, d + 1):
        a, b = (k // 2, k // 2) if k % 2 == 0 else (k // 2 + 1, k // 2)
        L = min(T[a][1], T[b][1])
        orc = ch.orc[L]
        p = orc.mul(ch.drop(T[a][0], L), ch.drop(T[b][0], L), ch.rlk[L])
        sp = T[a][2] * T[b][2]
        p = orc.add(p, p)
        if k % 2 == 0:
            p = orc.add_const(p, -int(np.rint(sp)))
        else:
            p = orc.add(p, orc.mul_const(ch.drop(T[1][0], L), int(np.rint(sp / T[1][2]))), sub=True)
        T[k] = (orc.rescale(p), L - 1, sp / float(ch.q(L)))
    Lmin = min(v[1] for v in T.values())
    qn = ch.q(Lmin)
    orc = ch.orc[Lmin]
    acc = None
    for k in range(1, d + 1):
        term = orc.mul_const(ch.drop(T[k][0], Lmin), int(np.rint(coeffs[k] * float(qn) * (su / T[k][2]))))
        acc = term if acc is None else orc.add(acc, term)
    s_acc = su * float(qn)
    acc = orc.add_const(acc, int(np.rint(coeffs[0] * s_acc)))
    return orc.rescale(acc), Lmin - 1, s_acc / float(qn)


def sign_iter(ch: LevelChain, V: np.ndarray, L: int, s: float, m: int, iters: int) -> tuple:
    """Odd iteration towards sign(x) for x = V/m in [-1, 1]: f(x) = (3x - x^3)/2, kept with
    integer constants only -- V' = V (3 m^2 - V^2) stands for f(x) with multiplier
    m' = 2 m^3.  Two levels per iteration.  Returns (ct, level, scale, multiplier)."""
    for _ in range(iters):
        z, Lz, sz = ch.mul_rescale(V, L, s, V, L, s)
        orc = ch.orc[Lz]
        w = orc.add_const(orc.mul_const(z, -1), int(np.rint(3.0 * float(m) * float(m) * sz)))
        V, L, s = ch.mul_rescale(V, L, s, w, Lz, sz)
        m = 2 * m ** 3
    return V, L, s, m


def membership(ch: LevelChain, qr: np.ndarray, Lq: int, sq: float, blocks, d: int, B: int, y_lo: float,
               y_hi: float, coeffs, m: int, iters: int) -> tuple:
    """Membership scan (paper section 3.1, "Membership search"): whether cos(q, x_i) >= tau is
    decided under encryption as the sign of <q_R, x_i> - tau |q_R|, with |q_R| from a
    low-degree Chebyshev series of the square root and the difference pre-scaled into [-1, 1].

    qr: the projected query at level Lq, scale sq, slot s = q_R[s mod d]; blocks: each the
    [G][B][Lq][N] pre-rotated diagonal plaintexts of up to N/2 candidates at scale
    2^log_scale; coeffs: the series of tau * sqrt(y) in u = (2y - y_lo - y_hi)/(y_hi - y_lo).
      1. score_i = Rescale(diagonal product), scale s_sc = sq * 2^log_scale / q;
      2. y = |q_R|^2 in every slot: Rescale(qr * qr), then y += Rotate(y, 2^k) for 2^k < d;
      3. u = alpha (y - mid): alpha = 2/(y_hi - y_lo) changes only the scale the
         ciphertext is read at (s_y / alpha), the shift is the constant round(-mid * s_y);
      4. t = sum_k c_k T_k(u) by cheb_eval with every c_k multiplied by s_sc / s_u, so t
         holds tau |q_R| at the scores' scale s_sc;
      5. out_i = sign_iter(score_i - t (score dropped to t's level), multiplier m).
    Returns (list of per-block ciphertexts, level, scale, multiplier)."""
    orc, keys = ch.orc[Lq], ch.keys[Lq]
    G = d // B
    qrot = orc.baby_rotations(qr, B, keys)
    scores = [orc.rescale(orc.bsgs_block(qrot, _c(pts).reshape(G, B, Lq, -1), B, G, keys)) for pts in blocks]
    s_sc = sq * 2.0 ** ch.top.log_scale / float(ch.q(Lq))
    y, Ly, sy = ch.mul_rescale(qr, Lq, sq, qr, Lq, sq)
    k = 1
    while k < d:
        y = ch.orc[Ly].add(y, ch.orc[Ly].rotate(y, k, ch.keys[Ly][k]))
        k <<= 1
    alpha, mid = 2.0 / (y_hi - y_lo), 0.5 * (y_hi + y_lo)
    u = ch.orc[Ly].add_const(y, int(np.rint(-mid * sy)))
    su = sy / alpha
    ratio = s_sc / su
    t, Lt, _ = cheb_eval(ch, u, Ly, su, [c * ratio for c in coeffs])
    outs, res = [], None
    for sc in scores:
        diff = ch.orc[Lt].add(ch.drop(sc, Lt), t, sub=True)
        res = sign_iter(ch, diff, Lt, s_sc, m, iters)
        outs.append(res[0])
    return outs, res[1], res[2], res[3]
