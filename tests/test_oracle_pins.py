"""Pins for the CPU oracle: each test checks it against something other than
itself -- schoolbook arithmetic, closed forms, invariants, big-integer
identities, float64 plaintext results -- so that a dropped term, a wrong sign
or index, or a transposed operand anywhere in the oracle fails one of them.

CPU only (no GPU marker)."""
import numpy as np
import pytest

from oracle import ckks
from paper_2608_21131_amd import gen


# ----------------------------------------------------------------------------
# helpers that are NOT the oracle's code: schoolbook / big-int definitions
# ----------------------------------------------------------------------------
def schoolbook_negacyclic(a, b, q):
    """c = a*b mod (X^N + 1, q) by the O(N^2) definition with Python ints."""
    n = len(a)
    c = [0] * n
    for i in range(n):
        ai = int(a[i])
        if ai == 0:
            continue
        for j in range(n):
            k = i + j
            v = ai * int(b[j])
            if k < n:
                c[k] += v
            else:
                c[k - n] -= v
    return np.array([x % q for x in c], dtype=np.uint64)


def small_primes_upto(m):
    sieve = np.ones(m + 1, dtype=bool)
    sieve[:2] = False
    for i in range(2, int(m ** 0.5) + 1):
        if sieve[i]:
            sieve[i * i::i] = False
    return np.nonzero(sieve)[0].astype(np.int64)


_SMALL = None


def trial_division_prime(p):
    """Primality by trial division up to sqrt(p) (independent of Miller-Rabin)."""
    global _SMALL
    if _SMALL is None:
        _SMALL = small_primes_upto(1 << 25)
    lim = int(p ** 0.5) + 1
    ds = _SMALL[_SMALL <= lim]
    return not np.any(np.int64(p) % ds == 0)


@pytest.fixture(scope="module")
def tiny():
    """A tiny ring for schoolbook checks (N = 32)."""
    par = ckks.Params(logn=5, L=3, K=1)
    return par, ckks.Oracle(par)


@pytest.fixture(scope="module")
def small():
    """A small ring for end-to-end checks (N = 1024, 3 + 1 primes)."""
    par = ckks.Params(logn=10, L=3, K=1)
    return par, ckks.Oracle(par)


@pytest.fixture(scope="module")
def small4():
    """N = 2048 with 4 + 2 primes: two primes per digit."""
    par = ckks.Params(logn=11, L=4, K=2)
    return par, ckks.Oracle(par)


def keyset(orc, s, steps, wid=0):
    par = orc.par
    keys = {}
    for r in steps:
        a = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, r), par.primes, par.dnum, par.n)
        e = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, r), (par.dnum, par.n))
        keys[r] = orc.keygen(s, r, a, e)
    return keys


def enc(orc, v, s, log_scale=40, wid=0):
    par = orc.par
    m = ckks.encode(v, par.n, log_scale)
    a = gen.uniform_residues(gen.rng(wid, gen.STREAM_ENC_A), par.q, 1, par.n)[0]
    e = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_ENC_E), par.n)
    return orc.encrypt(m, a, e, s)


def dec(orc, ct, s, log_scale):
    return ckks.decode_residues(orc.decrypt(ct, s), orc.par, log_scale)


# ----------------------------------------------------------------------------
# primes
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("logn,count", [(13, 4), (15, 10), (16, 15)])
def test_primes_are_the_largest_ntt_primes_below_2_50(logn, count):
    ps = ckks.find_primes(logn, count)
    m = 2 << logn
    assert ps == sorted(ps, reverse=True)
    for p in ps:
        assert p < (1 << 50) and p.bit_length() == 50
        assert p % m == 1
        assert trial_division_prime(p)
    # nothing was skipped: every candidate 1 mod 2N above the smallest is either listed or composite
    c = ((1 << 50) - 2) // m * m + 1
    while c >= ps[-1]:
        if c not in ps:
            assert not trial_division_prime(c), c
        c -= m


def test_golden_primes_file():
    """tests/golden/primes.txt (written by tests/golden/make_golden.py) matches."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "primes.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    for row in rows:
        logn, L, K = int(row[0]), int(row[1]), int(row[2])
        ps = [int(x, 16) for x in row[3:]]
        assert ps == ckks.find_primes(logn, L + K)


# ----------------------------------------------------------------------------
# ring arithmetic
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("logn", [3, 4, 5, 6])
def test_ring_product_equals_schoolbook_negacyclic(logn):
    par = ckks.Params(logn=logn, L=2, K=1)
    orc = ckks.Oracle(par)
    g = np.random.default_rng(logn)
    for limb in range(3):
        q = par.primes[limb]
        a = g.integers(0, q, par.n, dtype=np.uint64)
        b = g.integers(0, q, par.n, dtype=np.uint64)
        assert np.array_equal(orc.polymul(limb, a, b), schoolbook_negacyclic(a, b, q))
    # small signed polynomials: the RNS product, lifted by CRT, is the integer product
    a = g.integers(-1000, 1000, par.n)
    b = g.integers(-1000, 1000, par.n)
    prod = [orc.polymul(t, np.mod(a, par.primes[t]).astype(np.uint64),
                        np.mod(b, par.primes[t]).astype(np.uint64)) for t in range(2)]
    lifted = ckks.crt_centered(np.stack(prod), par.primes[:2])
    exact = np.zeros(par.n, dtype=object)
    for i in range(par.n):
        for j in range(par.n):
            k = i + j
            if k < par.n:
                exact[k] += int(a[i]) * int(b[j])
            else:
                exact[k - par.n] -= int(a[i]) * int(b[j])
    assert [int(x) for x in exact] == lifted


def test_transform_is_evaluation_at_odd_powers(tiny):
    par, orc = tiny
    n = par.n
    for limb in range(par.L + par.K):
        q = par.primes[limb]
        x = np.zeros(n, dtype=np.uint64)
        x[1] = 1
        A = orc.ntt(limb, x)  # A[j] = psi^{2j+1}
        psi = int(A[0])
        assert pow(psi, n, q) == q - 1  # primitive 2N-th root
        for k in (0, 1, 3, n - 1):
            mono = np.zeros(n, dtype=np.uint64)
            mono[k] = 1
            Ak = orc.ntt(limb, mono)
            assert all(int(Ak[j]) == pow(psi, k * (2 * j + 1), q) for j in range(n))
        r = np.random.default_rng(limb).integers(0, q, n, dtype=np.uint64)
        assert np.array_equal(orc.intt(limb, orc.ntt(limb, r)), r)


# ----------------------------------------------------------------------------
# automorphisms
# ----------------------------------------------------------------------------
def test_automorphism_definition_and_homomorphism(tiny):
    par, orc = tiny
    n, q = par.n, par.primes[0]
    g = np.random.default_rng(5)
    a = g.integers(0, q, n, dtype=np.uint64)
    b = g.integers(0, q, n, dtype=np.uint64)
    for gal in (5, 25, 2 * n - 1, 3):
        sa = orc.automorph(gal, a[None], [0])[0]
        # definition: a(X^gal) reduced mod X^N + 1, written out with Python ints
        ref = [0] * n
        for j in range(n):
            t = gal * j % (2 * n)
            if t < n:
                ref[t] = (ref[t] + int(a[j])) % q
            else:
                ref[t - n] = (ref[t - n] - int(a[j])) % q
        assert [int(x) for x in sa] == ref
        sb = orc.automorph(gal, b[None], [0])[0]
        ab = schoolbook_negacyclic(a, b, q)
        assert np.array_equal(orc.automorph(gal, ab[None], [0])[0], schoolbook_negacyclic(sa, sb, q))
    # composition and the order of 5
    s5 = orc.automorph(5, a[None], [0])
    s25 = orc.automorph(25, a[None], [0])
    assert np.array_equal(orc.automorph(5, s5, [0]), s25)
    assert pow(5, n // 2, 2 * n) == 1
    assert np.array_equal(orc.automorph(pow(5, n // 2, 2 * n), a[None], [0])[0], a)


# ----------------------------------------------------------------------------
# encoding
# ----------------------------------------------------------------------------
def test_encode_constant_vector_is_constant_polynomial():
    n = 256
    for c in (0.25, -0.7, 1.0):
        m = ckks.encode(np.full(n // 2, c), n, 40)
        assert m[0] == np.rint(c * 2 ** 40)
        assert np.all(m[1:] == 0)


@pytest.mark.parametrize("n", [16, 64, 512])
def test_encode_fft_matches_defining_sum(n):
    v = np.random.default_rng(n).standard_normal(n // 2)
    fast = ckks.encode_real(v, n, 2.0 ** 40)
    direct = ckks.encode_real_direct(v, n, 2.0 ** 40)
    assert np.max(np.abs(fast - direct)) < 1e-3  # values are ~2^40: relative 1e-15


def test_slot_product_is_ring_product():
    """decode(encode(u) * encode(v)) / scale^2 = u * v  (canonical embedding is a ring map)."""
    n = 64
    g = np.random.default_rng(7)
    u, v = g.standard_normal(n // 2), g.standard_normal(n // 2)
    mu, mv = ckks.encode(u, n, 30), ckks.encode(v, n, 30)
    prod = np.zeros(n, dtype=object)
    for i in range(n):
        for j in range(n):
            k = i + j
            t = int(mu[i]) * int(mv[j])
            if k < n:
                prod[k] += t
            else:
                prod[k - n] -= t
    z = ckks.decode_coeffs(np.array([float(x) for x in prod]) / 2.0 ** 60, n)
    assert np.max(np.abs(z.real - u * v)) < 1e-6
    assert np.max(np.abs(z.imag)) < 1e-6


def test_rotation_is_automorphism_by_power_of_5(small):
    par, orc = small
    n = par.n
    v = np.random.default_rng(3).standard_normal(n // 2)
    m = ckks.encode(v, n, 40)
    res = ckks.to_residues(m, par.q)
    for r in (1, 7, n // 4):
        gal = ckks.galois_element(n, r)
        rot = orc.automorph(gal, res, list(range(par.L)))
        z = ckks.decode_residues(rot, par, 40)
        assert np.max(np.abs(z - np.roll(v, -r))) < 1e-9


def test_decode_encode_roundtrip():
    n = 4096
    v = np.random.default_rng(11).uniform(-1, 1, n // 2)
    z = ckks.decode_coeffs(ckks.encode(v, n, 40).astype(np.float64) / 2.0 ** 40, n)
    assert np.max(np.abs(z.real - v)) < n * 2.0 ** -41


# ----------------------------------------------------------------------------
# basis conversion
# ----------------------------------------------------------------------------
def test_modup_conv_is_lift_plus_small_multiple(small4):
    """Conv_{D_i -> t}(x) = x + u * D_i (mod t) with one integer 0 <= u < |D_i| for all t."""
    par, orc = small4
    g = np.random.default_rng(17)
    c1 = np.stack([g.integers(0, q, par.n, dtype=np.uint64) for q in par.q])
    for i in range(par.dnum):
        ext = orc.modup_digit(i, c1)
        dig = par.digit(i)
        D = 1
        for t in dig:
            D *= par.primes[t]
        xs = ckks.crt_centered(c1[dig], [par.primes[t] for t in dig])
        xs = [x % D for x in xs]  # canonical lift in [0, D)
        for t in dig:
            assert np.array_equal(ext[t], c1[t])
        others = [t for t in range(par.L + par.K) if t not in dig]
        for k in range(0, par.n, 97):
            us = None
            for t in others:
                cand = {u for u in range(len(dig)) if (xs[k] + u * D) % par.primes[t] == int(ext[t, k])}
                us = cand if us is None else us & cand
            assert us, (i, k)


def test_moddown_inverts_multiplication_by_P(small4):
    par, orc = small4
    g = np.random.default_rng(19)
    x = np.stack([g.integers(0, q, par.n, dtype=np.uint64) for q in par.q])
    P = par.P
    y = np.stack([(x[t].astype(object) * P % par.primes[t]).astype(np.uint64) if t < par.L
                  else np.zeros(par.n, dtype=np.uint64) for t in range(par.L + par.K)])
    assert np.array_equal(orc.moddown(y), x)
    # y = P x + e with 0 <= e < P  ->  ModDown(y) = x - u, 0 <= u < K
    Q = par.Q
    xi = ckks.crt_centered(x, par.q)
    es = [int(v) for v in g.integers(0, 2 ** 62, par.n)]
    es = [(e * 7919 + 12345) % P for e in es]
    y = np.stack([np.array([(P * xi[k] + es[k]) % par.primes[t] for k in range(par.n)], dtype=np.uint64)
                  for t in range(par.L + par.K)])
    out = ckks.crt_centered(orc.moddown(y), par.q)
    for k in range(par.n):
        assert (xi[k] - out[k]) % Q in range(par.K), k


# ----------------------------------------------------------------------------
# encryption, key switching
# ----------------------------------------------------------------------------
def test_encrypt_decrypt_roundtrip(small):
    par, orc = small
    s = gen.ternary_secret(gen.rng(1, gen.STREAM_SECRET), par.n)
    v = np.random.default_rng(2).uniform(-1, 1, par.slots)
    ct = enc(orc, v, s, wid=1)
    assert np.max(np.abs(dec(orc, ct, s, 40) - v)) < 1e-6
    # decryption with the wrong key is garbage
    s2 = gen.ternary_secret(gen.rng(2, gen.STREAM_SECRET), par.n)
    assert np.max(np.abs(dec(orc, ct, s2, 40) - v)) > 1.0


@pytest.mark.parametrize("which", ["small", "small4"])
def test_rotation_decrypts_to_rolled_slots(which, request):
    par, orc = request.getfixturevalue(which)
    s = gen.ternary_secret(gen.rng(3, gen.STREAM_SECRET), par.n)
    v = np.random.default_rng(4).uniform(-1, 1, par.slots)
    ct = enc(orc, v, s, wid=3)
    steps = [1, 2, 5, par.slots // 2]
    keys = keyset(orc, s, steps, wid=3)
    for r in steps:
        z = dec(orc, orc.rotate(ct, r, keys[r]), s, 40)
        assert np.max(np.abs(z - np.roll(v, -r))) < 1e-6, r
    # composition
    z = dec(orc, orc.rotate(orc.rotate(ct, 1, keys[1]), 5, keys[5]), s, 40)
    assert np.max(np.abs(z - np.roll(v, -6))) < 1e-6
    # rotation by the slot count is the identity automorphism
    kS = keyset(orc, s, [par.slots], wid=3)
    z = dec(orc, orc.rotate(ct, par.slots, kS[par.slots]), s, 40)
    assert np.max(np.abs(z - v)) < 1e-6


def test_key_inner_product_carries_P_times_rotated_c1(small4):
    """u0 + u1*s = P * sigma(c1) * sigma(s) + sum_i sigma(ext_i) e_i   (mod P*Q),

    where c1 is lifted to [0, Q) and the last term is bounded by
    N * 19 * alpha * max(Q_i) * dnum; a wrong gadget, basis conversion or key
    term leaves a residue of size ~P*Q instead."""
    par, orc = small4
    n = par.n
    s = gen.ternary_secret(gen.rng(5, gen.STREAM_SECRET), n)
    keys = keyset(orc, s, [3], wid=5)
    g = np.random.default_rng(23)
    c1 = np.stack([g.integers(0, q, n, dtype=np.uint64) for q in par.q])
    u = orc.ks_inner(c1, 3, keys[3])
    gal = ckks.galois_element(n, 3)
    allp = list(range(par.L + par.K))
    s_res = ckks.to_residues(s, par.primes)
    ss = orc.automorph(gal, s_res, allp)
    lhs = [(u[0, t].astype(object) + orc.polymul(t, u[1, t], s_res[t]).astype(object)) % par.primes[t]
           for t in allp]
    c1_int = [x % par.Q for x in ckks.crt_centered(c1, par.q)]
    c1_res = np.stack([np.array([x % par.primes[t] for x in c1_int], dtype=np.uint64) for t in allp])
    sc1 = orc.automorph(gal, c1_res, allp)
    rhs = [(orc.polymul(t, sc1[t], ss[t]).astype(object) * (par.P % par.primes[t])) % par.primes[t]
           for t in allp]
    diff = np.stack([((lhs[t] - rhs[t]) % par.primes[t]).astype(np.uint64) for t in allp])
    d_int = ckks.crt_centered(diff, par.primes)
    qi_max = max(ckks._prod(par.primes[t] for t in par.digit(i)) for i in range(par.dnum))
    bound = n * 19 * par.alpha * qi_max * par.dnum
    assert max(abs(x) for x in d_int) < bound
    assert max(abs(x) for x in d_int) > 0


# ----------------------------------------------------------------------------
# plaintext identities of the packings (float64, no encryption)
# ----------------------------------------------------------------------------
def test_layout_b_plaintext_identity():
    S, d, B = 256, 32, 8
    g = np.random.default_rng(29)
    X = g.standard_normal((200, d))
    q = g.standard_normal(d)
    diags = ckks.diagonals(X, S, d)
    pre = ckks.prerotate(diags, B)
    qs = ckks.replicate(q, S)
    out = np.zeros(S)
    for gg in range(d // B):
        acc = sum(pre[gg, b] * np.roll(qs, -b) for b in range(B))
        out += np.roll(acc, -gg * B)
    assert np.allclose(out[:200], X @ q, atol=1e-12)
    assert np.allclose(out[200:], 0, atol=1e-12)


def test_layout_a_plaintext_identity():
    S, d = 256, 16
    g = np.random.default_rng(31)
    X = g.standard_normal((40, d))
    q = g.standard_normal(d)
    pts = ckks.pack_rows(X, S, d)
    qs = ckks.replicate(q, S)
    scores = []
    for w in range(pts.shape[0]):
        z = pts[w] * qs
        for k in range(int(np.log2(d))):
            z = z + np.roll(z, -(1 << k))
        scores.extend(z[:: d])
    assert np.allclose(np.array(scores)[:40], X @ q, atol=1e-12)


def test_projection_plaintext_identity():
    S, d_in, R, B = 2048, 64, 16, 4
    g = np.random.default_rng(37)
    W = g.standard_normal((d_in, R))
    q = g.standard_normal(d_in)
    e = ckks.projection_diagonals(W, S)
    pre = ckks.prerotate(e, B)
    qs = ckks.replicate(q, S)
    z = np.zeros(S)
    for gg in range(R // B):
        acc = sum(pre[gg, b] * np.roll(qs, -b) for b in range(B))
        z += np.roll(acc, -gg * B)
    for k in range(int(np.log2(d_in // R))):
        z = z + np.roll(z, -(R << k))
    assert np.allclose(z, np.tile(W.T @ q, S // R), atol=1e-10)


# ----------------------------------------------------------------------------
# end to end: decrypted scores against float64 inner products
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("B", [1, 4, 16])
def test_layout_b_scores_match_float64(small, B):
    par, orc = small
    d, rows = 16, 300
    s = gen.ternary_secret(gen.rng(6, gen.STREAM_SECRET), par.n)
    X = gen.gaussian_unit_rows(gen.rng(6, gen.STREAM_DB), rows, d)
    q = gen.gaussian_unit_rows(gen.rng(6, gen.STREAM_QUERY), 1, d)[0]
    ct = enc(orc, ckks.replicate(q, par.slots), s, wid=6)
    keys = keyset(orc, s, ckks.steps_for_bsgs(d, B), wid=6)
    qrot = orc.baby_rotations(ct, B, keys)
    out = orc.bsgs_block(qrot, ckks.layout_b_pts(X, par, d, B), B, d // B, keys)
    z = dec(orc, out, s, 80)
    assert np.max(np.abs(z[:rows] - X @ q)) < 1e-4
    assert np.max(np.abs(z[rows:])) < 1e-4


def test_layout_b_zero_padding_is_exact_cosine(small):
    """96-d vectors zero-padded to 128: the score is the 96-d cosine."""
    par, orc = small
    rows = 40
    s = gen.ternary_secret(gen.rng(7, gen.STREAM_SECRET), par.n)
    X = gen.gaussian_unit_rows(gen.rng(7, gen.STREAM_DB), rows, 96)
    q = gen.gaussian_unit_rows(gen.rng(7, gen.STREAM_QUERY), 1, 96)[0]
    qp = np.zeros(128)
    qp[:96] = q
    ct = enc(orc, ckks.replicate(qp, par.slots), s, wid=7)
    B = 16
    keys = keyset(orc, s, ckks.steps_for_bsgs(128, B), wid=7)
    out = orc.bsgs_block(orc.baby_rotations(ct, B, keys), ckks.layout_b_pts(X, par, 128, B), B, 128 // B, keys)
    z = dec(orc, out, s, 80)
    cos = X @ q / (np.linalg.norm(X, axis=1) * np.linalg.norm(q))
    assert np.max(np.abs(z[:rows] - cos)) < 1e-4


def test_layout_a_scores_match_float64(small):
    par, orc = small
    d = 16
    rows = 2 * par.slots // d + 5  # three plaintexts, last one ragged
    s = gen.ternary_secret(gen.rng(8, gen.STREAM_SECRET), par.n)
    X = gen.gaussian_unit_rows(gen.rng(8, gen.STREAM_DB), rows, d)
    q = gen.gaussian_unit_rows(gen.rng(8, gen.STREAM_QUERY), 1, d)[0]
    ct = enc(orc, ckks.replicate(q, par.slots), s, wid=8)
    steps = [1 << k for k in range(4)]
    keys = keyset(orc, s, steps, wid=8)
    pts = ckks.pack_rows(X, par.slots, d)
    scores = []
    for w in range(pts.shape[0]):
        pt = ckks.encode_residues(pts[w], par)
        z = orc.rotate_sum(orc.mul_plain(ct, pt), 1, 4, keys)
        scores.extend(dec(orc, z, s, 80)[::d])
    assert np.max(np.abs(np.array(scores)[:rows] - X @ q)) < 1e-4


def test_projection_then_scoring_with_norm_correction():
    par = ckks.Params(logn=11, L=4, K=2)
    orc = ckks.Oracle(par)
    d_in, R, B, rows = 64, 16, 4, 100
    s = gen.ternary_secret(gen.rng(9, gen.STREAM_SECRET), par.n)
    W = gen.projection_matrix(gen.rng(9, gen.STREAM_W), d_in, R, var=1.0 / R)
    q = gen.gaussian_unit_rows(gen.rng(9, gen.STREAM_QUERY), 1, d_in)[0]
    Xr = gen.normalize_rows(gen.gaussian_unit_rows(gen.rng(9, gen.STREAM_DB), rows, d_in) @ W)
    ct = enc(orc, ckks.replicate(q, par.slots), s, wid=9)
    c = d_in // R
    steps = sorted(set(ckks.steps_for_bsgs(R, B) + [R << k for k in range(int(np.log2(c)))]))
    keys = keyset(orc, s, steps, wid=9)
    # projection: hybrid diagonals, BSGS, one final fold
    e = ckks.projection_diagonals(W, par.slots)
    pre = ckks.prerotate(e, B)
    wpts = np.stack([[ckks.encode_residues(pre[g, b], par) for b in range(B)] for g in range(R // B)])
    z = orc.bsgs_block(orc.baby_rotations(ct, B, keys), wpts, B, R // B, keys)
    z = orc.rotate_sum(z, R, int(np.log2(c)), keys)
    qR = W.T @ q
    assert np.max(np.abs(dec(orc, z, s, 80) - np.tile(qR, par.slots // R))) < 1e-4
    # scoring the projected query (scale 2^120), then the client's norm correction
    out = orc.bsgs_block(orc.baby_rotations(z, B, keys), ckks.layout_b_pts(Xr, par, R, B), B, R // B, keys)
    raw = dec(orc, out, s, 120)[:rows]
    assert np.max(np.abs(raw - Xr @ qR)) < 1e-4
    cos = raw / np.linalg.norm(qR)
    assert np.max(np.abs(cos - Xr @ qR / np.linalg.norm(qR))) < 1e-4


# ----------------------------------------------------------------------------
# lower levels: restricted keys and dropped ciphertexts
# ----------------------------------------------------------------------------
def low_params(par, L_low):
    return ckks.Params(logn=par.logn, L=L_low, K=par.K, primes=par.q[:L_low] + par.p)


def restrict(par, L_low, x):
    """Limbs of a [..][L+K][N] array for the primes of the lower level."""
    idx = list(range(L_low)) + list(range(par.L, par.L + par.K))
    return x[..., idx, :]


@pytest.mark.parametrize("L_low", [2, 3])
def test_lower_level_key_is_restriction_of_full_key(small4, L_low):
    """Key generated at the lower level from the restricted randomness == restricted full key."""
    par, orc = small4
    s = gen.ternary_secret(gen.rng(12, gen.STREAM_SECRET), par.n)
    a = gen.uniform_residues(gen.rng(12, gen.STREAM_KEY_A, 3), par.primes, par.dnum, par.n)
    e = gen.rounded_gaussian(gen.rng(12, gen.STREAM_KEY_E, 3), (par.dnum, par.n))
    b_full, _ = orc.keygen(s, 3, a, e)
    lp = low_params(par, L_low)
    lo = ckks.Oracle(lp)
    b_low, _ = lo.keygen(s, 3, restrict(par, L_low, a)[:lp.dnum], e[:lp.dnum])
    assert np.array_equal(b_low, restrict(par, L_low, b_full)[:lp.dnum])


def test_dropped_ciphertext_decrypts_and_rotates(small4):
    par, orc = small4
    L_low = 2
    s = gen.ternary_secret(gen.rng(13, gen.STREAM_SECRET), par.n)
    v = np.random.default_rng(13).uniform(-1, 1, par.slots)
    ct = enc(orc, v, s, wid=13)
    lp = low_params(par, L_low)
    lo = ckks.Oracle(lp)
    ct_low = np.ascontiguousarray(ct[:, :L_low])
    assert np.max(np.abs(ckks.decode_residues(lo.decrypt(ct_low, s), lp, 40) - v)) < 1e-6
    a = gen.uniform_residues(gen.rng(13, gen.STREAM_KEY_A, 5), par.primes, par.dnum, par.n)
    e = gen.rounded_gaussian(gen.rng(13, gen.STREAM_KEY_E, 5), (par.dnum, par.n))
    key = lo.keygen(s, 5, restrict(par, L_low, a)[:lp.dnum], e[:lp.dnum])
    z = ckks.decode_residues(lo.decrypt(lo.rotate(ct_low, 5, key), s), lp, 40)
    assert np.max(np.abs(z - np.roll(v, -5))) < 1e-6


# ----------------------------------------------------------------------------
# encrypted database: tensor product, relinearisation key, relinearisation,
# ct x ct diagonal scoring
# ----------------------------------------------------------------------------
def negacyclic_square_int(s):
    """s^2 mod X^N + 1 over the integers (s small), by the definition."""
    n = len(s)
    full = np.convolve(s.astype(np.int64), s.astype(np.int64))  # degree 2N-2
    out = full[:n].copy()
    out[:n - 1] -= full[n:]
    return out


def relin_key(orc, s, wid):
    par = orc.par
    a = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, 0), par.primes, par.dnum, par.n)
    e = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, 0), (par.dnum, par.n))
    return orc.keygen_relin(s, a, e), e


def test_tensor_decrypts_to_product_of_decryptions(small):
    """(c0 + c1 s)(d0 + d1 s) = c0 d0 + (c0 d1 + c1 d0) s + c1 d1 s^2 exactly mod Q: the
    tensor's three components decrypted under (1, s, s^2) equal the ring product of the two
    decryptions (a dropped or misplaced cross term breaks the equality)."""
    par, orc = small
    s = gen.ternary_secret(gen.rng(30, gen.STREAM_SECRET), par.n)
    g = np.random.default_rng(30)
    x = np.stack([np.stack([g.integers(0, q, par.n, dtype=np.uint64) for q in par.q]) for _ in range(2)])
    y = np.stack([np.stack([g.integers(0, q, par.n, dtype=np.uint64) for q in par.q]) for _ in range(2)])
    d = orc.tensor(x, y)
    lhs = orc.decrypt3(d, s)
    mx, my = orc.decrypt(x, s), orc.decrypt(y, s)
    for t, q in enumerate(par.q):
        assert np.array_equal(lhs[t], orc.polymul(t, mx[t], my[t]))
    # and the tensor's first component is the plain product c0 d0 (schoolbook at a tiny ring)
    tp = ckks.Params(logn=5, L=2, K=1)
    to = ckks.Oracle(tp)
    xs = np.stack([np.stack([g.integers(0, q, tp.n, dtype=np.uint64) for q in tp.q]) for _ in range(2)])
    ys = np.stack([np.stack([g.integers(0, q, tp.n, dtype=np.uint64) for q in tp.q]) for _ in range(2)])
    ds = to.tensor(xs, ys)
    for t, q in enumerate(tp.q):
        assert np.array_equal(ds[0, t], schoolbook_negacyclic(xs[0, t], ys[0, t], q))
        cross = (schoolbook_negacyclic(xs[0, t], ys[1, t], q).astype(object)
                 + schoolbook_negacyclic(xs[1, t], ys[0, t], q).astype(object)) % q
        assert np.array_equal(ds[1, t], cross.astype(np.uint64))
        assert np.array_equal(ds[2, t], schoolbook_negacyclic(xs[1, t], ys[1, t], q))


def test_relin_key_is_gadget_times_s_squared(small4):
    """b_i + a_i s - gadget_i s^2 = e_i on every prime of Q u P, with s^2 formed here over
    the integers (not by the oracle)."""
    par, orc = small4
    s = gen.ternary_secret(gen.rng(31, gen.STREAM_SECRET), par.n)
    (b, a), e = relin_key(orc, s, 31)
    s2 = negacyclic_square_int(s)
    gad = ckks.gadget_table(par)
    for i in range(par.dnum):
        for t, q in enumerate(par.primes):
            st = [int(v) % q for v in s]
            sa = schoolbook_negacyclic(a[i, t], np.array(st, dtype=np.uint64), q) if par.n <= 64 else \
                orc.polymul(t, a[i, t], np.array(st, dtype=np.uint64))
            lhs = (b[i, t].astype(object) + sa.astype(object)
                   - int(gad[i, t]) * np.array([int(v) % q for v in s2], dtype=object)) % q
            assert np.array_equal(lhs, np.array([int(v) % q for v in e[i]], dtype=object)), (i, t)


def test_relin_preserves_the_decryption(small4):
    """decrypt(Relin(d)) = decrypt3(d) + small key-switch noise: the centred difference is far
    below the product scale (a wrong key, sign or missing ModDown leaves ~Q)."""
    par, orc = small4
    s = gen.ternary_secret(gen.rng(32, gen.STREAM_SECRET), par.n)
    rlk, _ = relin_key(orc, s, 32)
    v1 = gen.gaussian_unit_rows(gen.rng(32, gen.STREAM_QUERY), 1, par.slots)[0]
    v2 = gen.gaussian_unit_rows(gen.rng(32, gen.STREAM_DB), 1, par.slots)[0]
    x = enc(orc, v1, s, wid=32)
    y = enc(orc, v2, s, wid=33)
    d = orc.tensor(x, y)
    r = orc.relin(d, rlk)
    diff = np.stack([((orc.decrypt(r, s)[t].astype(object) - orc.decrypt3(d, s)[t].astype(object)) % q)
                     .astype(np.uint64) for t, q in enumerate(par.q)])
    assert max(abs(v) for v in ckks.crt_centered(diff, par.q)) < 2 ** 40
    z = ckks.decode_residues(orc.decrypt(r, s), par, 80)
    assert np.max(np.abs(z - v1 * v2)) < 1e-6


@pytest.mark.parametrize("B", [1, 4])
def test_encrypted_block_scores_match_float64(small, B):
    """Encrypted pre-rotated diagonals: per giant index the tensor sum, one relinearisation,
    then the giant sum; decrypted scores are the float64 inner products."""
    par, orc = small
    d, rows = 16, 300
    G = d // B
    s = gen.ternary_secret(gen.rng(34, gen.STREAM_SECRET), par.n)
    X = gen.gaussian_unit_rows(gen.rng(34, gen.STREAM_DB), rows, d)
    q = gen.gaussian_unit_rows(gen.rng(34, gen.STREAM_QUERY), 1, d)[0]
    ct = enc(orc, ckks.replicate(q, par.slots), s, wid=34)
    keys = keyset(orc, s, ckks.steps_for_bsgs(d, B), wid=34)
    rlk, _ = relin_key(orc, s, 34)
    coeffs = ckks.layout_b_coeffs(X, par, d, B)
    cts = np.empty((G, B, 2, par.L, par.n), dtype=np.uint64)
    for j, m in enumerate(coeffs):
        a = gen.uniform_residues(gen.rng(34, gen.STREAM_ENC_A, 1 + j), par.q, 1, par.n)[0]
        e = gen.rounded_gaussian(gen.rng(34, gen.STREAM_ENC_E, 1 + j), par.n)
        cts[j // B, j % B] = orc.encrypt(m, a, e, s)
    out = orc.bsgs_block_ct(orc.baby_rotations(ct, B, keys), cts, B, G, keys, rlk)
    z = dec(orc, out, s, 80)
    assert np.max(np.abs(z[:rows] - X @ q)) < 1e-4
    assert np.max(np.abs(z[rows:])) < 1e-4


def test_encrypted_projection_matches_float64(small4):
    """W's pre-rotated hybrid diagonals encrypted: the ct x ct diagonal product (one
    relinearisation per giant index) and the fold decrypt to W^T q, periodic in R, and the
    projected query then scores projected rows to their float64 inner products."""
    par, orc = small4
    d_in, R, B, rows = 64, 16, 4, 100
    G, c = R // B, d_in // R
    s = gen.ternary_secret(gen.rng(35, gen.STREAM_SECRET), par.n)
    W = gen.projection_matrix(gen.rng(35, gen.STREAM_W), d_in, R, var=1.0 / R)
    q = gen.gaussian_unit_rows(gen.rng(35, gen.STREAM_QUERY), 1, d_in)[0]
    ct = enc(orc, ckks.replicate(q, par.slots), s, wid=35)
    steps = sorted(set(ckks.steps_for_bsgs(R, B) + [R << k for k in range(int(np.log2(c)))]))
    keys = keyset(orc, s, steps, wid=35)
    rlk, _ = relin_key(orc, s, 35)
    pre = ckks.prerotate(ckks.projection_diagonals(W, par.slots), B)
    wct = np.empty((G, B, 2, par.L, par.n), dtype=np.uint64)
    for g in range(G):
        for b in range(B):
            a = gen.uniform_residues(gen.rng(35, gen.STREAM_ENC_A, 1 + g * B + b), par.q, 1, par.n)[0]
            e = gen.rounded_gaussian(gen.rng(35, gen.STREAM_ENC_E, 1 + g * B + b), par.n)
            wct[g, b] = orc.encrypt(ckks.encode(pre[g, b], par.n, 40), a, e, s)
    z = orc.bsgs_block_ct(orc.baby_rotations(ct, B, keys), wct, B, G, keys, rlk)
    z = orc.rotate_sum(z, R, int(np.log2(c)), keys)
    qR = W.T @ q
    assert np.max(np.abs(dec(orc, z, s, 80) - np.tile(qR, par.slots // R))) < 1e-4
    Xr = gen.normalize_rows(gen.gaussian_unit_rows(gen.rng(35, gen.STREAM_DB), rows, d_in) @ W)
    out = orc.bsgs_block(orc.baby_rotations(z, B, keys), ckks.layout_b_pts(Xr, par, R, B), B, G, keys)
    assert np.max(np.abs(dec(orc, out, s, 120)[:rows] - Xr @ qR)) < 1e-4


# ----------------------------------------------------------------------------
# membership path: rescale, Chebyshev direct evaluator, sign iteration
# ----------------------------------------------------------------------------
def test_rescale_is_rounded_division_by_the_last_prime(small4):
    """Coefficient-wise, rescale(c) = round(c / q_last) mod Q' for c lifted to [0, Q), with
    the remainder taken in (-q_last/2, q_last/2] -- checked with big integers."""
    par, orc = small4
    g = np.random.default_rng(40)
    ct = np.stack([np.stack([g.integers(0, q, par.n, dtype=np.uint64) for q in par.q]) for _ in range(2)])
    out = orc.rescale(ct)
    ql = par.q[-1]
    for h in range(2):
        big = ckks.crt_centered(ct[h], par.q)
        for k in range(0, par.n, 97):
            c = int(big[k]) % par.Q
            r = c % ql
            if r > (ql - 1) // 2:
                r -= ql
            v = (c - r) // ql
            assert [int(out[h, t, k]) for t in range(par.L - 1)] == [v % q for q in par.q[:-1]], (h, k)


def test_rescale_of_multiple_of_last_prime_is_exact(small4):
    """c = q_last * x  ->  rescale(c) = x exactly, for a small signed polynomial x."""
    par, orc = small4
    x = np.random.default_rng(41).integers(-1000, 1000, par.n)
    ql = par.q[-1]
    c = np.stack([np.array([(ql * int(v)) % q for v in x], dtype=np.uint64) for q in par.q])[None]
    out = orc.rescale(c)[0]
    for t, q in enumerate(par.q[:-1]):
        assert np.array_equal(out[t], np.array([int(v) % q for v in x], dtype=np.uint64))


def _chain(logn, L, K, wid):
    top = ckks.Params(logn=logn, L=L, K=K, log_scale=50)
    s = gen.ternary_secret(gen.rng(wid, gen.STREAM_SECRET), top.n)
    ra = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, 0), top.primes, top.dnum, top.n)
    re_ = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, 0), (top.dnum, top.n))
    return ckks.LevelChain(top, s, (ra, re_), {}, rot_levels=[]), s


def _enc_at(ch, v, s, wid, tag, scale_bits=50):
    top = ch.top
    m = ckks.encode(v, top.n, scale_bits)
    a = gen.uniform_residues(gen.rng(wid, gen.STREAM_ENC_A, tag), top.q, 1, top.n)[0]
    e = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_ENC_E, tag), top.n)
    return ch.orc[top.L].encrypt(m, a, e, s)


def _dec_at(ch, ct, L, scale, s):
    orc = ch.orc[L]
    return ckks.decode_residues(orc.decrypt(ct, s), orc.par, 0) / scale


def test_chebyshev_direct_evaluator_matches_numpy():
    """Degree-7 Chebyshev series of an encrypted u in [-1, 1] (levels 7 -> 3): decrypted
    values equal numpy's chebval of the decrypted input within 1e-6."""
    ch, s = _chain(10, 7, 2, 42)
    top = ch.top
    u = np.random.default_rng(42).uniform(-1, 1, top.slots)
    coeffs = np.random.default_rng(43).uniform(-1, 1, 8)
    ct = _enc_at(ch, u, s, 42, 1)
    out, L, sc = ckks.cheb_eval(ch, ct, top.L, 2.0 ** 50, coeffs)
    assert L == top.L - 4
    z = _dec_at(ch, out, L, sc, s)
    assert np.max(np.abs(z - np.polynomial.chebyshev.chebval(u, coeffs))) < 1e-6


def test_sign_iteration_matches_the_odd_polynomial():
    """Two iterations of f(x) = (3x - x^3)/2 on x = V/4 (integer constants, tracked
    multiplier 4 -> 128 -> 2^22): decrypted V / m equals f(f(x)) within 1e-6 and has the
    sign of x."""
    ch, s = _chain(10, 6, 2, 44)
    top = ch.top
    x = np.random.default_rng(44).uniform(-0.5, 0.5, top.slots)
    ct = _enc_at(ch, 4 * x, s, 44, 1)
    V, L, sc, m = ckks.sign_iter(ch, ct, top.L, 2.0 ** 50, 4, 2)
    assert (L, m) == (top.L - 4, 2 * 128 ** 3)
    z = _dec_at(ch, V, L, sc, s) / m
    f = lambda t: (3 * t - t ** 3) / 2
    assert np.max(np.abs(z - f(f(x)))) < 1e-6
    big = np.abs(x) > 1e-3
    assert np.all(np.sign(z[big]) == np.sign(x[big]))


def _membership_setup(logn, L, K, wid, d, B, rot_levels):
    top = ckks.Params(logn=logn, L=L, K=K, log_scale=50)
    s = gen.ternary_secret(gen.rng(wid, gen.STREAM_SECRET), top.n)
    ra = gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, 0), top.primes, top.dnum, top.n)
    re_ = gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, 0), (top.dnum, top.n))
    steps = sorted(set(ckks.steps_for_bsgs(d, B) + [1 << k for k in range(int(np.log2(d)))]))
    rot = {r: (gen.uniform_residues(gen.rng(wid, gen.STREAM_KEY_A, r), top.primes, top.dnum, top.n),
               gen.rounded_gaussian(gen.rng(wid, gen.STREAM_KEY_E, r), (top.dnum, top.n))) for r in steps}
    return ckks.LevelChain(top, s, (ra, re_), rot, rot_levels=rot_levels), s


def _membership_model(X, qR, tau, y_lo, y_hi, coeffs, m, iters):
    """float64 model of the scan: f^iters((<q_R, x> - chebval(u(|q_R|^2)))/m)."""
    y = float(qR @ qR)
    u = (2 * y - y_lo - y_hi) / (y_hi - y_lo)
    t = np.polynomial.chebyshev.chebval(u, coeffs)
    x = (X @ qR - t) / m
    for _ in range(iters):
        x = (3 * x - x ** 3) / 2
    return x, t


@pytest.mark.parametrize("y_lo,y_hi", [(0.5, 2.5), (0.6, 1.6)])
def test_membership_scan_decides_the_threshold(y_lo, y_hi):
    """Membership scan on levels 11 -> 2 (N = 2^11, d = 16, two blocks): every output / m
    equals the float64 model f(f((<q_R, x_i> - t)/m)) within 1e-5, where t is the
    degree-7 Chebyshev interpolant of tau sqrt(y) at y = |q_R|^2 (itself within 1e-4 of
    tau |q_R|), and the output's sign is the decision cos(q_R, x_i) >= tau wherever the
    margin exceeds the interpolation error.  The second domain has width 1, so the map
    onto [-1, 1] doubles y (carried by the scale) and the series must be rescaled to the
    scores' scale by a factor near 2."""
    d, B, tau, m, iters = 16, 4, 0.6, 4, 2
    ch, s = _membership_setup(11, 11, 3, 45, d, B, rot_levels=[11, 10])
    top = ch.top
    g = np.random.default_rng(45)
    X = gen.normalize_rows(g.standard_normal((1024 + 500, d)))
    qR = 1.1 * gen.normalize_rows((X[3] + 0.4 * g.standard_normal(d))[None])[0]
    half, mid = (y_hi - y_lo) / 2, (y_hi + y_lo) / 2
    coeffs = np.polynomial.chebyshev.chebinterpolate(lambda u: tau * np.sqrt(mid + half * u), 7)
    ct = _enc_at(ch, ckks.replicate(qR, top.slots), s, 45, 1)
    blocks = [ckks.layout_b_pts(X[:1024], top, d, B), ckks.layout_b_pts(X[1024:], top, d, B)]
    outs, L, sc, mo = ckks.membership(ch, ct, top.L, 2.0 ** 50, blocks, d, B, y_lo, y_hi, coeffs, m, iters)
    assert (L, mo) == (top.L - 9, 2 * 128 ** 3)
    want, t = _membership_model(np.vstack([X, np.zeros((2 * top.slots - len(X), d))]), qR, tau, y_lo, y_hi, coeffs, m, iters)
    assert abs(t - tau * np.linalg.norm(qR)) < 1e-4
    z = np.concatenate([_dec_at(ch, o, L, sc, s) for o in outs]) / mo
    assert np.max(np.abs(z - want)) < 1e-5
    margin = (X @ qR - tau * np.linalg.norm(qR))
    ok = np.abs(margin) > 2e-4
    assert np.all(np.sign(z[:len(X)][ok]) == np.sign(margin[ok]))
    assert 0 < np.count_nonzero(margin > 0) < len(X) // 4
