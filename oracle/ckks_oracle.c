/*
 * ckks_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU reference for the integer part of the
 * encrypted scoring path: RNS-CKKS ring arithmetic, Galois automorphisms,
 * fast basis conversion, hybrid key switching (ModUp / inner product /
 * ModDown), the diagonal baby-step/giant-step matrix-vector product with
 * plaintext pre-rotation, and the rotate-and-sum fold.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may load
 * this library. It shares no code, header, table or constant with the GPU
 * library: every constant it needs is either derived here from the primes or
 * computed by oracle/ckks.py with Python big integers from its definition.
 *
 * Conventions (all arrays are host memory, row-major, coefficient form):
 *   - a polynomial over prime index l is N words in [0, q_l);
 *   - an RNS polynomial over a prime list is [nlimbs][N];
 *   - a ciphertext is [2][L][N]  (c0, c1), decrypting as c0 + c1*s;
 *   - primes[0..L-1] are the ciphertext primes q_i, primes[L..L+K-1] the
 *     special primes p_k (the product P).
 *
 * Arithmetic is u64 residues with unsigned __int128 products reduced by '%'.
 * The negacyclic number-theoretic transform below is only a device to form
 * ring products (a*b mod X^N+1) fast; it is pinned against the schoolbook
 * negacyclic convolution by the tests.  Sums of ring products are formed in
 * the transform domain, which is exact because the transform is linear.
 *
 * Parallelism: OpenMP over independent limbs / polynomials only; every result
 * is a pure function of the inputs.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef uint64_t u64;
typedef int64_t i64;
typedef unsigned __int128 u128;

/* ------------------------------------------------------------------ */
/* scalar modular arithmetic                                           */
/* ------------------------------------------------------------------ */
static inline u64 mulm(u64 a, u64 b, u64 q) { return (u64)(((u128)a * b) % q); }
static inline u64 addm(u64 a, u64 b, u64 q) { u64 s = a + b; return s >= q ? s - q : s; }
static inline u64 subm(u64 a, u64 b, u64 q) { return a >= b ? a - b : a + (q - b); }
static inline u64 negm(u64 a, u64 q) { return a == 0 ? 0 : q - a; }
static u64 powm(u64 b, u64 e, u64 q) {
  u64 r = 1 % q;
  b %= q;
  while (e) {
    if (e & 1) r = mulm(r, b, q);
    b = mulm(b, b, q);
    e >>= 1;
  }
  return r;
}
/* signed integer -> residue in [0, q) */
static inline u64 from_signed(i64 v, u64 q) {
  if (v >= 0) return (u64)v % q;
  u64 m = (u64)(-(v + 1)) % q; /* -(v+1) >= 0 avoids overflow at INT64_MIN */
  return q - 1 - m;
}

/* ------------------------------------------------------------------ */
/* context: ring degree, primes, transform tables, key-switch tables   */
/* ------------------------------------------------------------------ */
typedef struct {
  int logn, n;
  int L, K;         /* ciphertext primes, special primes */
  int alpha, dnum;  /* primes per digit, number of digits */
  u64* primes;      /* [L+K] */
  /* transform tables per prime: psi^j, psi^-j, omega^j, omega^-j  (j < N) */
  u64** psi_pow;
  u64** psi_ipow;
  u64** om_pow;
  u64** om_ipow;
  u64* n_inv;       /* N^-1 mod q */
  /* fast basis conversion tables (set by or_set_ks_tables):
   *   digit i has source primes src(i) = {i*alpha, ..., min((i+1)alpha, L)-1}
   *   modup_inv[i][j]     = (D_i / q_{src j})^-1 mod q_{src j}
   *   modup_hat[i][j][t]  = (D_i / q_{src j}) mod prime t, t over all L+K primes
   *   down_inv[k]         = (P / p_k)^-1 mod p_k
   *   down_hat[k][t]      = (P / p_k) mod q_t, t < L
   *   p_inv[t]            = P^-1 mod q_t, t < L                              */
  u64* modup_inv;
  u64* modup_hat;
  u64* down_inv;
  u64* down_hat;
  u64* p_inv;
  int* rev;         /* bit reversal permutation of log n bits */
} octx;

static int bitrev(int x, int bits) {
  int r = 0;
  for (int i = 0; i < bits; ++i) { r = (r << 1) | (x & 1); x >>= 1; }
  return r;
}

/* smallest generator-derived primitive 2N-th root of unity mod q */
static u64 find_psi(u64 q, int n) {
  u64 two_n = 2 * (u64)n;
  for (u64 x = 2; x < q; ++x) {
    u64 y = powm(x, (q - 1) / two_n, q);
    if (powm(y, (u64)n, q) == q - 1) return y; /* order exactly 2N */
  }
  return 0;
}

void* or_create(int logn, int L, int K, const u64* primes) {
  octx* c = (octx*)calloc(1, sizeof(octx));
  c->logn = logn;
  c->n = 1 << logn;
  c->L = L;
  c->K = K;
  c->alpha = K;
  c->dnum = (L + K - 1) / K;
  int np = L + K, n = c->n;
  c->primes = (u64*)malloc(sizeof(u64) * np);
  memcpy(c->primes, primes, sizeof(u64) * np);
  c->psi_pow = (u64**)malloc(sizeof(u64*) * np);
  c->psi_ipow = (u64**)malloc(sizeof(u64*) * np);
  c->om_pow = (u64**)malloc(sizeof(u64*) * np);
  c->om_ipow = (u64**)malloc(sizeof(u64*) * np);
  c->n_inv = (u64*)malloc(sizeof(u64) * np);
  c->rev = (int*)malloc(sizeof(int) * n);
  for (int i = 0; i < n; ++i) c->rev[i] = bitrev(i, logn);
  for (int l = 0; l < np; ++l) {
    u64 q = primes[l];
    u64 psi = find_psi(q, n);
    u64 ipsi = powm(psi, q - 2, q);
    u64 om = mulm(psi, psi, q), iom = mulm(ipsi, ipsi, q);
    c->psi_pow[l] = (u64*)malloc(sizeof(u64) * n);
    c->psi_ipow[l] = (u64*)malloc(sizeof(u64) * n);
    c->om_pow[l] = (u64*)malloc(sizeof(u64) * n);
    c->om_ipow[l] = (u64*)malloc(sizeof(u64) * n);
    u64 a = 1, b = 1, x = 1, y = 1;
    for (int j = 0; j < n; ++j) {
      c->psi_pow[l][j] = a; a = mulm(a, psi, q);
      c->psi_ipow[l][j] = b; b = mulm(b, ipsi, q);
      c->om_pow[l][j] = x; x = mulm(x, om, q);
      c->om_ipow[l][j] = y; y = mulm(y, iom, q);
    }
    c->n_inv[l] = powm((u64)n, q - 2, q);
  }
  return c;
}

void or_destroy(void* p) {
  octx* c = (octx*)p;
  if (!c) return;
  int np = c->L + c->K;
  for (int l = 0; l < np; ++l) {
    free(c->psi_pow[l]); free(c->psi_ipow[l]); free(c->om_pow[l]); free(c->om_ipow[l]);
  }
  free(c->psi_pow); free(c->psi_ipow); free(c->om_pow); free(c->om_ipow);
  free(c->n_inv); free(c->rev); free(c->primes);
  free(c->modup_inv); free(c->modup_hat); free(c->down_inv); free(c->down_hat); free(c->p_inv);
  free(c);
}

/* tables computed with big integers by the Python side from their definition */
void or_set_ks_tables(void* p, const u64* modup_inv, const u64* modup_hat, const u64* down_inv,
                      const u64* down_hat, const u64* p_inv) {
  octx* c = (octx*)p;
  int np = c->L + c->K;
  size_t n_inv = (size_t)c->dnum * c->alpha, n_hat = n_inv * np;
  c->modup_inv = (u64*)malloc(sizeof(u64) * n_inv);
  c->modup_hat = (u64*)malloc(sizeof(u64) * n_hat);
  c->down_inv = (u64*)malloc(sizeof(u64) * c->K);
  c->down_hat = (u64*)malloc(sizeof(u64) * c->K * c->L);
  c->p_inv = (u64*)malloc(sizeof(u64) * c->L);
  memcpy(c->modup_inv, modup_inv, sizeof(u64) * n_inv);
  memcpy(c->modup_hat, modup_hat, sizeof(u64) * n_hat);
  memcpy(c->down_inv, down_inv, sizeof(u64) * c->K);
  memcpy(c->down_hat, down_hat, sizeof(u64) * c->K * c->L);
  memcpy(c->p_inv, p_inv, sizeof(u64) * c->L);
}

/* ------------------------------------------------------------------ */
/* negacyclic transform (a device for ring products only)              */
/*   forward:  A[k] = sum_j a[j] psi^{j} omega^{jk}   (omega = psi^2)   */
/*   i.e. A[k] = a(psi^{2k+1}); inverse undoes it exactly.             */
/* ------------------------------------------------------------------ */
static void cyclic_dft(const octx* c, int l, u64* a, const u64* wtab) {
  /* iterative radix-2 decimation-in-time on bit-reversed input */
  int n = c->n;
  u64 q = c->primes[l];
  for (int i = 0; i < n; ++i) {
    int r = c->rev[i];
    if (i < r) { u64 t = a[i]; a[i] = a[r]; a[r] = t; }
  }
  for (int len = 2; len <= n; len <<= 1) {
    int half = len >> 1, step = n / len;
    for (int s = 0; s < n; s += len) {
      for (int j = 0; j < half; ++j) {
        u64 w = wtab[(size_t)j * step];
        u64 u = a[s + j], v = mulm(a[s + j + half], w, q);
        a[s + j] = addm(u, v, q);
        a[s + j + half] = subm(u, v, q);
      }
    }
  }
}

void or_ntt(void* p, int l, u64* a) {
  octx* c = (octx*)p;
  u64 q = c->primes[l];
  for (int j = 0; j < c->n; ++j) a[j] = mulm(a[j], c->psi_pow[l][j], q);
  cyclic_dft(c, l, a, c->om_pow[l]);
}

void or_intt(void* p, int l, u64* a) {
  octx* c = (octx*)p;
  u64 q = c->primes[l];
  cyclic_dft(c, l, a, c->om_ipow[l]);
  for (int j = 0; j < c->n; ++j) a[j] = mulm(mulm(a[j], c->n_inv[l], q), c->psi_ipow[l][j], q);
}

/* out = a * b in Z_{q_l}[X]/(X^N+1) */
void or_polymul(void* p, int l, const u64* a, const u64* b, u64* out) {
  octx* c = (octx*)p;
  int n = c->n;
  u64 q = c->primes[l];
  u64* x = (u64*)malloc(sizeof(u64) * n);
  memcpy(x, a, sizeof(u64) * n);
  memcpy(out, b, sizeof(u64) * n);
  or_ntt(c, l, x);
  or_ntt(c, l, out);
  for (int j = 0; j < n; ++j) out[j] = mulm(out[j], x[j], q);
  or_intt(c, l, out);
  free(x);
}

/* ------------------------------------------------------------------ */
/* Galois automorphism sigma_g: X -> X^g  (g odd), coefficient form.   */
/* coefficient j moves to t = g*j mod 2N; if t >= N it lands on t-N    */
/* with its sign flipped (X^N = -1).                                    */
/* ------------------------------------------------------------------ */
static void automorph_poly(int n, u64 g, u64 q, const u64* in, u64* out) {
  u64 two_n = 2 * (u64)n;
  for (int j = 0; j < n; ++j) {
    u64 t = (u64)(((u128)g * (u64)j) % two_n);
    if (t < (u64)n) out[t] = in[j];
    else out[t - n] = negm(in[j], q);
  }
}

void or_automorph(void* p, u64 g, int nlimbs, const int* limb_ids, const u64* in, u64* out) {
  octx* c = (octx*)p;
  int n = c->n;
  for (int i = 0; i < nlimbs; ++i)
    automorph_poly(n, g, c->primes[limb_ids[i]], in + (size_t)i * n, out + (size_t)i * n);
}

/* ------------------------------------------------------------------ */
/* fast basis conversion, no correction term:                           */
/*   Conv_{S->t}(x) = sum_{j in S} [x_j * (S/s_j)^-1]_{s_j} * (S/s_j mod t)  mod t
 * src: [ns][N] canonical residues; inv[j] = (S/s_j)^-1 mod s_j;
 * hat[j*stride + t] = (S/s_j) mod target t.                            */
static void conv_coeffwise(int n, int ns, const u64* src_primes, const u64* src, const u64* inv,
                           const u64* hat, int hat_stride, int nt, const int* tgt_ids,
                           const u64* tgt_primes, u64* dst /* [nt][N] */) {
  u64* y = (u64*)malloc(sizeof(u64) * ns);
  for (int k = 0; k < n; ++k) {
    for (int j = 0; j < ns; ++j) y[j] = mulm(src[(size_t)j * n + k], inv[j], src_primes[j]);
    for (int t = 0; t < nt; ++t) {
      u64 qt = tgt_primes[t], acc = 0;
      for (int j = 0; j < ns; ++j) acc = addm(acc, mulm(y[j] % qt, hat[(size_t)j * hat_stride + tgt_ids[t]], qt), qt);
      dst[(size_t)t * n + k] = acc;
    }
  }
  free(y);
}

/* ModUp of digit i: given c1 [L][N] (coefficient form), produce the digit
 * extended to all L+K primes: [L+K][N].  Own primes keep their residues,
 * every other prime gets Conv_{D_i -> t}. */
void or_modup_digit(void* p, int i, const u64* c1, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, K = c->K, np = L + K;
  int lo = i * c->alpha, hi = lo + c->alpha;
  if (hi > L) hi = L;
  int ns = hi - lo;
  u64 sp[64] = {0};
  for (int j = 0; j < ns; ++j) sp[j] = c->primes[lo + j];
  int tgt[64] = {0};
  u64 tp[64] = {0};
  int nt = 0;
  for (int t = 0; t < np; ++t) {
    if (t >= lo && t < hi) {
      memcpy(out + (size_t)t * n, c1 + (size_t)t * n, sizeof(u64) * n);
    } else {
      tgt[nt] = t;
      tp[nt] = c->primes[t];
      nt++;
    }
  }
  u64* tmp = (u64*)malloc(sizeof(u64) * (size_t)nt * n);
  conv_coeffwise(n, ns, sp, c1 + (size_t)lo * n, c->modup_inv + (size_t)i * c->alpha,
                 c->modup_hat + (size_t)i * c->alpha * np, np, nt, tgt, tp, tmp);
  for (int t = 0; t < nt; ++t) memcpy(out + (size_t)tgt[t] * n, tmp + (size_t)t * n, sizeof(u64) * n);
  free(tmp);
}

/* ModDown: x over Q u P [L+K][N] -> (x_Q - Conv_{P->Q}(x_P)) * P^-1 over Q [L][N] */
void or_moddown(void* p, const u64* x, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, K = c->K;
  int tgt[64] = {0};
  for (int t = 0; t < L; ++t) tgt[t] = t;
  u64* conv = (u64*)malloc(sizeof(u64) * (size_t)L * n);
  conv_coeffwise(n, K, c->primes + L, x + (size_t)L * n, c->down_inv, c->down_hat, L, L, tgt, c->primes, conv);
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    for (int k = 0; k < n; ++k) {
      size_t o = (size_t)t * n + k;
      out[o] = mulm(subm(x[o], conv[o], q), c->p_inv[t], q);
    }
  }
  free(conv);
}

/* ------------------------------------------------------------------ */
/* keys, encryption, decryption                                         */
/* ------------------------------------------------------------------ */

/* b_i = -a_i*s + e_i + gad[i][t] * sigma_g(s)  over every prime t of Q u P.
 * a: [dnum][L+K][N]; e: [dnum][N] small integers; s: [N] ternary;
 * gad: [dnum][L+K] = (P * Qhat_i * [Qhat_i^-1]_{Q_i}) mod prime t;  b: out [dnum][L+K][N] */
void or_keygen(void* p, const i64* s, u64 g, const u64* a, const i64* e, const u64* gad, u64* b) {
  octx* c = (octx*)p;
  int n = c->n, np = c->L + c->K, dnum = c->dnum;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int i = 0; i < dnum; ++i) {
    for (int t = 0; t < np; ++t) {
      u64 q = c->primes[t];
      u64* sp = (u64*)malloc(sizeof(u64) * n);
      u64* sg = (u64*)malloc(sizeof(u64) * n);
      u64* as = (u64*)malloc(sizeof(u64) * n);
      for (int k = 0; k < n; ++k) sp[k] = from_signed(s[k], q);
      automorph_poly(n, g, q, sp, sg);
      const u64* ai = a + ((size_t)i * np + t) * n;
      or_polymul(c, t, ai, sp, as);
      u64* bi = b + ((size_t)i * np + t) * n;
      u64 gt = gad[(size_t)i * np + t];
      for (int k = 0; k < n; ++k) {
        u64 v = negm(as[k], q);
        v = addm(v, from_signed(e[(size_t)i * n + k], q), q);
        v = addm(v, mulm(gt, sg[k], q), q);
        bi[k] = v;
      }
      free(sp); free(sg); free(as);
    }
  }
}

/* secret-key encryption at full level: c1 = a, c0 = -a*s + e + m  (mod each q_t, t < L) */
void or_encrypt(void* p, const i64* m, const u64* a, const i64* e, const i64* s, u64* ct) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* sp = (u64*)malloc(sizeof(u64) * n);
    u64* as = (u64*)malloc(sizeof(u64) * n);
    for (int k = 0; k < n; ++k) sp[k] = from_signed(s[k], q);
    const u64* at = a + (size_t)t * n;
    or_polymul(c, t, at, sp, as);
    u64* c0 = ct + (size_t)t * n;
    u64* c1 = ct + ((size_t)L + t) * n;
    for (int k = 0; k < n; ++k) {
      u64 v = negm(as[k], q);
      v = addm(v, from_signed(e[k], q), q);
      v = addm(v, from_signed(m[k], q), q);
      c0[k] = v;
      c1[k] = at[k];
    }
    free(sp); free(as);
  }
}

/* m' = c0 + c1*s  (mod each q_t), coefficient form [L][N] */
void or_decrypt(void* p, const u64* ct, const i64* s, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* sp = (u64*)malloc(sizeof(u64) * n);
    for (int k = 0; k < n; ++k) sp[k] = from_signed(s[k], q);
    or_polymul(c, t, ct + ((size_t)L + t) * n, sp, out + (size_t)t * n);
    for (int k = 0; k < n; ++k) out[(size_t)t * n + k] = addm(out[(size_t)t * n + k], ct[(size_t)t * n + k], q);
    free(sp);
  }
}

/* ------------------------------------------------------------------ */
/* key switching for a rotation                                        */
/* ------------------------------------------------------------------ */

/* Steps 1-4 of a rotation's key switch on c1 [L][N] with key (kb, ka), each
 * [dnum][L+K][N]:  decompose c1 into digits, extend each digit to Q u P,
 * apply sigma_g, and form (u0, u1) = sum_i sigma_g(ext_i) * (b_i, a_i).
 * Output u: [2][L+K][N] over Q u P (not yet divided by P). */
void or_ks_inner(void* p, const u64* c1, u64 g, const u64* kb, const u64* ka, u64* u) {
  octx* c = (octx*)p;
  int n = c->n, np = c->L + c->K, dnum = c->dnum;
  size_t poly = (size_t)np * n;
  u64* ext = (u64*)malloc(sizeof(u64) * poly * dnum);
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < dnum; ++i) or_modup_digit(c, i, c1, ext + (size_t)i * poly);
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < np; ++t) {
    u64 q = c->primes[t];
    u64* x = (u64*)malloc(sizeof(u64) * n);
    u64* kbt = (u64*)malloc(sizeof(u64) * n);
    u64* kat = (u64*)malloc(sizeof(u64) * n);
    u64* acc0 = (u64*)calloc(n, sizeof(u64));
    u64* acc1 = (u64*)calloc(n, sizeof(u64));
    for (int i = 0; i < dnum; ++i) {
      automorph_poly(n, g, q, ext + (size_t)i * poly + (size_t)t * n, x);
      memcpy(kbt, kb + (size_t)i * poly + (size_t)t * n, sizeof(u64) * n);
      memcpy(kat, ka + (size_t)i * poly + (size_t)t * n, sizeof(u64) * n);
      or_ntt(c, t, x);
      or_ntt(c, t, kbt);
      or_ntt(c, t, kat);
      for (int k = 0; k < n; ++k) {
        acc0[k] = addm(acc0[k], mulm(x[k], kbt[k], q), q);
        acc1[k] = addm(acc1[k], mulm(x[k], kat[k], q), q);
      }
    }
    or_intt(c, t, acc0);
    or_intt(c, t, acc1);
    memcpy(u + (size_t)t * n, acc0, sizeof(u64) * n);
    memcpy(u + poly + (size_t)t * n, acc1, sizeof(u64) * n);
    free(x); free(kbt); free(kat); free(acc0); free(acc1);
  }
  free(ext);
}

/* Rotate(ct, r) with g = 5^r mod 2N:  out = (sigma_g(c0) + ModDown(u0), ModDown(u1)) */
void or_rotate(void* p, const u64* ct, u64 g, const u64* kb, const u64* ka, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, np = L + c->K;
  size_t poly = (size_t)np * n;
  u64* u = (u64*)malloc(sizeof(u64) * 2 * poly);
  or_ks_inner(c, ct + (size_t)L * n, g, kb, ka, u);
  u64* d0 = (u64*)malloc(sizeof(u64) * (size_t)L * n);
  or_moddown(c, u, d0);
  or_moddown(c, u + poly, out + (size_t)L * n);
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* o = out + (size_t)t * n;
    automorph_poly(n, g, q, ct + (size_t)t * n, o);
    for (int k = 0; k < n; ++k) o[k] = addm(o[k], d0[(size_t)t * n + k], q);
  }
  free(u); free(d0);
}

/* ct_out = ct + Rotate(ct, r) repeated for r = first_shift * 2^k, k < steps.
 * gs[k] and key pointers per step. ct is updated in place. */
void or_rotate_sum(void* p, u64* ct, int steps, const u64* gs, const u64* const* kbs, const u64* const* kas) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
  size_t ctw = (size_t)2 * L * n;
  u64* r = (u64*)malloc(sizeof(u64) * ctw);
  for (int k = 0; k < steps; ++k) {
    or_rotate(c, ct, gs[k], kbs[k], kas[k], r);
    for (int t = 0; t < 2 * L; ++t) {
      u64 q = c->primes[t % L];
      for (int j = 0; j < n; ++j) ct[(size_t)t * n + j] = addm(ct[(size_t)t * n + j], r[(size_t)t * n + j], q);
    }
  }
  free(r);
}

/* ct x pt: out = (c0 * m, c1 * m) over the L ciphertext primes; pt: [L][N] */
void or_mul_plain(void* p, const u64* ct, const u64* pt, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int h = 0; h < 2; ++h)
    for (int t = 0; t < L; ++t)
      or_polymul(c, t, ct + ((size_t)h * L + t) * n, pt + (size_t)t * n, out + ((size_t)h * L + t) * n);
}

/* ------------------------------------------------------------------ */
/* baby-step / giant-step diagonal product with pre-rotated plaintexts */
/* ------------------------------------------------------------------ */

/* acc = sum_{b<B} pt[b] (*) qrot[b]  for one giant index g.
 * qrot_hat: [B][2][L][N] the baby rotations already in the transform domain;
 * pts_g: [B][L][N] coefficient form; out: [2][L][N] coefficient form.
 * The sum of ring products is formed in the transform domain (exact: linear). */
static void mac_group(octx* c, int B, const u64* qrot_hat, const u64* pts_g, u64* out) {
  int n = c->n, L = c->L;
  size_t ctw = (size_t)2 * L * n;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* acc0 = (u64*)calloc(n, sizeof(u64));
    u64* acc1 = (u64*)calloc(n, sizeof(u64));
    u64* y = (u64*)malloc(sizeof(u64) * n);
    for (int b = 0; b < B; ++b) {
      memcpy(y, pts_g + ((size_t)b * L + t) * n, sizeof(u64) * n);
      or_ntt(c, t, y);
      const u64* x0 = qrot_hat + (size_t)b * ctw + (size_t)t * n;
      const u64* x1 = qrot_hat + (size_t)b * ctw + ((size_t)L + t) * n;
      for (int k = 0; k < n; ++k) {
        acc0[k] = addm(acc0[k], mulm(x0[k], y[k], q), q);
        acc1[k] = addm(acc1[k], mulm(x1[k], y[k], q), q);
      }
    }
    or_intt(c, t, acc0);
    or_intt(c, t, acc1);
    memcpy(out + (size_t)t * n, acc0, sizeof(u64) * n);
    memcpy(out + ((size_t)L + t) * n, acc1, sizeof(u64) * n);
    free(acc0); free(acc1); free(y);
  }
}

/* One block of the diagonal product.
 *   qrot  [B][2][L][N]   qrot[b] = Rotate(q, b)  (qrot[0] = q)
 *   pts   [G][B][L][N]   pre-rotated diagonals pt[g][b]
 *   gs[g]                Galois element 5^{gB} mod 2N for g = 1..G-1 (gs[0] unused)
 *   kbs[g], kas[g]       key for rotation gB (g >= 1)
 * out [2][L][N]:
 *   c0 = acc_0.c0 + sum_{g>=1} sigma_{gB}(acc_g.c0) + ModDown(sum_{g>=1} u0_g)
 *   c1 = acc_0.c1 + ModDown(sum_{g>=1} u1_g)
 * where (u0_g, u1_g) is the key-switch inner product of acc_g.c1 for rotation gB. */
void or_bsgs_block(void* p, int B, int G, const u64* qrot, const u64* pts, const u64* gs,
                   const u64* const* kbs, const u64* const* kas, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, np = L + c->K;
  size_t ctw = (size_t)2 * L * n, ptw = (size_t)L * n, poly = (size_t)np * n;
  u64* acc = (u64*)malloc(sizeof(u64) * ctw);
  u64* usum = (u64*)calloc(2 * poly, sizeof(u64));
  u64* u = (u64*)malloc(sizeof(u64) * 2 * poly);
  u64* tmp = (u64*)malloc(sizeof(u64) * n);
  u64* qhat = (u64*)malloc(sizeof(u64) * ctw * B);
  memcpy(qhat, qrot, sizeof(u64) * ctw * B);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < 2 * L; ++t) or_ntt(c, t % L, qhat + (size_t)b * ctw + (size_t)t * n);
  mac_group(c, B, qhat, pts, out); /* g = 0: no rotation */
  for (int g = 1; g < G; ++g) {
    mac_group(c, B, qhat, pts + (size_t)g * B * ptw, acc);
    or_ks_inner(c, acc + (size_t)L * n, gs[g], kbs[g], kas[g], u);
    for (int t = 0; t < np; ++t) {
      u64 q = c->primes[t];
      for (int h = 0; h < 2; ++h)
        for (int k = 0; k < n; ++k) {
          size_t o = (size_t)h * poly + (size_t)t * n + k;
          usum[o] = addm(usum[o], u[o], q);
        }
    }
    for (int t = 0; t < L; ++t) {
      u64 q = c->primes[t];
      automorph_poly(n, gs[g], q, acc + (size_t)t * n, tmp);
      for (int k = 0; k < n; ++k) out[(size_t)t * n + k] = addm(out[(size_t)t * n + k], tmp[k], q);
    }
  }
  if (G > 1) {
    u64* d = (u64*)malloc(sizeof(u64) * ptw);
    for (int h = 0; h < 2; ++h) {
      or_moddown(c, usum + (size_t)h * poly, d);
      for (int t = 0; t < L; ++t) {
        u64 q = c->primes[t];
        for (int k = 0; k < n; ++k) {
          size_t o = ((size_t)h * L + t) * n + k;
          out[o] = addm(out[o], d[(size_t)t * n + k], q);
        }
      }
    }
    free(d);
  }
  free(acc); free(usum); free(u); free(tmp); free(qhat);
}

/* ------------------------------------------------------------------ */
/* encrypted database: ct x ct products with lazy relinearisation       */
/* ------------------------------------------------------------------ */

/* Relinearisation key (switches s^2 to s): for every digit i and prime t of
 * Q u P,  b_i = -a_i*s + e_i + gad[i][t] * s^2.  s^2 is the negacyclic square
 * of s reduced mod the prime.  a: [dnum][L+K][N]; e: [dnum][N]; b: out. */
void or_keygen_relin(void* p, const i64* s, const u64* a, const i64* e, const u64* gad, u64* b) {
  octx* c = (octx*)p;
  int n = c->n, np = c->L + c->K, dnum = c->dnum;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int i = 0; i < dnum; ++i) {
    for (int t = 0; t < np; ++t) {
      u64 q = c->primes[t];
      u64* sp = (u64*)malloc(sizeof(u64) * n);
      u64* s2 = (u64*)malloc(sizeof(u64) * n);
      u64* as = (u64*)malloc(sizeof(u64) * n);
      for (int k = 0; k < n; ++k) sp[k] = from_signed(s[k], q);
      or_polymul(c, t, sp, sp, s2);
      const u64* ai = a + ((size_t)i * np + t) * n;
      or_polymul(c, t, ai, sp, as);
      u64* bi = b + ((size_t)i * np + t) * n;
      u64 gt = gad[(size_t)i * np + t];
      for (int k = 0; k < n; ++k) {
        u64 v = negm(as[k], q);
        v = addm(v, from_signed(e[(size_t)i * n + k], q), q);
        v = addm(v, mulm(gt, s2[k], q), q);
        bi[k] = v;
      }
      free(sp); free(s2); free(as);
    }
  }
}

/* Tensor product of two ciphertexts over Q: (a0, a1) x (b0, b1) =
 * (a0 b0, a0 b1 + a1 b0, a1 b1), which decrypts under (1, s, s^2).
 * x, y: [2][L][N]; out: [3][L][N]; all coefficient form. */
void or_tensor(void* p, const u64* x, const u64* y, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* m = (u64*)malloc(sizeof(u64) * n);
    const u64 *x0 = x + (size_t)t * n, *x1 = x + ((size_t)L + t) * n;
    const u64 *y0 = y + (size_t)t * n, *y1 = y + ((size_t)L + t) * n;
    u64 *d0 = out + (size_t)t * n, *d1 = out + ((size_t)L + t) * n, *d2 = out + ((size_t)2 * L + t) * n;
    or_polymul(c, t, x0, y0, d0);
    or_polymul(c, t, x0, y1, d1);
    or_polymul(c, t, x1, y0, m);
    for (int k = 0; k < n; ++k) d1[k] = addm(d1[k], m[k], q);
    or_polymul(c, t, x1, y1, d2);
    free(m);
  }
}

/* Relinearise a three-component ciphertext d = (d0, d1, d2) [3][L][N]:
 * (u0, u1) = key-switch inner product of d2 with (kb, ka) (no automorphism);
 * out = (d0 + ModDown(u0), d1 + ModDown(u1))  [2][L][N]. */
void or_relin(void* p, const u64* d, const u64* kb, const u64* ka, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, np = L + c->K;
  size_t poly = (size_t)np * n, ptw = (size_t)L * n;
  u64* u = (u64*)malloc(sizeof(u64) * 2 * poly);
  u64* w = (u64*)malloc(sizeof(u64) * ptw);
  or_ks_inner(c, d + 2 * ptw, 1, kb, ka, u);
  for (int h = 0; h < 2; ++h) {
    or_moddown(c, u + (size_t)h * poly, w);
    for (int t = 0; t < L; ++t) {
      u64 q = c->primes[t];
      for (int k = 0; k < n; ++k) {
        size_t o = (size_t)t * n + k;
        out[(size_t)h * ptw + o] = addm(d[(size_t)h * ptw + o], w[o], q);
      }
    }
  }
  free(u); free(w);
}

/* acc = sum_{b<B} ct[b] x qrot[b] for one giant index g, three components.
 * qrot_hat: [B][2][L][N] transform domain; cts_g: [B][2][L][N] coefficient
 * form; out: [3][L][N] coefficient form.  Formed in the transform domain
 * (exact: the transform is linear and multiplicative). */
static void mac_group_ct(octx* c, int B, const u64* qrot_hat, const u64* cts_g, u64* out) {
  int n = c->n, L = c->L;
  size_t ctw = (size_t)2 * L * n;
#pragma omp parallel for schedule(dynamic)
  for (int t = 0; t < L; ++t) {
    u64 q = c->primes[t];
    u64* acc0 = (u64*)calloc(n, sizeof(u64));
    u64* acc1 = (u64*)calloc(n, sizeof(u64));
    u64* acc2 = (u64*)calloc(n, sizeof(u64));
    u64* y0 = (u64*)malloc(sizeof(u64) * n);
    u64* y1 = (u64*)malloc(sizeof(u64) * n);
    for (int b = 0; b < B; ++b) {
      memcpy(y0, cts_g + (size_t)b * ctw + (size_t)t * n, sizeof(u64) * n);
      memcpy(y1, cts_g + (size_t)b * ctw + ((size_t)L + t) * n, sizeof(u64) * n);
      or_ntt(c, t, y0);
      or_ntt(c, t, y1);
      const u64* x0 = qrot_hat + (size_t)b * ctw + (size_t)t * n;
      const u64* x1 = qrot_hat + (size_t)b * ctw + ((size_t)L + t) * n;
      for (int k = 0; k < n; ++k) {
        acc0[k] = addm(acc0[k], mulm(y0[k], x0[k], q), q);
        acc1[k] = addm(acc1[k], addm(mulm(y0[k], x1[k], q), mulm(y1[k], x0[k], q), q), q);
        acc2[k] = addm(acc2[k], mulm(y1[k], x1[k], q), q);
      }
    }
    or_intt(c, t, acc0);
    or_intt(c, t, acc1);
    or_intt(c, t, acc2);
    memcpy(out + (size_t)t * n, acc0, sizeof(u64) * n);
    memcpy(out + ((size_t)L + t) * n, acc1, sizeof(u64) * n);
    memcpy(out + ((size_t)2 * L + t) * n, acc2, sizeof(u64) * n);
    free(acc0); free(acc1); free(acc2); free(y0); free(y1);
  }
}

/* One block of the diagonal product against an encrypted block:
 *   cts [G][B][2][L][N]  the encrypted pre-rotated diagonals ct[g][b]
 *   rel_g = Relin(sum_b ct[g][b] x qrot[b])    (one relinearisation per g)
 * then the giant sum of or_bsgs_block on the rel_g:
 *   c0 = rel_0.c0 + sum_{g>=1} sigma_{gB}(rel_g.c0) + ModDown(sum_{g>=1} u0_g)
 *   c1 = rel_0.c1 + ModDown(sum_{g>=1} u1_g). */
void or_bsgs_block_ct(void* p, int B, int G, const u64* qrot, const u64* cts, const u64* gs,
                      const u64* const* kbs, const u64* const* kas, const u64* rkb, const u64* rka, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L, np = L + c->K;
  size_t ctw = (size_t)2 * L * n, ptw = (size_t)L * n, poly = (size_t)np * n;
  u64* acc3 = (u64*)malloc(sizeof(u64) * 3 * ptw);
  u64* rel = (u64*)malloc(sizeof(u64) * ctw);
  u64* usum = (u64*)calloc(2 * poly, sizeof(u64));
  u64* u = (u64*)malloc(sizeof(u64) * 2 * poly);
  u64* tmp = (u64*)malloc(sizeof(u64) * n);
  u64* qhat = (u64*)malloc(sizeof(u64) * ctw * B);
  memcpy(qhat, qrot, sizeof(u64) * ctw * B);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < 2 * L; ++t) or_ntt(c, t % L, qhat + (size_t)b * ctw + (size_t)t * n);
  mac_group_ct(c, B, qhat, cts, acc3);
  or_relin(c, acc3, rkb, rka, out); /* g = 0: no rotation */
  for (int g = 1; g < G; ++g) {
    mac_group_ct(c, B, qhat, cts + (size_t)g * B * ctw, acc3);
    or_relin(c, acc3, rkb, rka, rel);
    or_ks_inner(c, rel + (size_t)L * n, gs[g], kbs[g], kas[g], u);
    for (int t = 0; t < np; ++t) {
      u64 q = c->primes[t];
      for (int h = 0; h < 2; ++h)
        for (int k = 0; k < n; ++k) {
          size_t o = (size_t)h * poly + (size_t)t * n + k;
          usum[o] = addm(usum[o], u[o], q);
        }
    }
    for (int t = 0; t < L; ++t) {
      u64 q = c->primes[t];
      automorph_poly(n, gs[g], q, rel + (size_t)t * n, tmp);
      for (int k = 0; k < n; ++k) out[(size_t)t * n + k] = addm(out[(size_t)t * n + k], tmp[k], q);
    }
  }
  if (G > 1) {
    u64* d = (u64*)malloc(sizeof(u64) * ptw);
    for (int h = 0; h < 2; ++h) {
      or_moddown(c, usum + (size_t)h * poly, d);
      for (int t = 0; t < L; ++t) {
        u64 q = c->primes[t];
        for (int k = 0; k < n; ++k) {
          size_t o = ((size_t)h * L + t) * n + k;
          out[o] = addm(out[o], d[(size_t)t * n + k], q);
        }
      }
    }
    free(d);
  }
  free(acc3); free(rel); free(usum); free(u); free(tmp); free(qhat);
}

/* ------------------------------------------------------------------ */
/* rescaling and constants (the deep membership path)                   */
/* ------------------------------------------------------------------ */

/* Rescale: divide by the last ciphertext prime q_{L-1} with rounding and drop
 * it.  ct [npolys][L][N] coefficient form -> out [npolys][L-1][N]:
 *   out_t = (c_t - r) * q_{L-1}^{-1} mod q_t,
 * r the centred residue of c mod q_{L-1} (in (-q_{L-1}/2, q_{L-1}/2]), so that
 * out = round(c / q_{L-1}) coefficient-wise. */
void or_rescale(void* p, const u64* ct, int npolys, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
  u64 ql = c->primes[L - 1];
  for (int h = 0; h < npolys; ++h) {
    const u64* last = ct + ((size_t)h * L + L - 1) * n;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < L - 1; ++t) {
      u64 q = c->primes[t];
      u64 inv = powm(ql % q, q - 2, q);
      const u64* src = ct + ((size_t)h * L + t) * n;
      u64* dst = out + ((size_t)h * (L - 1) + t) * n;
      for (int k = 0; k < n; ++k) {
        u64 x = last[k];
        u64 r = x <= (ql - 1) / 2 ? x % q : negm((ql - x) % q, q);
        dst[k] = mulm(subm(src[k], r, q), inv, q);
      }
    }
  }
}

/* out[h][t] = x[h][t] * c_t mod q_t for npolys polynomials over the L
 * ciphertext primes; c: [L] residues of an integer constant. */
void or_mul_const(void* p, const u64* x, int npolys, const u64* cres, u64* out) {
  octx* c = (octx*)p;
  int n = c->n, L = c->L;
  for (int h = 0; h < npolys; ++h)
    for (int t = 0; t < L; ++t) {
      u64 q = c->primes[t];
      for (int k = 0; k < n; ++k) {
        size_t o = ((size_t)h * L + t) * n + k;
        out[o] = mulm(x[o], cres[t], q);
      }
    }
}
