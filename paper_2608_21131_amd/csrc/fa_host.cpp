// Host side of libfa: parameter set-up, the C ABI entry points and the
// orchestration of the encrypted scoring path on the caller's stream.
//
// Paper: Section 2 ("Measured prototype vs. deployment", "Reproducing this")
// for the block-of-n/2-rows-as-d-diagonals scorer; Section 3.1 ("How",
// "Detail") for the diagonal matrix-vector method, baby-step/giant-step with
// plaintext pre-rotation of the database, and the single final fold;
// Section 3.1 ("Membership search") for the threshold path.
//
// In order:
//   errors, modular arithmetic and prime selection;
//   encoding (FFT tables) and the context (tables, level contexts);
//   keys, encryption, decryption and export (test and client side);
//   decoding and enrollment of database blocks and projections;
//   workspace arena, key switching (ModUp, key products, ModDown), rotations,
//     relinearisation, lanes;
//   scoring: baby phase, multiply-accumulate, giant phase, the encrypted-
//     database variant, prepared queries and query batches;
//   the membership path: rescale, ct x ct products, constants, the chain of
//     levels, Chebyshev evaluator, sign iteration, the one-call scan;
//   rotations, rotate-and-sum, phase profiling and the projection.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "fa_internal.h"

using u64 = uint64_t;
using u128 = unsigned __int128;

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
static thread_local std::string g_err;

static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPCHK(x)                                                                  \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) return fail(FA_E_HIP, "%s: %s", #x, hipGetErrorString(e_)); \
  } while (0)

static int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(FA_E_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return FA_OK;
}

// ---------------------------------------------------------------------------
// modular arithmetic on the host (table construction)
// ---------------------------------------------------------------------------
static u64 mulmod(u64 a, u64 b, u64 m) { return (u64)((u128)a * b % m); }
static u64 powmod(u64 b, u64 e, u64 m) {
  u64 r = 1 % m;
  b %= m;
  while (e) {
    if (e & 1) r = mulmod(r, b, m);
    b = mulmod(b, b, m);
    e >>= 1;
  }
  return r;
}
static u64 invmod(u64 a, u64 p) { return powmod(a % p, p - 2, p); }  // p prime

static bool is_prime(u64 n) {
  if (n < 2) return false;
  static const u64 bases[] = {2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37};
  for (u64 p : bases)
    if (n % p == 0) return n == p;
  u64 d = n - 1;
  int r = 0;
  while ((d & 1) == 0) {
    d >>= 1;
    ++r;
  }
  for (u64 a : bases) {
    u64 x = powmod(a, d, n);
    if (x == 1 || x == n - 1) continue;
    bool comp = true;
    for (int i = 1; i < r; ++i) {
      x = mulmod(x, x, n);
      if (x == n - 1) {
        comp = false;
        break;
      }
    }
    if (comp) return false;
  }
  return true;
}

// The `count` largest primes below 2^50 that are 1 mod 2N, descending.
static std::vector<u64> select_primes(int logn, int count) {
  const u64 m = 2ull << logn;
  u64 c = (((1ull << 50) - 2) / m) * m + 1;
  std::vector<u64> out;
  while ((int)out.size() < count && c > m) {
    if (is_prime(c)) out.push_back(c);
    c -= m;
  }
  return out;
}

// A primitive 2N-th root of unity mod q: x^((q-1)/2N) for the first odd x
// giving an element whose N-th power is -1.
static u64 primitive_root_2n(u64 q, int logn) {
  const u64 n = 1ull << logn;
  for (u64 x = 3;; x += 2) {
    u64 y = powmod(x, (q - 1) / (2 * n), q);
    if (powmod(y, n, q) == q - 1) return y;
  }
}

static uint32_t bitrev(uint32_t x, int bits) {
  uint32_t r = 0;
  for (int i = 0; i < bits; ++i) {
    r = (r << 1) | (x & 1);
    x >>= 1;
  }
  return r;
}

static uint32_t galois(int n, long step) {
  const long slots = n / 2;
  long r = ((step % slots) + slots) % slots;
  return (uint32_t)powmod(5, (u64)r, 2ull * n);
}

// ---------------------------------------------------------------------------
// float64 encoding / decoding on the host (client and enrollment side)
// ---------------------------------------------------------------------------
namespace {
using cplx = std::complex<double>;

// Tables of the host transforms for ring degree n, built once per n and
// shared by every context (they depend on n only).
struct FftTables {
  std::vector<cplx> root_fwd, root_inv;  // e^{-2 pi i k / n}, e^{+2 pi i k / n}, k < n/2
  std::vector<cplx> twist;               // e^{i pi k / n}, k < n
  std::vector<u64> e;                    // slot exponents 5^j mod 2n, j < n/2
};
const FftTables& fft_tables(int n) {
  static std::mutex mu;
  static std::map<int, std::unique_ptr<FftTables>> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto& slot = cache[n];
  if (!slot) {
    auto t = std::make_unique<FftTables>();
    t->root_fwd.resize(n / 2);
    t->root_inv.resize(n / 2);
    for (int k = 0; k < n / 2; ++k) {
      const double ang = 2.0 * M_PI * (double)k / (double)n;
      t->root_fwd[k] = cplx(std::cos(ang), -std::sin(ang));
      t->root_inv[k] = cplx(std::cos(ang), std::sin(ang));
    }
    t->twist.resize(n);
    for (int k = 0; k < n; ++k) {
      const double ang = M_PI * (double)k / (double)n;
      t->twist[k] = cplx(std::cos(ang), std::sin(ang));
    }
    t->e.resize(n / 2);
    u64 x = 1;
    for (int j = 0; j < n / 2; ++j) {
      t->e[j] = x;
      x = x * 5 % (2ull * n);
    }
    slot = std::move(t);
  }
  return *slot;
}

// in-place radix-2 FFT of length n with the root table of the wanted sign
// (root_fwd: sum x_t e^{-2 pi i k t / n}; root_inv: e^{+...})
void fft(std::vector<cplx>& a, const std::vector<cplx>& root) {
  const size_t n = a.size();
  for (size_t i = 1, j = 0; i < n; ++i) {
    size_t bit = n >> 1;
    for (; j & bit; bit >>= 1) j ^= bit;
    j ^= bit;
    if (i < j) std::swap(a[i], a[j]);
  }
  for (size_t len = 2; len <= n; len <<= 1) {
    const size_t step = n / len;
    for (size_t s = 0; s < n; s += len)
      for (size_t j = 0; j < len / 2; ++j) {
        const cplx u = a[s + j], v = a[s + j + len / 2] * root[j * step];
        a[s + j] = u + v;
        a[s + j + len / 2] = u - v;
      }
  }
}

const std::vector<u64>& slot_exps(int n) { return fft_tables(n).e; }

// m_k = rint(scale * (2/N) sum_j v_j cos(pi k e_j / N)) via one length-N FFT:
// sum_j v_j (w^{-k e_j} + w^{k e_j}) = w^{-k} sum_t Z_t e^{-2 pi i k t / N},
// w = e^{i pi / N}, Z_t = v_j at t = (e_j - 1)/2 and t = (2N - e_j - 1)/2.
void encode_one(int n, const std::vector<u64>& e, const double* v, int nv, double scale, int64_t* out) {
  const FftTables& tb = fft_tables(n);
  std::vector<cplx> z(n, cplx(0, 0));
  for (int j = 0; j < nv; ++j) {
    z[(e[j] - 1) / 2] = v[j];
    z[(2 * (u64)n - e[j] - 1) / 2] = v[j];
  }
  fft(z, tb.root_fwd);
  for (int k = 0; k < n; ++k) {
    // Re(z_k w^-k), w = e^{i pi / N}
    const double re = z[k].real() * tb.twist[k].real() + z[k].imag() * tb.twist[k].imag();
    out[k] = (int64_t)std::nearbyint(scale * re / (double)n);
  }
}

template <class F>
void parallel_for(int count, F f) {
  int nt = (int)std::thread::hardware_concurrency();
  nt = std::max(1, std::min(nt, 16));
  nt = std::min(nt, count);
  if (nt <= 1) {
    for (int i = 0; i < count; ++i) f(i);
    return;
  }
  std::vector<std::thread> th;
  for (int w = 0; w < nt; ++w)
    th.emplace_back([&, w]() {
      for (int i = w; i < count; i += nt) f(i);
    });
  for (auto& t : th) t.join();
}
}  // namespace

// ---------------------------------------------------------------------------
// context
// ---------------------------------------------------------------------------
template <class T>
static int dev_alloc(T** p, size_t count) {
  hipError_t e = hipMalloc((void**)p, count * sizeof(T));
  if (e != hipSuccess) {
    *p = nullptr;
    return fail(FA_E_NOMEM, "hipMalloc(%zu bytes): %s", count * sizeof(T), hipGetErrorString(e));
  }
  return FA_OK;
}

// ---------------------------------------------------------------------------
// buffer descriptors: every check runs on the host before anything is enqueued
// ---------------------------------------------------------------------------
static size_t obj_bytes(const fa_ctx* c, uint32_t n_polys) { return (size_t)n_polys * c->L * c->n * 8; }

static const char* kind_name(uint32_t n_polys) {
  return n_polys == 1 ? "plaintexts" : n_polys == 2 ? "ciphertexts" : "objects";
}

// An input buffer: at least min_count objects of n_polys polynomials at the
// context's level, its capacity covering its contents.
static int in_check(const fa_ctx* c, const fa_buf* b, const char* fn, const char* what, uint32_t n_polys,
                    uint32_t min_count) {
  if (!b || !b->dev) return fail(FA_E_INVAL, "%s: %s is null", fn, what);
  if (b->n_polys != n_polys)
    return fail(FA_E_SHAPE, "%s: %s holds %u polynomials per object, the call takes %s (%u)", fn, what, b->n_polys,
                kind_name(n_polys), n_polys);
  if ((int)b->limbs != c->L)
    return fail(FA_E_SHAPE, "%s: %s is at %u primes, the context at %d", fn, what, b->limbs, c->L);
  if (b->count < min_count) return fail(FA_E_SHAPE, "%s: %s holds %u %s, at least %u needed", fn, what, b->count,
                                        kind_name(n_polys), min_count);
  if (b->bytes < (size_t)b->count * obj_bytes(c, n_polys))
    return fail(FA_E_SHAPE, "%s: %s claims %u objects in %zu bytes", fn, what, b->count, b->bytes);
  return FA_OK;
}

// An output buffer: room for `objects` objects of n_polys polynomials.
static int out_check(const fa_ctx* c, const fa_buf* b, const char* fn, const char* what, size_t objects,
                     uint32_t n_polys) {
  if (!b || !b->dev) return fail(FA_E_INVAL, "%s: %s is null", fn, what);
  if (b->bytes < objects * obj_bytes(c, n_polys))
    return fail(FA_E_SHAPE, "%s: %s has %zu bytes, %zu %s need %zu", fn, what, b->bytes, objects,
                kind_name(n_polys), objects * obj_bytes(c, n_polys));
  return FA_OK;
}

static void out_set(const fa_ctx* c, fa_buf* b, uint32_t n_polys, size_t count, int32_t log_scale) {
  b->n_polys = n_polys;
  b->count = (uint32_t)count;
  b->limbs = (uint32_t)c->L;
  b->log_scale = log_scale;
}

// log2 of the ciphertext modulus Q
static double log2_q(const fa_ctx* c) {
  double v = 0.0;
  for (int t = 0; t < c->L; ++t) v += std::log2((double)c->primes[t]);
  return v;
}

// A product's scale must leave room below Q/2 for values of magnitude up to
// 2^7 (sums of d products of unit entries, plus noise), else it wraps mod Q.
static int scale_check(const fa_ctx* c, const char* fn, long log_scale) {
  if (log_scale < 0 || (double)log_scale > log2_q(c) - 8.0)
    return fail(FA_E_SHAPE, "%s: the product scale 2^%ld does not fit below Q = 2^%.1f with 8 bits to spare", fn,
                log_scale, log2_q(c));
  return FA_OK;
}

static bool overlap(const fa_buf* a, const fa_buf* b) {
  const char* a0 = (const char*)a->dev;
  const char* b0 = (const char*)b->dev;
  return a0 < b0 + b->bytes && b0 < a0 + a->bytes;
}

// The blocks a scoring request names: ids[j] (or j when ids is null) among the
// n_resident resident blocks, each holding at least min_count objects of
// n_polys polynomials at the context's level, all at one scale.
static int gather_blocks(const fa_ctx* c, const char* fn, const fa_buf* blocks, int n_resident, const int32_t* ids,
                         int n_blocks, uint32_t n_polys, uint32_t min_count, std::vector<const double*>& ptrs,
                         int32_t* log_scale) {
  if (n_blocks < 1) return fail(FA_E_SHAPE, "%s: n_blocks must be positive", fn);
  if (!blocks) return fail(FA_E_INVAL, "%s: null block list", fn);
  if (n_resident < 1) return fail(FA_E_SHAPE, "%s: n_resident must be positive", fn);
  if (!ids && n_blocks > n_resident)
    return fail(FA_E_SHAPE, "%s: %d blocks requested without ids from %d resident", fn, n_blocks, n_resident);
  ptrs.resize(n_blocks);
  for (int j = 0; j < n_blocks; ++j) {
    const int id = ids ? ids[j] : j;
    if (id < 0 || id >= n_resident) return fail(FA_E_INVAL, "%s: block id %d outside [0, %d)", fn, id, n_resident);
    char what[48];
    snprintf(what, sizeof what, "block %d", id);
    int rc = in_check(c, &blocks[id], fn, what, n_polys, min_count);
    if (rc) return rc;
    if (j == 0) *log_scale = blocks[id].log_scale;
    else if (blocks[id].log_scale != *log_scale)
      return fail(FA_E_SHAPE, "%s: block %d is at scale 2^%d, block %d at 2^%d", fn, id, blocks[id].log_scale,
                  ids ? ids[0] : 0, *log_scale);
    ptrs[j] = (const double*)blocks[id].dev;
  }
  return FA_OK;
}

extern "C" {

const char* fa_last_error(void) { return g_err.c_str(); }

void fa_ctx_destroy(fa_ctx* c) {
  if (!c) return;
  (void)hipFree(c->d_pr);
  (void)hipFree(c->d_twa_fwd);
  (void)hipFree(c->d_twa_inv);
  (void)hipFree(c->d_twt_fwd);
  (void)hipFree(c->d_twt_inv);
  (void)hipFree(c->d_twr_fwd);
  (void)hipFree(c->d_twr_inv);
  (void)hipFree(c->d_mu_hat);
  (void)hipFree(c->d_md_hat);
  (void)hipFree(c->d_mu_scale);
  (void)hipFree(c->d_md_scale);
  (void)hipFree(c->d_s);
  for (auto& kv : c->keys) (void)hipFree(kv.second);
  (void)hipFree(c->d_rlk);
  for (auto& e : c->ev)
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < c->n_aux; ++i) {
    (void)hipStreamDestroy(c->aux[i]);
    (void)hipEventDestroy(c->join_ev[i]);
  }
  if (c->fork_ev) (void)hipEventDestroy(c->fork_ev);
  if (c->side) (void)hipStreamDestroy(c->side);
  if (c->side_fork) (void)hipEventDestroy(c->side_fork);
  if (c->side_join) (void)hipEventDestroy(c->side_join);
  (void)hipFree(c->d_export);
  delete c;
}

}  // extern "C"

// Builds a context over an explicit prime list (L ciphertext primes, then K special primes).
static int ctx_build(const fa_params* prm, const std::vector<u64>& primes, fa_ctx** out) {
  fa_ctx* c = new (std::nothrow) fa_ctx();
  if (!c) return fail(FA_E_NOMEM, "out of host memory");
  c->logn = (int)prm->log_n;
  c->n = 1 << c->logn;
  c->L = (int)prm->L;
  c->K = (int)prm->K;
  c->np = c->L + c->K;
  c->alpha = c->K;
  c->dnum = (c->L + c->K - 1) / c->K;
  c->log_scale = (int)prm->log_scale;
  (void)hipGetDevice(&c->device);
  // set-up of fa_rotate_static: the fixed scratch array's address on this device
  c->static_scratch = fa::static_scratch(c->device, &c->static_scratch_err);
  c->primes = primes;
  const int n = c->n, np = c->np, L = c->L, K = c->K;
  // P mod q_t, P^-1 mod q_t
  c->p_mod_q.assign(L, 0);
  std::vector<DevPrime> hp(np);
  for (int t = 0; t < np; ++t) {
    const u64 q = c->primes[t];
    hp[t].q = (double)q;
    hp[t].qinv = 1.0 / (double)q;
    hp[t].ninv = (double)invmod((u64)n, q);
    hp[t].pinv = 0.0;
    hp[t].pmod = 0.0;
    if (t < L) {
      u64 pm = 1;
      for (int k = 0; k < K; ++k) pm = mulmod(pm, c->primes[L + k] % q, q);
      c->p_mod_q[t] = pm;
      hp[t].pmod = (double)pm;
      hp[t].pinv = (double)invmod(pm, q);
    }
  }
  // twiddles: first-pass table psi^{brev(k)} (k < 256), second-pass table T and
  // per-row factors F (see fa_kernels.hip), each also for psi^-1
  const int SA = c->logn - 8, H = 1 << SA;
  std::vector<double> twa_f((size_t)np * 256), twa_i((size_t)np * 256), twt_f((size_t)np * 256),
      twt_i((size_t)np * 256), twr_f((size_t)np * H * 8), twr_i((size_t)np * H * 8);
  c->psi.resize(np);
  c->h_ninv.resize(np);
  for (int t = 0; t < np; ++t) {
    const u64 q = c->primes[t];
    const u64 psi = primitive_root_2n(q, c->logn);
    const u64 ipsi = invmod(psi, q);
    c->psi[t] = psi;
    c->h_ninv[t] = hp[t].ninv;
    for (int k = 0; k < 256; ++k) {
      const u64 e = bitrev((uint32_t)k, c->logn);
      twa_f[(size_t)t * 256 + k] = (double)powmod(psi, e, q);
      twa_i[(size_t)t * 256 + k] = (double)powmod(ipsi, e, q);
    }
    twt_f[(size_t)t * 256] = 1.0;
    twt_i[(size_t)t * 256] = 1.0;
    for (int s1 = 0; s1 < 8; ++s1)
      for (int i1 = 0; i1 < (1 << s1); ++i1) {
        const u64 e = (u64)bitrev((uint32_t)i1, s1) * (u64)(n >> s1);
        twt_f[(size_t)t * 256 + (1 << s1) + i1] = (double)powmod(psi, e, q);
        twt_i[(size_t)t * 256 + (1 << s1) + i1] = (double)powmod(ipsi, e, q);
      }
    for (int r = 0; r < H; ++r) {
      const u64 e0 = 2 * (u64)bitrev((uint32_t)r, SA) + 1;
      for (int s1 = 0; s1 < 8; ++s1) {
        const u64 e = e0 << (7 - s1);
        twr_f[((size_t)t * H + r) * 8 + s1] = (double)powmod(psi, e, q);
        twr_i[((size_t)t * H + r) * 8 + s1] = (double)powmod(ipsi, e, q);
      }
    }
  }
  // basis-conversion constants: products of primes reduced prime by prime;
  // the inverse factors are folded into the scaling of the inverse transforms
  std::vector<double> mu_hat((size_t)c->dnum * c->alpha * np, 0.0);
  c->h_mu_scale.assign(L, 0.0);
  for (int i = 0; i < c->dnum; ++i) {
    const int lo = i * c->alpha, hi = std::min(lo + c->alpha, L);
    for (int j = lo; j < hi; ++j) {
      // (D_i / d_j) mod every prime t, and its inverse mod d_j
      for (int t = 0; t < np; ++t) {
        u64 v = 1;
        for (int jj = lo; jj < hi; ++jj)
          if (jj != j) v = mulmod(v, c->primes[jj] % c->primes[t], c->primes[t]);
        mu_hat[((size_t)i * c->alpha + (j - lo)) * np + t] = (double)v;
      }
      u64 v = 1;
      for (int jj = lo; jj < hi; ++jj)
        if (jj != j) v = mulmod(v, c->primes[jj] % c->primes[j], c->primes[j]);
      const u64 q = c->primes[j];
      c->h_mu_scale[j] = (double)mulmod(invmod(v, q), invmod((u64)n, q), q);
    }
  }
  std::vector<double> md_hat((size_t)K * L);
  c->h_md_scale.assign(K, 0.0);
  for (int k = 0; k < K; ++k) {
    const u64 pk = c->primes[L + k];
    u64 v = 1;
    for (int kk = 0; kk < K; ++kk)
      if (kk != k) v = mulmod(v, c->primes[L + kk] % pk, pk);
    c->h_md_scale[k] = (double)mulmod(invmod(v, pk), invmod((u64)n, pk), pk);
    for (int t = 0; t < L; ++t) {
      const u64 q = c->primes[t];
      u64 w = 1;
      for (int kk = 0; kk < K; ++kk)
        if (kk != k) w = mulmod(w, c->primes[L + kk] % q, q);
      md_hat[(size_t)k * L + t] = (double)w;
    }
  }
  int rc;
  if ((rc = dev_alloc(&c->d_pr, np)) || (rc = dev_alloc(&c->d_twa_fwd, twa_f.size())) ||
      (rc = dev_alloc(&c->d_twa_inv, twa_i.size())) || (rc = dev_alloc(&c->d_twt_fwd, twt_f.size())) ||
      (rc = dev_alloc(&c->d_twt_inv, twt_i.size())) || (rc = dev_alloc(&c->d_twr_fwd, twr_f.size())) ||
      (rc = dev_alloc(&c->d_twr_inv, twr_i.size())) || (rc = dev_alloc(&c->d_mu_hat, mu_hat.size())) ||
      (rc = dev_alloc(&c->d_md_hat, md_hat.size())) || (rc = dev_alloc(&c->d_mu_scale, (size_t)L)) ||
      (rc = dev_alloc(&c->d_md_scale, (size_t)K)) ||
      (rc = dev_alloc(&c->d_s, (size_t)np * n))) {
    fa_ctx_destroy(c);
    return rc;
  }
  hipError_t e = hipSuccess;
  auto up = [&](double* d, const std::vector<double>& h) {
    if (e == hipSuccess) e = hipMemcpy(d, h.data(), h.size() * 8, hipMemcpyHostToDevice);
  };
  if (e == hipSuccess) e = hipMemcpy(c->d_pr, hp.data(), np * sizeof(DevPrime), hipMemcpyHostToDevice);
  up(c->d_twa_fwd, twa_f);
  up(c->d_twa_inv, twa_i);
  up(c->d_twt_fwd, twt_f);
  up(c->d_twt_inv, twt_i);
  up(c->d_twr_fwd, twr_f);
  up(c->d_twr_inv, twr_i);
  up(c->d_mu_hat, mu_hat);
  up(c->d_md_hat, md_hat);
  up(c->d_mu_scale, c->h_mu_scale);
  up(c->d_md_scale, c->h_md_scale);
  if (e == hipSuccess) e = hipMemset(c->d_s, 0, (size_t)np * n * 8);
  if (e != hipSuccess) {
    fa_ctx_destroy(c);
    return fail(FA_E_HIP, "fa_ctx_create: %s", hipGetErrorString(e));
  }
  *out = c;
  return FA_OK;
}

extern "C" {

int fa_ctx_create(const fa_params* prm, fa_ctx** out) {
  if (!prm || !out) return fail(FA_E_INVAL, "fa_ctx_create: null argument");
  if (prm->log_n < 10 || prm->log_n > 16) return fail(FA_E_INVAL, "log_n must be in [10, 16], got %u", prm->log_n);
  if (prm->L < 1 || prm->L > 16) return fail(FA_E_INVAL, "L must be in [1, 16], got %u", prm->L);
  if (prm->K < 1 || prm->K > 4) return fail(FA_E_INVAL, "K must be in [1, 4], got %u", prm->K);
  // the key-switch kernels are instantiated for 1..8 digits
  if ((prm->L + prm->K - 1) / prm->K > 8)
    return fail(FA_E_INVAL, "L=%u, K=%u gives %u key-switch digits; at most 8 are supported", prm->L, prm->K,
                (prm->L + prm->K - 1) / prm->K);
  if (prm->log_scale < 1 || prm->log_scale > 60) return fail(FA_E_INVAL, "log_scale must be in [1, 60]");
  const int np = (int)(prm->L + prm->K);
  std::vector<u64> primes;
  if (prm->primes) {
    // explicit primes: the residue arithmetic needs them in (2^49, 2^50), the
    // negacyclic transform needs 2N | q - 1, and the CRT needs them distinct
    const u64 m = 2ull << prm->log_n;
    for (int t = 0; t < np; ++t) {
      const u64 q = prm->primes[t];
      if (q <= (1ull << 49) || q >= (1ull << 50)) return fail(FA_E_INVAL, "prime %d = %llu is not in (2^49, 2^50)", t, (unsigned long long)q);
      if (q % m != 1) return fail(FA_E_INVAL, "prime %d = %llu is not 1 mod 2N", t, (unsigned long long)q);
      if (!is_prime(q)) return fail(FA_E_INVAL, "%llu (entry %d) is not prime", (unsigned long long)q, t);
      for (int u = 0; u < t; ++u)
        if (prm->primes[u] == q) return fail(FA_E_INVAL, "prime %llu is listed twice", (unsigned long long)q);
      primes.push_back(q);
    }
  } else {
    primes = select_primes((int)prm->log_n, np);
    if ((int)primes.size() != np) return fail(FA_E_INVAL, "not enough 50-bit NTT primes");
  }
  return ctx_build(prm, primes, out);
}

int fa_ctx_create_level(const fa_ctx* parent, uint32_t L_low, fa_ctx** out) {
  if (!parent || !out) return fail(FA_E_INVAL, "fa_ctx_create_level: null argument");
  if (L_low < 1 || (int)L_low > parent->L) return fail(FA_E_INVAL, "L_low=%u must be in [1, %d]", L_low, parent->L);
  const fa_params prm{(uint32_t)parent->logn, L_low, (uint32_t)parent->K, (uint32_t)parent->log_scale, nullptr};
  std::vector<u64> primes(parent->primes.begin(), parent->primes.begin() + L_low);
  primes.insert(primes.end(), parent->primes.begin() + parent->L, parent->primes.end());
  fa_ctx* c = nullptr;
  int rc = ctx_build(&prm, primes, &c);
  if (rc) return rc;
  // restrict the parent's secret and rotation keys (NTT-form limbs per prime:
  // both contexts use the same root per prime, so the limbs carry over)
  const size_t n = c->n;
  hipError_t e = hipSuccess;
  auto limb_src = [&](int t) { return t < (int)L_low ? t : parent->L + (t - (int)L_low); };
  for (int t = 0; t < c->np && e == hipSuccess; ++t)
    e = hipMemcpy(c->d_s + (size_t)t * n, parent->d_s + (size_t)limb_src(t) * n, n * 8, hipMemcpyDeviceToDevice);
  // every key (rotations and relinearisation) restricted the same way
  std::vector<std::pair<const double*, double**>> todo;
  for (auto& kv : parent->keys) todo.push_back({kv.second, &c->keys[kv.first]});
  if (parent->d_rlk) todo.push_back({parent->d_rlk, &c->d_rlk});
  for (auto& kt : todo) {
    if (e != hipSuccess) break;
    double* key = nullptr;
    if ((rc = dev_alloc(&key, (size_t)c->dnum * 2 * c->np * n))) {
      fa_ctx_destroy(c);
      return rc;
    }
    *kt.second = key;
    for (int i = 0; i < c->dnum && e == hipSuccess; ++i)
      for (int h = 0; h < 2 && e == hipSuccess; ++h)
        for (int t = 0; t < c->np && e == hipSuccess; ++t)
          e = hipMemcpy(key + (((size_t)i * 2 + h) * c->np + t) * n,
                        kt.first + (((size_t)i * 2 + h) * parent->np + limb_src(t)) * n, n * 8,
                        hipMemcpyDeviceToDevice);
  }
  if (e != hipSuccess) {
    fa_ctx_destroy(c);
    return fail(FA_E_HIP, "fa_ctx_create_level: %s", hipGetErrorString(e));
  }
  *out = c;
  return FA_OK;
}

int fa_drop_level(const fa_ctx* parent, const fa_ctx* child, const fa_buf* ct, fa_buf* out, void* stream) {
  if (!parent || !child) return fail(FA_E_INVAL, "fa_drop_level: null context");
  if (child->n != parent->n || child->L > parent->L) return fail(FA_E_SHAPE, "fa_drop_level: not a lower level");
  for (int t = 0; t < child->L; ++t)
    if (child->primes[t] != parent->primes[t]) return fail(FA_E_SHAPE, "fa_drop_level: prime %d differs", t);
  int rc = in_check(parent, ct, "fa_drop_level", "ct", 2, 1);
  if (rc || (rc = out_check(child, out, "fa_drop_level", "out", ct->count, 2))) return rc;
  const size_t n = parent->n;
  hipStream_t s = (hipStream_t)stream;
  for (uint32_t j = 0; j < ct->count; ++j)
    for (int h = 0; h < 2; ++h)
      HIPCHK(hipMemcpyAsync((double*)out->dev + ((size_t)2 * j + h) * child->L * n,
                            (const double*)ct->dev + ((size_t)2 * j + h) * parent->L * n, (size_t)child->L * n * 8,
                            hipMemcpyDeviceToDevice, s));
  out_set(child, out, 2, ct->count, ct->log_scale);
  return FA_OK;
}

int fa_ctx_primes(const fa_ctx* c, uint64_t* out) {
  if (!c || !out) return fail(FA_E_INVAL, "fa_ctx_primes: null argument");
  std::copy(c->primes.begin(), c->primes.end(), out);
  return FA_OK;
}
size_t fa_ct_bytes(const fa_ctx* c) { return c ? obj_bytes(c, 2) : 0; }
size_t fa_pt_bytes(const fa_ctx* c) { return c ? obj_bytes(c, 1) : 0; }
size_t fa_key_bytes(const fa_ctx* c) { return c ? (size_t)c->dnum * 2 * c->np * c->n * 8 : 0; }

// ---------------------------------------------------------------------------
// secret, keys, encryption
// ---------------------------------------------------------------------------
int fa_set_secret(fa_ctx* c, const int64_t* s) {
  if (!c || !s) return fail(FA_E_INVAL, "fa_set_secret: null argument");
  for (int k = 0; k < c->n; ++k)
    if (s[k] < -1 || s[k] > 1) return fail(FA_E_INVAL, "secret coefficient %d is not ternary", k);
  int64_t* ds = nullptr;
  int rc = dev_alloc(&ds, c->n);
  if (rc) return rc;
  HIPCHK(hipMemcpy(ds, s, (size_t)c->n * 8, hipMemcpyHostToDevice));
  fa::int_to_res(c, ds, 1, c->np, c->d_s, 0);
  fa::ntt_fwd_strided(c, c->d_s, c->n, c->np, c->np, 0, 0);
  if ((rc = check_launch("fa_set_secret"))) return rc;
  HIPCHK(hipDeviceSynchronize());
  (void)hipFree(ds);
  return FA_OK;
}

int fa_keygen(fa_ctx* c, const int64_t* s, const int32_t* steps, int n_steps, const uint64_t* a, const int64_t* e) {
  if (!c || !s || (!steps && n_steps) || (!a && n_steps) || (!e && n_steps) || n_steps < 0)
    return fail(FA_E_INVAL, "fa_keygen: bad argument");
  for (int i = 0; i < n_steps; ++i)
    if (steps[i] < 1 || steps[i] >= c->n / 2) return fail(FA_E_INVAL, "rotation step %d out of [1, N/2)", steps[i]);
  int rc = fa_set_secret(c, s);
  if (rc) return rc;
  const size_t n = c->n, np = c->np, dnum = c->dnum;
  const size_t key_words = dnum * 2 * np * n;
  uint64_t* du = nullptr;
  int64_t* de = nullptr;
  double* den = nullptr;
  if ((rc = dev_alloc(&du, dnum * np * n)) || (rc = dev_alloc(&de, dnum * n)) ||
      (rc = dev_alloc(&den, dnum * np * n))) {
    (void)hipFree(du);
    (void)hipFree(de);
    return rc;
  }
  for (int r = 0; r < n_steps; ++r) {
    double* key = nullptr;
    auto it = c->keys.find(steps[r]);
    if (it != c->keys.end()) {
      key = it->second;
    } else {
      if ((rc = dev_alloc(&key, key_words))) break;
      c->keys[steps[r]] = key;
    }
    const uint64_t* ar = a + (size_t)r * dnum * np * n;
    const int64_t* er = e + (size_t)r * dnum * n;
    hipError_t he = hipMemcpy(du, ar, dnum * np * n * 8, hipMemcpyHostToDevice);
    if (he == hipSuccess) he = hipMemcpy(de, er, dnum * n * 8, hipMemcpyHostToDevice);
    if (he != hipSuccess) {
      rc = fail(FA_E_HIP, "fa_keygen upload: %s", hipGetErrorString(he));
      break;
    }
    // a part (digit i, slot 1) <- NTT(a_i); e residues -> NTT
    for (size_t i = 0; i < dnum; ++i)
      fa::u64_to_res(du + i * np * n, np * n, key + (i * 2 + 1) * np * n, 0);
    for (size_t i = 0; i < dnum; ++i) fa::ntt_fwd_strided(c, key + (i * 2 + 1) * np * n, n, (int)np, (int)np, 0, 0);
    fa::int_to_res(c, de, (int)dnum, (int)np, den, 0);
    fa::ntt_fwd_strided(c, den, n, (int)(dnum * np), (int)np, 0, 0);
    fa::keygen_combine(c, key, den, galois(c->n, steps[r]), 0);
    if ((rc = check_launch("fa_keygen"))) break;
    he = hipDeviceSynchronize();
    if (he != hipSuccess) {
      rc = fail(FA_E_HIP, "fa_keygen: %s", hipGetErrorString(he));
      break;
    }
  }
  (void)hipFree(du);
  (void)hipFree(de);
  (void)hipFree(den);
  return rc;
}

int fa_has_key(const fa_ctx* c, int step) { return c && c->keys.count(step) ? 1 : 0; }

int fa_keygen_relin(fa_ctx* c, const int64_t* s, const uint64_t* a, const int64_t* e) {
  if (!c || !s || !a || !e) return fail(FA_E_INVAL, "fa_keygen_relin: null argument");
  int rc = fa_set_secret(c, s);
  if (rc) return rc;
  const size_t n = c->n, np = c->np, dnum = c->dnum;
  if (!c->d_rlk && (rc = dev_alloc(&c->d_rlk, dnum * 2 * np * n))) return rc;
  double* key = c->d_rlk;
  uint64_t* du = nullptr;
  int64_t* de = nullptr;
  double* den = nullptr;
  if ((rc = dev_alloc(&du, dnum * np * n)) || (rc = dev_alloc(&de, dnum * n)) ||
      (rc = dev_alloc(&den, dnum * np * n))) {
    (void)hipFree(du);
    (void)hipFree(de);
    return rc;
  }
  hipError_t he = hipMemcpy(du, a, dnum * np * n * 8, hipMemcpyHostToDevice);
  if (he == hipSuccess) he = hipMemcpy(de, e, dnum * n * 8, hipMemcpyHostToDevice);
  if (he != hipSuccess) {
    rc = fail(FA_E_HIP, "fa_keygen_relin upload: %s", hipGetErrorString(he));
  } else {
    for (size_t i = 0; i < dnum; ++i) fa::u64_to_res(du + i * np * n, np * n, key + (i * 2 + 1) * np * n, 0);
    for (size_t i = 0; i < dnum; ++i) fa::ntt_fwd_strided(c, key + (i * 2 + 1) * np * n, n, (int)np, (int)np, 0, 0);
    fa::int_to_res(c, de, (int)dnum, (int)np, den, 0);
    fa::ntt_fwd_strided(c, den, n, (int)(dnum * np), (int)np, 0, 0);
    fa::keygen_combine(c, key, den, 0u, 0);  // gal 0: gadget times s^2
    rc = check_launch("fa_keygen_relin");
    if (!rc && (he = hipDeviceSynchronize()) != hipSuccess) rc = fail(FA_E_HIP, "fa_keygen_relin: %s", hipGetErrorString(he));
  }
  (void)hipFree(du);
  (void)hipFree(de);
  (void)hipFree(den);
  return rc;
}

int fa_has_relin_key(const fa_ctx* c) { return c && c->d_rlk ? 1 : 0; }


int fa_encrypt(fa_ctx* c, const int64_t* m, int32_t log_scale, const uint64_t* a, const int64_t* e, fa_buf* ct,
               void* stream) {
  if (!c || !m || !a || !e) return fail(FA_E_INVAL, "fa_encrypt: null argument");
  int rc0 = out_check(c, ct, "fa_encrypt", "ct", 1, 2);
  if (rc0) return rc0;
  if (log_scale < 0 || log_scale > 1000) return fail(FA_E_INVAL, "fa_encrypt: log_scale %d out of range", log_scale);
  hipStream_t s = (hipStream_t)stream;
  const size_t n = c->n, L = c->L;
  for (size_t k = 0; k < n; ++k)
    if (m[k] > (INT64_C(1) << 62) || m[k] < -(INT64_C(1) << 62) || e[k] > 1024 || e[k] < -1024)
      return fail(FA_E_INVAL, "fa_encrypt: coefficient %zu out of range", k);
  std::vector<int64_t> me(n);
  for (size_t k = 0; k < n; ++k) me[k] = m[k] + e[k];
  uint64_t* du = nullptr;
  int64_t* dm = nullptr;
  double* dv = nullptr;
  int rc;
  if ((rc = dev_alloc(&du, L * n)) || (rc = dev_alloc(&dm, n)) || (rc = dev_alloc(&dv, L * n))) {
    (void)hipFree(du);
    (void)hipFree(dm);
    return rc;
  }
  double* dct = (double*)ct->dev;
  HIPCHK(hipMemcpyAsync(du, a, L * n * 8, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(dm, me.data(), n * 8, hipMemcpyHostToDevice, s));
  fa::u64_to_res(du, L * n, dct + L * n, s);
  fa::ntt_fwd_strided(c, dct + L * n, n, (int)L, (int)L, 0, s);
  fa::int_to_res(c, dm, 1, (int)L, dv, s);
  fa::ntt_fwd_strided(c, dv, n, (int)L, (int)L, 0, s);
  fa::enc_combine(c, dct, dv, s);
  if ((rc = check_launch("fa_encrypt"))) return rc;
  HIPCHK(hipStreamSynchronize(s));
  (void)hipFree(du);
  (void)hipFree(dm);
  (void)hipFree(dv);
  out_set(c, ct, 2, 1, log_scale);
  return FA_OK;
}

int fa_encrypt_pts(fa_ctx* c, const fa_buf* pts_b, const uint64_t* a, const int64_t* e, fa_buf* cts_b,
                   void* stream) {
  if (!c || !a || !e) return fail(FA_E_INVAL, "fa_encrypt_pts: null argument");
  int rc0 = in_check(c, pts_b, "fa_encrypt_pts", "pts", 1, 1);
  if (rc0 || (rc0 = out_check(c, cts_b, "fa_encrypt_pts", "cts", pts_b->count, 2))) return rc0;
  const int n_pts = (int)pts_b->count;
  const void* pts = pts_b->dev;
  void* cts = cts_b->dev;
  hipStream_t s = (hipStream_t)stream;
  const size_t n = c->n, L = c->L;
  for (size_t k = 0; k < (size_t)n_pts * n; ++k)
    if (e[k] > 1024 || e[k] < -1024) return fail(FA_E_INVAL, "fa_encrypt_pts: noise coefficient %zu out of range", k);
  const int chunk = 16;
  uint64_t* du = nullptr;
  int64_t* de = nullptr;
  double* dv = nullptr;
  int rc;
  if ((rc = dev_alloc(&du, (size_t)chunk * L * n)) || (rc = dev_alloc(&de, (size_t)chunk * n)) ||
      (rc = dev_alloc(&dv, (size_t)chunk * L * n))) {
    (void)hipFree(du);
    (void)hipFree(de);
    return rc;
  }
  const double* dp = (const double*)pts;
  double* dc = (double*)cts;
  hipError_t he = hipSuccess;
  for (int p0 = 0; p0 < n_pts && he == hipSuccess && !rc; p0 += chunk) {
    const int m = std::min(chunk, n_pts - p0);
    he = hipMemcpyAsync(du, a + (size_t)p0 * L * n, (size_t)m * L * n * 8, hipMemcpyHostToDevice, s);
    if (he == hipSuccess) he = hipMemcpyAsync(de, e + (size_t)p0 * n, (size_t)m * n * 8, hipMemcpyHostToDevice, s);
    if (he != hipSuccess) break;
    // v = NTT(e) + m (the plaintexts are already in NTT form); c1 = NTT(a); c0 = -c1 s + v
    fa::int_to_res(c, de, m, (int)L, dv, s);
    fa::ntt_fwd_strided(c, dv, n, m * (int)L, (int)L, 0, s);
    fa::add_limbs(c, dv, dp + (size_t)p0 * L * n, m * (int)L, (int)L, s);
    for (int j = 0; j < m; ++j) {
      double* ct = dc + (size_t)(p0 + j) * 2 * L * n;
      fa::u64_to_res(du + (size_t)j * L * n, L * n, ct + L * n, s);
      fa::ntt_fwd_strided(c, ct + L * n, n, (int)L, (int)L, 0, s);
      fa::enc_combine(c, ct, dv + (size_t)j * L * n, s);
    }
    rc = check_launch("fa_encrypt_pts");
    if (!rc) he = hipStreamSynchronize(s);
  }
  (void)hipFree(du);
  (void)hipFree(de);
  (void)hipFree(dv);
  if (!rc && he != hipSuccess) rc = fail(FA_E_HIP, "fa_encrypt_pts: %s", hipGetErrorString(he));
  if (!rc) out_set(c, cts_b, 2, n_pts, pts_b->log_scale);
  return rc;
}

static int export_polys(fa_ctx* c, const double* src, int n_polys, uint64_t* out, hipStream_t s, bool decrypt) {
  const size_t n = c->n, L = c->L;
  const size_t words = (size_t)n_polys * L * n;
  std::lock_guard<std::mutex> lock(c->export_mu);
  if (c->export_words < words) {
    if (c->d_export) {
      HIPCHK(hipStreamSynchronize(s));
      (void)hipFree(c->d_export);
      c->d_export = nullptr;
      c->export_words = 0;
    }
    int rc = dev_alloc(&c->d_export, 2 * words);
    if (rc) return rc;
    c->export_words = words;
  }
  double* tmp = c->d_export;
  uint64_t* du = reinterpret_cast<uint64_t*>(c->d_export + c->export_words);
  if (decrypt) {
    fa::dec_combine(c, src, tmp, s);
  } else {
    HIPCHK(hipMemcpyAsync(tmp, src, words * 8, hipMemcpyDeviceToDevice, s));
  }
  fa::ntt_inv_strided(c, tmp, n, (int)(n_polys * L), (int)L, 0, s);
  fa::res_to_u64(tmp, words, du, s);
  int rc = check_launch("export");
  if (rc) return rc;
  HIPCHK(hipMemcpyAsync(out, du, words * 8, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  return FA_OK;
}

int fa_decrypt(fa_ctx* c, const fa_buf* ct, uint64_t* out, void* stream) {
  if (!c || !out) return fail(FA_E_INVAL, "fa_decrypt: null argument");
  int rc = in_check(c, ct, "fa_decrypt", "ct", 2, 1);
  if (rc) return rc;
  return export_polys(c, (const double*)ct->dev, 1, out, (hipStream_t)stream, true);
}

int fa_import_coeffs(fa_ctx* c, const uint64_t* coeffs, fa_buf* buf, void* stream) {
  if (!c || !coeffs || !buf || !buf->dev) return fail(FA_E_INVAL, "fa_import_coeffs: null argument");
  if (buf->n_polys < 1 || buf->n_polys > 3 || buf->count < 1)
    return fail(FA_E_SHAPE, "fa_import_coeffs: %u objects of %u polynomials", buf->count, buf->n_polys);
  int rc0 = in_check(c, buf, "fa_import_coeffs", "buf", buf->n_polys, 1);
  if (rc0) return rc0;
  const int n_polys = (int)(buf->n_polys * buf->count);
  const size_t n = c->n, L = c->L;
  for (size_t p = 0; p < (size_t)n_polys; ++p)
    for (size_t t = 0; t < L; ++t) {
      const uint64_t* r = coeffs + (p * L + t) * n;
      for (size_t k = 0; k < n; ++k)
        if (r[k] >= c->primes[t])
          return fail(FA_E_INVAL, "fa_import_coeffs: residue %zu of polynomial %zu, limb %zu is not below its prime",
                      k, p, t);
    }
  hipStream_t s = (hipStream_t)stream;
  const int chunk = 16;  // polynomials staged per copy
  uint64_t* du = nullptr;
  int rc = dev_alloc(&du, (size_t)std::min(chunk, n_polys) * L * n);
  if (rc) return rc;
  double* dst = (double*)buf->dev;
  for (int p0 = 0; p0 < n_polys && !rc; p0 += chunk) {
    const int m = std::min(chunk, n_polys - p0);
    const size_t words = (size_t)m * L * n;
    hipError_t he = hipMemcpyAsync(du, coeffs + (size_t)p0 * L * n, words * 8, hipMemcpyHostToDevice, s);
    if (he != hipSuccess) {
      rc = fail(FA_E_HIP, "fa_import_coeffs: %s", hipGetErrorString(he));
      break;
    }
    double* d = dst + (size_t)p0 * L * n;
    fa::u64_to_res(du, words, d, s);
    fa::ntt_fwd_strided(c, d, n, m * (int)L, (int)L, 0, s);
    rc = check_launch("fa_import_coeffs");
    he = hipStreamSynchronize(s);  // the staging buffer is reused by the next chunk
    if (!rc && he != hipSuccess) rc = fail(FA_E_HIP, "fa_import_coeffs: %s", hipGetErrorString(he));
  }
  (void)hipFree(du);
  return rc;
}

int fa_export_coeffs(fa_ctx* c, const fa_buf* buf, uint64_t* out, void* stream) {
  if (!c || !buf || !out) return fail(FA_E_INVAL, "fa_export_coeffs: null argument");
  if (buf->n_polys < 1 || buf->n_polys > 3 || buf->count < 1)
    return fail(FA_E_SHAPE, "fa_export_coeffs: %u objects of %u polynomials", buf->count, buf->n_polys);
  int rc = in_check(c, buf, "fa_export_coeffs", "buf", buf->n_polys, 1);
  if (rc) return rc;
  return export_polys(c, (const double*)buf->dev, (int)(buf->n_polys * buf->count), out, (hipStream_t)stream, false);
}

// ---------------------------------------------------------------------------
// encoding
// ---------------------------------------------------------------------------
int fa_encode(const fa_ctx* c, const double* slots, int n_slots, int log_scale, int64_t* out) {
  if (!c || !slots || !out) return fail(FA_E_INVAL, "fa_encode: null argument");
  if (n_slots < 0 || n_slots > c->n / 2) return fail(FA_E_SHAPE, "fa_encode: n_slots %d > N/2", n_slots);
  if (log_scale < 0 || log_scale > 61) return fail(FA_E_INVAL, "fa_encode: log_scale out of range");
  const std::vector<u64>& e = slot_exps(c->n);
  encode_one(c->n, e, slots, n_slots, std::ldexp(1.0, log_scale), out);
  return FA_OK;
}

}  // extern "C"

// Centred CRT of nl residues -> double by balanced mixed radix (Garner):
// x = a_0 + q_0 (a_1 + q_1 (a_2 + ...)) with every digit a_i in
// [-(q_i-1)/2, (q_i-1)/2].  For odd moduli these representations cover exactly
// the centred range [-(Q-1)/2, (Q-1)/2], so the digits are those of the centred
// residue.  Digit j: v = x mod q_j, then v <- (v - a_i) q_i^-1 mod q_j for
// i < j.  Every prime lies in (2^49, 2^50), so |a_i| < q_i / 2 < q_j and
// a_i mod q_j is a_i or a_i + q_j.  Horner in double from the top digit then
// rounds once per step.
namespace {
constexpr int kMaxGarner = 16;
struct Garner {
  int nl = 0;
  u64 q[kMaxGarner];
  u64 inv[kMaxGarner][kMaxGarner], inv_sh[kMaxGarner][kMaxGarner];  // q_i^-1 mod q_j (i < j), Shoup companion
};
// Shoup companion of a constant w < q: floor(w 2^64 / q)
u64 shoup(u64 w, u64 q) { return (u64)(((u128)w << 64) / q); }
// a * w mod q for a < 2^64 and w < q < 2^63, with wsh = shoup(w, q)
inline u64 mul_shoup(u64 a, u64 w, u64 wsh, u64 q) {
  const u64 hq = (u64)(((u128)a * wsh) >> 64);
  const u64 r = a * w - hq * q;  // in [0, 2q)
  return r >= q ? r - q : r;
}
Garner make_garner(const fa_ctx* c, int nl) {
  Garner g;
  g.nl = nl;
  for (int i = 0; i < nl; ++i) g.q[i] = c->primes[i];
  for (int i = 0; i < nl; ++i)
    for (int j = i + 1; j < nl; ++j) {
      g.inv[i][j] = invmod(g.q[i] % g.q[j], g.q[j]);
      g.inv_sh[i][j] = shoup(g.inv[i][j], g.q[j]);
    }
  return g;
}
// the centred integer with residues res[t * stride] (t < nl), as a double;
// NL > 0 fixes the prime count at compile time (the loops unroll), NL = 0 reads it from g
template <int NL = 0>
inline double garner_to_double(const Garner& g, const uint64_t* res, size_t stride) {
  const int nl = NL > 0 ? NL : g.nl;
  int64_t a[kMaxGarner];
  for (int j = 0; j < nl; ++j) {
    const u64 qj = g.q[j];
    u64 v = res[(size_t)j * stride];
    if (v >= qj) v %= qj;  // fa_decrypt hands out canonical residues; others are reduced here
    for (int i = 0; i < j; ++i) {
      const u64 ai = a[i] < 0 ? (u64)(a[i] + (int64_t)qj) : (u64)a[i];
      v = v >= ai ? v - ai : v + qj - ai;
      v = mul_shoup(v, g.inv[i][j], g.inv_sh[i][j], qj);
    }
    a[j] = v > (qj - 1) / 2 ? (int64_t)v - (int64_t)qj : (int64_t)v;
  }
  double x = (double)a[nl - 1];
  for (int i = nl - 2; i >= 0; --i) x = (double)a[i] + (double)g.q[i] * x;
  return x;
}

// A_t = sum_k x_k e^{+2 pi i k t / n} over split real / imaginary arrays that
// already hold x in bit-reversed order (x_k at index brev(k)); n a power of
// two, radix-2 stages in place, A_t at index t.  twr / twi hold the stages'
// twiddles one after the other: for the stage of span len (len = 4, 8, ...,
// n), e^{+2 pi i j / len} for j < len/2 at offset len/2 - 2 (see dec_tables);
// the span-2 stage needs none.
void fft_pos_brev_in(double* re, double* im, int n, const double* twr, const double* twi) {
  for (int s0 = 0; s0 < n; s0 += 2) {
    const double ur = re[s0], ui = im[s0], vr = re[s0 + 1], vi = im[s0 + 1];
    re[s0] = ur + vr;
    im[s0] = ui + vi;
    re[s0 + 1] = ur - vr;
    im[s0 + 1] = ui - vi;
  }
  for (int len = 4; len <= n; len <<= 1) {
    const int h = len / 2;
    const double* wr = twr + (h - 2);  // stage offsets: 0, 2, 6, 14, ... = h - 2
    const double* wi = twi + (h - 2);
    for (int s0 = 0; s0 < n; s0 += len) {
      double* ar = re + s0;
      double* ai = im + s0;
      double* br = re + s0 + h;
      double* bi = im + s0 + h;
      for (int j = 0; j < h; ++j) {
        const double vr = br[j] * wr[j] - bi[j] * wi[j];
        const double vi = br[j] * wi[j] + bi[j] * wr[j];
        const double ur = ar[j], ui = ai[j];
        ar[j] = ur + vr;
        ai[j] = ui + vi;
        br[j] = ur - vr;
        bi[j] = ui - vi;
      }
    }
  }
}

// decode tables of ring degree n: e^{+2 pi i k / (n/2)} for k < n/4 (split),
// and the slot -> transform index map t_j = (5^j mod 2n - 1) / 4
struct DecTables {
  std::vector<double> twr, twi;  // per-stage twiddles of fft_pos_brev_in for length n/2
  std::vector<uint32_t> brev;    // bit reversal over log2(n/2) bits
  std::vector<uint32_t> slot_t;
};
const DecTables& dec_tables(int n) {
  static std::mutex mu;
  static std::map<int, std::unique_ptr<DecTables>> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto& slot = cache[n];
  if (!slot) {
    auto t = std::make_unique<DecTables>();
    const int h = n / 2;
    // stage of span len: e^{+2 pi i j / len}, j < len/2, at offset len/2 - 2;
    // taken from the length-h table (index j h / len) so every stage uses the
    // same rounded values as a single table would
    std::vector<double> cr(h / 2), ci(h / 2);
    for (int k = 0; k < h / 2; ++k) {
      const double ang = 2.0 * M_PI * (double)k / (double)h;
      cr[k] = std::cos(ang);
      ci[k] = std::sin(ang);
    }
    t->twr.assign(h > 2 ? h - 2 : 0, 0.0);
    t->twi.assign(h > 2 ? h - 2 : 0, 0.0);
    for (int len = 4; len <= h; len <<= 1)
      for (int j = 0; j < len / 2; ++j) {
        t->twr[len / 2 - 2 + j] = cr[(size_t)j * (h / len)];
        t->twi[len / 2 - 2 + j] = ci[(size_t)j * (h / len)];
      }
    int bits = 0;
    while ((1 << bits) < h) ++bits;
    t->brev.resize(h);
    for (int k = 0; k < h; ++k) t->brev[k] = bitrev((uint32_t)k, bits);
    const std::vector<u64>& e = fft_tables(n).e;
    t->slot_t.resize(h);
    for (int j = 0; j < h; ++j) t->slot_t[j] = (uint32_t)((e[j] - 1) / 4);
    slot = std::move(t);
  }
  return *slot;
}
}  // namespace

extern "C" {

int fa_decode(const fa_ctx* c, const uint64_t* res, int log_scale, double* out, int n_slots) {
  if (!c || !res || !out) return fail(FA_E_INVAL, "fa_decode: null argument");
  if (n_slots < 0 || n_slots > c->n / 2) return fail(FA_E_SHAPE, "fa_decode: n_slots %d > N/2", n_slots);
  const int n = c->n, h = n / 2;
  // The decrypted value m' = m + e is far below the product of the first few
  // primes: |m'| < 2^(log_scale + 20) for slot values below 2^12 in magnitude,
  // so the centred CRT over just enough primes already returns it exactly.
  int nl = 0;
  double bits = 0.0;
  while (nl < c->L && bits < log_scale + 22.0) bits += std::log2((double)c->primes[nl++]);
  if (nl > kMaxGarner) return fail(FA_E_SHAPE, "fa_decode: %d primes needed (at most %d)", nl, kMaxGarner);
  const Garner g = make_garner(c, nl);
  // Every slot exponent e_j = 5^j mod 2N is 1 mod 4, and X^(N/2) = i at such a
  // root: m(zeta^e) = w(zeta^e) with w_k = m_k + i m_{k+N/2} (k < N/2).  With
  // e = 4t + 1, w(zeta^e) = sum_k (w_k zeta^k) e^{+2 pi i k t / (N/2)}, one
  // transform of length N/2.
  const FftTables& tb = fft_tables(n);
  const DecTables& dt = dec_tables(n);
  std::vector<double> re(h), im(h);
  // One host thread: a client decodes its result blocks several at a time, and
  // threads started inside each decode made those concurrent calls several
  // times slower than serial ones.
  auto crt = [&](auto nlc) {
    constexpr int NL = decltype(nlc)::value;
    for (int k = 0; k < h; ++k) {
      const double lo = garner_to_double<NL>(g, res + k, (size_t)n);
      const double hi = garner_to_double<NL>(g, res + k + h, (size_t)n);
      const double cr = tb.twist[k].real(), ci = tb.twist[k].imag();
      const uint32_t kb = dt.brev[k];
      re[kb] = lo * cr - hi * ci;
      im[kb] = lo * ci + hi * cr;
    }
  };
  switch (nl) {
    case 1: crt(std::integral_constant<int, 1>{}); break;
    case 2: crt(std::integral_constant<int, 2>{}); break;
    case 3: crt(std::integral_constant<int, 3>{}); break;
    case 4: crt(std::integral_constant<int, 4>{}); break;
    default: crt(std::integral_constant<int, 0>{}); break;
  }
  fft_pos_brev_in(re.data(), im.data(), h, dt.twr.data(), dt.twi.data());
  const double inv_scale = std::ldexp(1.0, -log_scale);
  for (int j = 0; j < n_slots; ++j) out[j] = re[dt.slot_t[j]] * inv_scale;
  return FA_OK;
}

// Plaintexts from integer coefficients: residues then forward NTT.
static int upload_int_pts(fa_ctx* c, const int64_t* coeffs, int n_pts, double* pts, hipStream_t s) {
  const size_t n = c->n, L = c->L;
  const int chunk = 64;
  int64_t* dm = nullptr;
  int rc = dev_alloc(&dm, (size_t)chunk * n);
  if (rc) return rc;
  for (int p0 = 0; p0 < n_pts; p0 += chunk) {
    const int m = std::min(chunk, n_pts - p0);
    HIPCHK(hipMemcpyAsync(dm, coeffs + (size_t)p0 * n, (size_t)m * n * 8, hipMemcpyHostToDevice, s));
    double* dst = pts + (size_t)p0 * L * n;
    fa::int_to_res(c, dm, m, (int)L, dst, s);
    fa::ntt_fwd_strided(c, dst, n, m * (int)L, (int)L, 0, s);
    if ((rc = check_launch("encode"))) break;
    HIPCHK(hipStreamSynchronize(s));
  }
  (void)hipFree(dm);
  return rc;
}

int fa_encode_db_block_int(fa_ctx* c, const int64_t* coeffs, int n_pts, int32_t log_scale, fa_buf* pts,
                           void* stream) {
  if (!c || !coeffs) return fail(FA_E_INVAL, "fa_encode_db_block_int: null argument");
  if (n_pts < 1) return fail(FA_E_SHAPE, "fa_encode_db_block_int: n_pts must be positive");
  if (log_scale < 0 || log_scale > 1000) return fail(FA_E_INVAL, "fa_encode_db_block_int: log_scale out of range");
  int rc = out_check(c, pts, "fa_encode_db_block_int", "pts", n_pts, 1);
  if (rc) return rc;
  for (size_t i = 0; i < (size_t)n_pts * c->n; ++i)
    if (coeffs[i] > (INT64_C(1) << 62) || coeffs[i] < -(INT64_C(1) << 62))
      return fail(FA_E_INVAL, "fa_encode_db_block_int: coefficient out of range");
  rc = upload_int_pts(c, coeffs, n_pts, (double*)pts->dev, (hipStream_t)stream);
  if (!rc) out_set(c, pts, 1, n_pts, log_scale);
  return rc;
}

int fa_encode_db_block(fa_ctx* c, const float* rows, int n_rows, int dim, int d, int layout, int baby_step,
                       fa_buf* pts_b, void* stream) {
  if (!c || !rows || !pts_b || !pts_b->dev) return fail(FA_E_INVAL, "fa_encode_db_block: null argument");
  const int S = c->n / 2;
  if (d < 1 || (d & (d - 1)) || d > S) return fail(FA_E_SHAPE, "d=%d must be a power of two <= N/2", d);
  if (dim < 1 || dim > d) return fail(FA_E_SHAPE, "dim=%d must be in [1, d=%d]", dim, d);
  if (n_rows < 1) return fail(FA_E_SHAPE, "n_rows must be positive");
  const std::vector<u64>& e = slot_exps(c->n);
  const double scale = std::ldexp(1.0, c->log_scale);
  std::vector<int64_t> coeffs;
  int n_pts;
  if (layout == FA_LAYOUT_DIAG) {
    if (n_rows > S) return fail(FA_E_SHAPE, "a diagonal block holds at most N/2=%d rows, got %d", S, n_rows);
    if (baby_step < 1 || d % baby_step) return fail(FA_E_INVAL, "baby_step %d must divide d=%d", baby_step, d);
    n_pts = d;
    if (int rc = out_check(c, pts_b, "fa_encode_db_block", "pts", n_pts, 1)) return rc;
    coeffs.assign((size_t)n_pts * c->n, 0);
    parallel_for(n_pts, [&](int j) {
      const int g = j / baby_step;
      const int shift = g * baby_step;  // pre-rotation right by gB
      std::vector<double> v(S, 0.0);
      for (int i = 0; i < n_rows; ++i) {
        const int col = (i + j) % d;
        const double x = col < dim ? (double)rows[(size_t)i * dim + col] : 0.0;
        v[(i + shift) % S] = x;
      }
      encode_one(c->n, e, v.data(), S, scale, coeffs.data() + (size_t)j * c->n);
    });
  } else if (layout == FA_LAYOUT_ROW) {
    const int per = S / d;
    n_pts = (n_rows + per - 1) / per;
    if (int rc = out_check(c, pts_b, "fa_encode_db_block", "pts", n_pts, 1)) return rc;
    coeffs.assign((size_t)n_pts * c->n, 0);
    parallel_for(n_pts, [&](int w) {
      std::vector<double> v(S, 0.0);
      for (int t = 0; t < per; ++t) {
        const int row = w * per + t;
        if (row >= n_rows) break;
        for (int u = 0; u < dim; ++u) v[(size_t)t * d + u] = rows[(size_t)row * dim + u];
      }
      encode_one(c->n, e, v.data(), S, scale, coeffs.data() + (size_t)w * c->n);
    });
  } else {
    return fail(FA_E_INVAL, "unknown layout %d", layout);
  }
  const int rc = upload_int_pts(c, coeffs.data(), n_pts, (double*)pts_b->dev, (hipStream_t)stream);
  if (!rc) out_set(c, pts_b, 1, n_pts, c->log_scale);
  return rc;
}

int fa_encode_projection(fa_ctx* c, const float* W, int d_in, int r, int baby_step, fa_buf* pts, void* stream) {
  if (!c || !W || !pts || !pts->dev) return fail(FA_E_INVAL, "fa_encode_projection: null argument");
  const int S = c->n / 2;
  if (r < 1 || (r & (r - 1)) || d_in < r || d_in % r || (d_in & (d_in - 1)) || d_in > S)
    return fail(FA_E_SHAPE, "d_in=%d, r=%d: powers of two with r | d_in and d_in <= N/2", d_in, r);
  if (baby_step < 1 || r % baby_step) return fail(FA_E_INVAL, "baby_step %d must divide r=%d", baby_step, r);
  if (int rc = out_check(c, pts, "fa_encode_projection", "pts", r, 1)) return rc;
  const std::vector<u64>& e = slot_exps(c->n);
  const double scale = std::ldexp(1.0, c->log_scale);
  std::vector<int64_t> coeffs((size_t)r * c->n);
  parallel_for(r, [&](int j) {
    const int shift = (j / baby_step) * baby_step;  // pre-rotation right by gB
    std::vector<double> v(S);
    for (int s = 0; s < S; ++s)
      v[(s + shift) % S] = (double)W[(size_t)((s + j) % d_in) * r + (s % r)];
    encode_one(c->n, e, v.data(), S, scale, coeffs.data() + (size_t)j * c->n);
  });
  const int rc = upload_int_pts(c, coeffs.data(), r, (double*)pts->dev, (hipStream_t)stream);
  if (!rc) out_set(c, pts, 1, r, c->log_scale);
  return rc;
}

// ---------------------------------------------------------------------------
// workspace carving
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {
constexpr int kRotBatch = 16;  // most rotations key-switched per launch group

// Rotations per launch group of one query's baby steps (1..kRotBatch;
// FA_ROT_BATCH overrides it): 8 with several key-switch digits (measured
// 0.05 ms faster than 16 on the 12-prime rerank level), 16 with one digit (the
// fused special-prime kernel's launches stay large).  The environment is read
// once, by a thread-safe static initialiser.
int rot_batch(const fa_ctx* c) {
  static const int v = [] {
    const char* e = getenv("FA_ROT_BATCH");
    const int r = e ? atoi(e) : 0;
    return (r < 1 || r > kRotBatch) ? 0 : r;
  }();
  return v ? v : (c->dnum > 1 ? 8 : kRotBatch);
}

struct Arena {
  char* base;
  size_t cap, used;
  double* take(size_t words) {
    const size_t bytes = (words * 8 + 255) & ~(size_t)255;
    if (used + bytes > cap) return nullptr;
    double* p = (double*)(base + used);
    used += bytes;
    return p;
  }
};
size_t rup(size_t words) { return (words * 8 + 255) & ~(size_t)255; }

// workspace of a batch of `nb` full rotations (own ModUp each)
size_t rotate_ws(const fa_ctx* c, int nb) {
  const size_t n = c->n;
  return rup((size_t)nb * c->L * n) + rup((size_t)nb * c->dnum * c->np * n) + rup((size_t)nb * 2 * c->np * n) +
         rup((size_t)nb * 2 * c->L * n);
}

// Lanes (the caller's stream plus auxiliary streams) that independent
// key-switch batches of one scoring call are spread over; FA_STREAMS tunes it.
int lanes_wanted() {
  static const int v = [] {
    const char* e = getenv("FA_STREAMS");
    const int r = e ? atoi(e) : 2;
    return r < 1 ? 1 : (r > FA_MAXAUX + 1 ? FA_MAXAUX + 1 : r);
  }();
  return v;
}

// workspace of the baby rotations (qrot itself is separate)
size_t baby_ws(const fa_ctx* c, int B) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t rb = std::max(1, std::min(rot_batch(c), B - 1));
  const size_t lanes = lanes_wanted();
  return rup(L * n) + rup(dn * np * n) + lanes * rup(rb * 2 * np * n) + lanes * rup(rb * 2 * L * n);
}
// baby steps per launch group of a query batch: 64 rotations per group from
// four queries on (16, 32, 64, 128 measured; 64 keeps the workspace near
// 2 GB per lane), kRotBatch for fewer queries so that one or two still fill
// both lanes
int batch_steps(int nq) {
  nq = std::max(1, nq);
  return std::max(1, (nq >= 4 ? 64 : kRotBatch) / nq);
}
// workspace of the baby rotations of n_q queries prepared together (the
// rotated queries themselves are separate): one query's row-passed c1,
// every query's extended digits, and per lane the key-switch products and
// conversions of one launch group (batch_steps(n_q) x n_q rotations)
size_t baby_batch_ws(const fa_ctx* c, int nq, int B) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t items = (size_t)std::max(1, std::min(batch_steps(nq), B - 1)) * nq;
  const size_t lanes = lanes_wanted();
  return rup(L * n) + (size_t)nq * rup(dn * np * n) + lanes * rup(items * 2 * np * n) + lanes * rup(items * 2 * L * n);
}
// blocks whose giant steps are processed together (a query batch's blocks
// share chunks; 16 measured faster than 8 for batches, 32 no faster than 16)
constexpr int kGiantChunk = 16;
// scratch of the giant steps of one query (accumulators not included)
size_t giant_scratch_ws(const fa_ctx* c, int nb, int d, int B) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t G = d / B;
  if (G <= 1) return 0;
  const size_t lanes = lanes_wanted();
  const size_t cb = std::min(nb, kGiantChunk);
  return lanes * rup(std::max(cb, G - 1) * L * n) + rup(cb * (G - 1) * dn * np * n) + rup(cb * 2 * np * n) +
         rup(cb * 2 * L * n);
}
// workspace of the multiply-accumulate and the giant steps of nq queries
// (the giant steps of all nq queries run together, over nq * nb blocks)
size_t giant_ws(const fa_ctx* c, int nb, int d, int B, int nq = 1) {
  const size_t G = d / B;
  return rup((size_t)nq * nb * G * 2 * c->L * c->n) + giant_scratch_ws(c, nq * nb, d, B);
}
size_t qrot_words(const fa_ctx* c, int B) { return (size_t)(B - 1) * 2 * c->L * c->n + 1; }
size_t score_ws(const fa_ctx* c, int nb, int d, int B) {
  return baby_ws(c, B) + rup(qrot_words(c, B)) + giant_ws(c, nb, d, B);
}
}  // namespace

// Extended digits (NTT form) of the c1 of `batch` ciphertexts cts + b * ct_stride.
// y (per item [L][N]) receives c1 after the row pass of its inverse transform
// (scratch); ext receives every converted limb (pass_b false: the first
// forward pass only).  The ciphertexts are only read.
static void modup(fa_ctx* c, const double* cts, size_t ct_stride, int batch, double* y, size_t y_stride,
                  double* ext, size_t ext_stride, hipStream_t s, bool pass_b = true) {
  const size_t n = c->n, L = c->L;
  {
    // the row pass of the inverse transform; the fused ModUp kernel finishes it
    fa::LimbBatch inv(c, s, false, true);
    for (int b = 0; b < batch; ++b)
      for (size_t t = 0; t < L; ++t)
        inv.add(y + (size_t)b * y_stride + t * n, (int)t, cts + (size_t)b * ct_stride + (L + t) * n);
  }
  std::vector<fa::MuItem> it(batch);
  for (int b = 0; b < batch; ++b) it[b] = {y + (size_t)b * y_stride, ext + (size_t)b * ext_stride};
  fa::modup_fused(c, it.data(), batch, s, pass_b);
}

// ModDown of `count` polynomials u_i = u + i * np * N over Q u P (NTT form):
// out_i = bases_i[pi_gal_i] + (u_i,Q - Conv_{P->Q}(u_i,P)) * P^-1.  The special-
// prime limbs of u are overwritten (the row pass of their inverse transform;
// inv_b_done: already done by the caller); conv is scratch.  With pass_b
// false only the special-prime inverse and the conversion's first pass run
// (bases, outs and gals unused): moddown_ks finishes.
static void moddown_polys(fa_ctx* c, double* u, int count, double* conv, const double* const* bases,
                          double* const* outs, const uint32_t* gals, hipStream_t s, bool pass_b = true,
                          bool inv_b_done = false) {
  const size_t n = c->n, L = c->L, np = c->np;
  if (!inv_b_done) {
    // the row pass of the inverse transform, in place; the fused ModDown
    // kernel finishes it
    fa::LimbBatch inv(c, s, false, true);
    for (int i = 0; i < count; ++i)
      for (int k = 0; k < c->K; ++k) inv.add(u + (size_t)i * np * n + (L + k) * n, (int)L + k);
  }
  std::vector<fa::MdItem> it(count);
  for (int i = 0; i < count; ++i) {
    double* ui = u + (size_t)i * np * n;
    it[i] = {ui + L * n, conv + (size_t)i * L * n, ui, pass_b ? bases[i] : nullptr, pass_b ? outs[i] : nullptr,
             pass_b ? gals[i] : 1u};
  }
  fa::moddown_fused(c, it.data(), count, s, pass_b);
}

// Key switch and ModDown of `count` rotations: outs[j] = (c0s[j][pi] + ModDown(u_0),
// ModDown(u_1)) with u = sum_i sigma(ext_i) key_i.  The special-prime part of u
// goes through u (per rotation [2][np][N]); the ciphertext-prime part is formed
// inside the finishing kernel.  conv: per rotation [2][L][N] scratch.
static void ks_moddown(fa_ctx* c, const fa::KsItem* ks, int count, const double* const* c0s, double* const* outs,
                       double* u, double* conv, hipStream_t s, const double* const* b1s = nullptr, int nq = 1) {
  const size_t n = c->n, L = c->L;
  if (c->dnum == 1) {
    // one digit: the special-prime sum and the first inverse pass in one
    // kernel (measured faster at 2 and 3 primes; with more digits the fused
    // kernel's longer load phase made it slower)
    fa::ks_inv_b(c, ks, count, s, nq);
    moddown_polys(c, u, 2 * count, conv, nullptr, nullptr, nullptr, s, false, true);
  } else {
    fa::ks_inner(c, ks, count, false, s, c->L, nq);
    moddown_polys(c, u, 2 * count, conv, nullptr, nullptr, nullptr, s, false);
  }
  std::vector<fa::MdKsItem> it(count);
  for (int j = 0; j < count; ++j)
    it[j] = {conv + (size_t)2 * j * L * n, ks[j].ext, ks[j].c1, ks[j].key, c0s[j], b1s ? b1s[j] : nullptr, outs[j],
             ks[j].gal};
  fa::moddown_ks(c, it.data(), count, s, nq);
}

// Auxiliary streams for `lanes` lanes (lane 0 is the caller's stream).
static int ensure_lanes(fa_ctx* c, int lanes) {
  if (!c->fork_ev) HIPCHK(hipEventCreateWithFlags(&c->fork_ev, hipEventDisableTiming));
  while (c->n_aux < lanes - 1) {
    const int i = c->n_aux;
    HIPCHK(hipStreamCreateWithFlags(&c->aux[i], hipStreamNonBlocking));
    HIPCHK(hipEventCreateWithFlags(&c->join_ev[i], hipEventDisableTiming));
    c->n_aux++;
  }
  return FA_OK;
}
static hipStream_t lane_stream(fa_ctx* c, hipStream_t s, int lane) { return lane == 0 ? s : c->aux[lane - 1]; }
static int fork_lanes(fa_ctx* c, hipStream_t s, int lanes) {
  if (lanes < 2) return FA_OK;
  HIPCHK(hipEventRecord(c->fork_ev, s));
  for (int i = 0; i < lanes - 1; ++i) HIPCHK(hipStreamWaitEvent(c->aux[i], c->fork_ev, 0));
  return FA_OK;
}
static int join_lanes(fa_ctx* c, hipStream_t s, int lanes) {
  for (int i = 0; i < lanes - 1; ++i) {
    HIPCHK(hipEventRecord(c->join_ev[i], c->aux[i]));
    HIPCHK(hipStreamWaitEvent(s, c->join_ev[i], 0));
  }
  return FA_OK;
}

// Hoisted rotations of one ciphertext q by steps[0..m-1]: one decomposition of
// c1 shared by all, each rotation with its own key switch and ModDown.
// ext must already hold the extended digits of q.c1 (NTT form).  Batches of
// rotations go round-robin to `lanes` lanes, lane l using scratch u/conv +
// l * (per-lane size).
static int rotations_from_ext(fa_ctx* c, const double* q, const double* ext, const int* steps, int m,
                              double* const* outs, double* u, double* conv, hipStream_t s, int lanes, int rbmax,
                              size_t u_lane, size_t c_lane) {
  const size_t n = c->n, L = c->L, np = c->np;
  for (int r0 = 0, j0 = 0; r0 < m; r0 += rbmax, ++j0) {
    const int rb = std::min(rbmax, m - r0);
    const int lane = j0 % lanes;
    hipStream_t ls = lane_stream(c, s, lane);
    double* ul = u + lane * u_lane;
    double* cl = conv + lane * c_lane;
    fa::KsItem ks[kRotBatch];
    const double* c0s[kRotBatch];
    for (int j = 0; j < rb; ++j) {
      auto it = c->keys.find(steps[r0 + j]);
      if (it == c->keys.end()) return fail(FA_E_NOKEY, "no rotation key for step %d", steps[r0 + j]);
      const uint32_t gal = galois(c->n, steps[r0 + j]);
      ks[j] = {ext, q + L * n, it->second, ul + (size_t)j * 2 * np * n, nullptr, gal};
      c0s[j] = q;
    }
    ks_moddown(c, ks, rb, c0s, outs + r0, ul, cl, ls);
  }
  return check_launch("rotation");
}

// Full rotation of `nb` ciphertexts by the same step: outs[b] = Rotate(cts[b], step).
static int rotate_batch(fa_ctx* c, const double* cts, int nb, int step, double* outs, Arena& ar, hipStream_t s) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  auto it = c->keys.find(step);
  if (it == c->keys.end()) return fail(FA_E_NOKEY, "no rotation key for step %d", step);
  const size_t mark = ar.used;
  double* y = ar.take((size_t)nb * L * n);
  double* ext = ar.take((size_t)nb * dn * np * n);
  double* u = ar.take((size_t)nb * 2 * np * n);
  double* conv = ar.take((size_t)nb * 2 * L * n);
  if (!y || !ext || !u || !conv) return fail(FA_E_NOMEM, "workspace too small for rotation");
  const size_t ctw = 2 * L * n;
  modup(c, cts, ctw, nb, y, L * n, ext, dn * np * n, s);
  std::vector<fa::KsItem> ks(nb);
  std::vector<const double*> c0s(nb);
  std::vector<double*> douts(nb);
  const uint32_t gal = galois(c->n, step);
  for (int b = 0; b < nb; ++b) {
    const double* ct = cts + (size_t)b * ctw;
    ks[b] = {ext + (size_t)b * dn * np * n, ct + L * n, it->second, u + (size_t)b * 2 * np * n, nullptr, gal};
    c0s[b] = ct;
    douts[b] = outs + (size_t)b * ctw;
  }
  ks_moddown(c, ks.data(), nb, c0s.data(), douts.data(), u, conv, s);
  ar.used = mark;
  return check_launch("rotate_batch");
}

// Relinearisation of `count` three-component ciphertexts d [count][3][L][N]:
// out[j] = (d0 + ModDown(u0), d1 + ModDown(u1)) with (u0, u1) the key-switch
// inner product of d2 with the relinearisation key (no automorphism), in
// batches of up to kRotBatch; out [count][2][L][N].
static size_t relin_ws(const fa_ctx* c) { return rotate_ws(c, kRotBatch); }
static int relin_batch(fa_ctx* c, const double* d, int count, double* out, Arena& ar, hipStream_t s) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  if (!c->d_rlk) return fail(FA_E_NOKEY, "no relinearisation key (fa_keygen_relin)");
  const size_t mark = ar.used;
  const int nbm = std::min(count, kRotBatch);
  double* y = ar.take((size_t)nbm * L * n);
  double* ext = ar.take((size_t)nbm * dn * np * n);
  double* u = ar.take((size_t)nbm * 2 * np * n);
  double* conv = ar.take((size_t)nbm * 2 * L * n);
  if (!y || !ext || !u || !conv) return fail(FA_E_NOMEM, "workspace too small for relinearisation");
  const size_t d3 = 3 * L * n, ctw = 2 * L * n;
  for (int j0 = 0; j0 < count; j0 += nbm) {
    const int nb = std::min(nbm, count - j0);
    // ModUp of the s^2 components: "ciphertexts" at d + 2LN with stride 3LN read as (., c1)
    modup(c, d + (size_t)j0 * d3 + L * n, d3, nb, y, L * n, ext, dn * np * n, s);
    std::vector<fa::KsItem> ks(nb);
    std::vector<const double*> c0s(nb), b1s(nb);
    std::vector<double*> outs(nb);
    for (int j = 0; j < nb; ++j) {
      const double* dj = d + (size_t)(j0 + j) * d3;
      ks[j] = {ext + (size_t)j * dn * np * n, dj + 2 * L * n, c->d_rlk, u + (size_t)j * 2 * np * n, nullptr, 1u};
      c0s[j] = dj;
      b1s[j] = dj + L * n;
      outs[j] = out + (size_t)(j0 + j) * ctw;
    }
    ks_moddown(c, ks.data(), nb, c0s.data(), outs.data(), u, conv, s, b1s.data());
  }
  ar.used = mark;
  return check_launch("relinearise");
}

// Baby rotations qrot[b-1] = Rotate(q, b), b = 1..B-1: one shared decomposition
// of q.c1, rotation batches spread over lanes.
static int baby_phase(fa_ctx* c, const double* q, int B, double* qrot, Arena& ar, hipStream_t s) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t ctw = 2 * L * n;
  if (B < 2) return FA_OK;
  for (int b = 1; b < B; ++b)
    if (!c->keys.count(b)) return fail(FA_E_NOKEY, "no rotation key for baby step %d", b);
  const int rb = std::max(1, std::min(rot_batch(c), B - 1));
  const int lanes = lanes_wanted();
  const size_t mark = ar.used;
  double* y = ar.take(L * n);
  double* ext = ar.take(dn * np * n);
  double* u = ar.take((size_t)lanes * (rup((size_t)rb * 2 * np * n) / 8));
  double* conv = ar.take((size_t)lanes * (rup((size_t)rb * 2 * L * n) / 8));
  if (!y || !ext || !u || !conv) return fail(FA_E_NOMEM, "workspace too small for the baby rotations");
  int rc = ensure_lanes(c, lanes);
  if (rc) return rc;
  modup(c, q, ctw, 1, y, L * n, ext, dn * np * n, s);
  std::vector<int> steps(B - 1);
  std::vector<double*> outs(B - 1);
  for (int b = 1; b < B; ++b) {
    steps[b - 1] = b;
    outs[b - 1] = qrot + (size_t)(b - 1) * ctw;
  }
  const int nbatch = (B - 1 + rb - 1) / rb;
  const int bl = std::min(lanes, nbatch);
  if ((rc = fork_lanes(c, s, bl))) return rc;
  rc = rotations_from_ext(c, q, ext, steps.data(), B - 1, outs.data(), u, conv, s, bl, rb,
                          rup((size_t)rb * 2 * np * n) / 8, rup((size_t)rb * 2 * L * n) / 8);
  if (rc) return rc;
  if ((rc = join_lanes(c, s, bl))) return rc;
  ar.used = mark;
  return FA_OK;
}

// Baby rotations of n_q queries, qrots[j][b-1] = Rotate(qs[j], b), b = 1..B-1:
// one ModUp per query, then launch groups of a few steps each holding the key
// switches of every query for those steps (step-major), so that a step's key,
// read from HBM for the first query, is found in the caches by the others.
// Each rotation runs the same kernels on the same inputs as in baby_phase, so
// the results are identical to preparing the queries one by one.
static int baby_phase_batch(fa_ctx* c, const double* const* qs, int nq, int B, double* const* qrots, Arena& ar,
                            hipStream_t s) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t ctw = 2 * L * n, ext_w = dn * np * n;
  if (B < 2) return FA_OK;
  for (int b = 1; b < B; ++b)
    if (!c->keys.count(b)) return fail(FA_E_NOKEY, "no rotation key for baby step %d", b);
  const int rbq = std::max(1, std::min(batch_steps(nq), B - 1));
  const size_t items = (size_t)rbq * nq;
  const int lanes = lanes_wanted();
  const size_t u_lane = rup(items * 2 * np * n) / 8, c_lane = rup(items * 2 * L * n) / 8;
  const size_t mark = ar.used;
  double* y = ar.take(L * n);
  double* ext = ar.take((size_t)nq * (rup(ext_w) / 8));
  double* u = ar.take((size_t)lanes * u_lane);
  double* conv = ar.take((size_t)lanes * c_lane);
  if (!y || !ext || !u || !conv) return fail(FA_E_NOMEM, "workspace too small for the baby rotations");
  int rc = ensure_lanes(c, lanes);
  if (rc) return rc;
  for (int j = 0; j < nq; ++j) modup(c, qs[j], ctw, 1, y, L * n, ext + (size_t)j * (rup(ext_w) / 8), ext_w, s);
  const int ngroup = (B - 1 + rbq - 1) / rbq;
  const int bl = std::min(lanes, ngroup);
  if ((rc = fork_lanes(c, s, bl))) return rc;
  std::vector<fa::KsItem> ks(items);
  std::vector<const double*> c0s(items);
  std::vector<double*> outs(items);
  for (int r0 = 1, j0 = 0; r0 < B; r0 += rbq, ++j0) {
    const int lane = j0 % bl;
    hipStream_t ls = lane_stream(c, s, lane);
    double* ul = u + lane * u_lane;
    double* cl = conv + lane * c_lane;
    int m = 0;
    for (int b = r0; b < std::min(B, r0 + rbq); ++b) {
      const double* key = c->keys[b];
      const uint32_t gal = galois(c->n, b);
      for (int j = 0; j < nq; ++j, ++m) {
        ks[m] = {ext + (size_t)j * (rup(ext_w) / 8), qs[j] + L * n, key, ul + (size_t)m * 2 * np * n, nullptr, gal};
        c0s[m] = qs[j];
        outs[m] = qrots[j] + (size_t)(b - 1) * ctw;
      }
    }
    ks_moddown(c, ks.data(), m, c0s.data(), outs.data(), ul, cl, ls, nullptr, nq);
  }
  if ((rc = join_lanes(c, s, bl))) return rc;
  ar.used = mark;
  return check_launch("prepare_batch");
}

// Giant steps of one query from its accumulators acc ([nb][G][2][L][N]):
// out[blk] = acc_0 + Rotate(acc_g, gB) summed over g >= 1 in Q u P with one
// ModDown per block; sigma(acc_g.c0) rides in the key-switch sum multiplied by
// P.  The first pass of every giant's ModUp runs on the lanes (round-robin over
// g); one fused kernel then finishes the transforms and forms the key-switch
// sums.  Scratch comes from ar (giant_ws minus the accumulators).
static int giant_phase(fa_ctx* c, const double* acc, int nb, int G, int B, double* const* outs, Arena& ar,
                       hipStream_t s) {
  const size_t n = c->n, L = c->L, np = c->np, dn = c->dnum;
  const size_t ctw = 2 * L * n;
  const size_t astride = (size_t)G * ctw;
  if (G == 1) {
    for (int blk = 0; blk < nb; ++blk)
      HIPCHK(hipMemcpyAsync(outs[blk], acc + (size_t)blk * ctw, ctw * 8, hipMemcpyDeviceToDevice, s));
    return FA_OK;
  }
  const int lanes = lanes_wanted();
  const int cbm = std::min(nb, kGiantChunk);
  const size_t gy_l = rup((size_t)std::max(cbm, G - 1) * L * n) / 8;
  const size_t ext_w = dn * np * n;
  const size_t mark = ar.used;
  double* gy = ar.take(lanes * gy_l);
  double* gext = ar.take((size_t)cbm * (G - 1) * ext_w);
  double* usum = ar.take((size_t)cbm * 2 * np * n);
  double* gconv = ar.take((size_t)cbm * 2 * L * n);
  if (!gy || !gext || !usum || !gconv) return fail(FA_E_NOMEM, "workspace too small for the giant steps");
  int rc = ensure_lanes(c, lanes);
  if (rc) return rc;
  std::vector<const double*> keys(G - 1);
  std::vector<uint32_t> ggal(G - 1);
  for (int g = 1; g < G; ++g) {
    keys[g - 1] = c->keys[g * B];
    ggal[g - 1] = galois(c->n, g * B);
  }
  for (int b0 = 0; b0 < nb; b0 += cbm) {
    const int cb = std::min(cbm, nb - b0);
    const double* accb = acc + (size_t)b0 * astride;
    // the ModUps of the giant accumulators in as few launch groups as the
    // lanes allow: one per block (over its G-1 giants) when there are fewer
    // blocks than giants, else one per giant (over the blocks)
    const bool per_block = cb < G - 1;
    const int gl = std::min(lanes, per_block ? cb : G - 1);
    if ((rc = fork_lanes(c, s, gl))) return rc;
    if (per_block) {
      for (int blk = 0; blk < cb; ++blk) {
        const int lane = blk % gl;
        modup(c, accb + (size_t)blk * astride + ctw, ctw, G - 1, gy + lane * gy_l, L * n,
              gext + (size_t)blk * (G - 1) * ext_w, ext_w, lane_stream(c, s, lane), false);
      }
    } else {
      for (int g = 1; g < G; ++g) {
        const int lane = (g - 1) % gl;
        modup(c, accb + (size_t)g * ctw, astride, cb, gy + lane * gy_l, L * n, gext + (size_t)(g - 1) * ext_w,
              (size_t)(G - 1) * ext_w, lane_stream(c, s, lane), false);
      }
    }
    if ((rc = join_lanes(c, s, gl))) return rc;
    fa::giant_ks(c, gext, accb, astride, keys.data(), ggal.data(), cb, G - 1, usum, s);
    std::vector<const double*> bases(2 * cb);
    std::vector<double*> douts(2 * cb);
    std::vector<uint32_t> gals(2 * cb, 1u);
    for (int blk = 0; blk < cb; ++blk) {
      const double* acc0 = accb + (size_t)blk * astride;
      bases[2 * blk] = acc0;
      bases[2 * blk + 1] = acc0 + L * n;
      douts[2 * blk] = outs[b0 + blk];
      douts[2 * blk + 1] = outs[b0 + blk] + L * n;
    }
    moddown_polys(c, usum, 2 * cb, gconv, bases.data(), douts.data(), gals.data(), s);
  }
  ar.used = mark;
  return FA_OK;
}

static int check_giant_keys(const fa_ctx* c, int d, int B) {
  for (int g = 1; g < d / B; ++g)
    if (!c->keys.count(g * B)) return fail(FA_E_NOKEY, "no rotation key for giant step %d", g * B);
  return FA_OK;
}

// Multiply-accumulate of nq queries' baby rotations against nb blocks (one
// pass over the plaintexts per group of up to FA_MAXQ queries), then each
// query's giant steps into outs[j].
static int mac_giant_phase(fa_ctx* c, const double* const* q, const double* const* qrot, int nq,
                           const double* const* blocks, int nb, int d, int B, double* const* outs, Arena& ar,
                           hipStream_t s) {
  const size_t ctw = 2 * (size_t)c->L * c->n;
  const int G = d / B;
  int rc = check_giant_keys(c, d, B);
  if (rc) return rc;
  // the queries' accumulators one after the other: their giant steps then run
  // as those of nq * nb blocks (larger launches, keys shared across queries)
  double* acc_all = ar.take((size_t)nq * nb * G * ctw);
  if (!acc_all) return fail(FA_E_NOMEM, "workspace too small for score_block");
  std::vector<double*> acc(nq);
  std::vector<double*> bouts((size_t)nq * nb);
  for (int j = 0; j < nq; ++j) {
    acc[j] = acc_all + (size_t)j * nb * G * ctw;
    for (int blk = 0; blk < nb; ++blk) bouts[(size_t)j * nb + blk] = outs[j] + (size_t)blk * ctw;
  }
  if (c->prof) HIPCHK(hipEventRecord(c->ev[1], s));
  fa::mac_diag(c, q, qrot, nq, blocks, nb, B, G, acc.data(), s);
  if (c->prof) HIPCHK(hipEventRecord(c->ev[2], s));
  if ((rc = giant_phase(c, acc_all, nq * nb, G, B, bouts.data(), ar, s))) return rc;
  if (c->prof) {
    HIPCHK(hipEventRecord(c->ev[3], s));
    c->prof_done = true;
  }
  return check_launch("score_block");
}

// Diagonal-layout scoring (baby-step / giant-step) of q against nb blocks.
static int score_diag(fa_ctx* c, const double* q, const double* const* blocks, int nb, int d, int B, double* out,
                      Arena& ar, hipStream_t s) {
  double* qrot = ar.take(qrot_words(c, B));
  if (!qrot) return fail(FA_E_NOMEM, "workspace too small for score_block");
  for (int g = 1; g < d / B; ++g)
    if (!c->keys.count(g * B)) return fail(FA_E_NOKEY, "no rotation key for giant step %d", g * B);
  if (c->prof) HIPCHK(hipEventRecord(c->ev[0], s));
  int rc = baby_phase(c, q, B, qrot, ar, s);
  if (rc) return rc;
  const double* qq = qrot;
  return mac_giant_phase(c, &q, &qq, 1, blocks, nb, d, B, &out, ar, s);
}

// Encrypted blocks (ct x ct): baby rotations, the tensor multiply-accumulate
// (three components per (block, giant)), one relinearisation per (block,
// giant), then the giant steps of the plaintext path on the relinearised sums.
static size_t score_enc_ws(const fa_ctx* c, int nb, int d, int B) {
  const size_t G = d / B, ln = (size_t)c->L * c->n;
  return baby_ws(c, B) + rup(qrot_words(c, B)) + rup((size_t)nb * G * 3 * ln) + giant_ws(c, nb, d, B) +
         relin_ws(c);
}
static int score_diag_enc(fa_ctx* c, const double* q, const double* const* blocks, int nb, int d, int B,
                          double* out, Arena& ar, hipStream_t s) {
  const size_t ln = (size_t)c->L * c->n;
  const int G = d / B;
  if (!c->d_rlk) return fail(FA_E_NOKEY, "no relinearisation key (fa_keygen_relin)");
  int rc = check_giant_keys(c, d, B);
  if (rc) return rc;
  double* qrot = ar.take(qrot_words(c, B));
  double* acc3 = ar.take((size_t)nb * G * 3 * ln);
  double* acc = ar.take((size_t)nb * G * 2 * ln);
  if (!qrot || !acc3 || !acc) return fail(FA_E_NOMEM, "workspace too small for score_block");
  if (c->prof) HIPCHK(hipEventRecord(c->ev[0], s));
  if ((rc = baby_phase(c, q, B, qrot, ar, s))) return rc;
  if (c->prof) HIPCHK(hipEventRecord(c->ev[1], s));
  fa::mac_diag_ct(c, q, qrot, blocks, nb, B, G, acc3, s);
  if (c->prof) HIPCHK(hipEventRecord(c->ev[2], s));
  if ((rc = relin_batch(c, acc3, nb * G, acc, ar, s))) return rc;
  std::vector<double*> bouts(nb);
  for (int blk = 0; blk < nb; ++blk) bouts[blk] = out + (size_t)blk * 2 * ln;
  if ((rc = giant_phase(c, acc, nb, G, B, bouts.data(), ar, s))) return rc;
  if (c->prof) {
    HIPCHK(hipEventRecord(c->ev[3], s));
    c->prof_done = true;
  }
  return check_launch("score_block(encrypted)");
}

extern "C" {

size_t fa_workspace_bytes(const fa_ctx* c, int op, int n_blocks, int d, int baby_step) {
  if (!c) return 0;
  switch (op) {
    case FA_OP_SCORE:
      if (baby_step < 1 || d < baby_step) return 0;
      return score_ws(c, std::max(1, n_blocks), d, baby_step);
    case FA_OP_PROJECT:
      if (baby_step < 1 || d < baby_step) return 0;
      return std::max(score_ws(c, 1, d, baby_step), rotate_ws(c, 1));
    case FA_OP_ROTATE_SUM:
    case FA_OP_ROTATE:
      return rotate_ws(c, std::min(std::max(1, n_blocks), kRotBatch)) + rup((fa_ct_bytes(c) / 8) * kRotBatch);
    case FA_OP_PREPARE:
      if (baby_step < 1) return 0;
      return baby_ws(c, baby_step);
    case FA_OP_SCORE_PREPARED:
      if (baby_step < 1 || d < baby_step) return 0;
      return giant_ws(c, std::max(1, n_blocks), d, baby_step);
    case FA_OP_SCORE_ENC:
      if (baby_step < 1 || d < baby_step) return 0;
      return score_enc_ws(c, std::max(1, n_blocks), d, baby_step);
    case FA_OP_PROJECT_ENC:
      if (baby_step < 1 || d < baby_step) return 0;
      return std::max(score_enc_ws(c, 1, d, baby_step), rotate_ws(c, 1));
    default:
      return 0;
  }
}

size_t fa_prepared_bytes(const fa_ctx* c, int baby_step) {
  return (c && baby_step >= 1) ? qrot_words(c, baby_step) * 8 : 0;
}

// The query ciphertext and its prepared baby rotations: prep must hold the
// baby_step - 1 rotations of q, at q's level and scale.
static int prep_check(const fa_ctx* c, const char* fn, const fa_buf* q, const fa_buf* prep, int baby_step) {
  int rc = in_check(c, q, fn, "q", 2, 1);
  if (rc) return rc;
  if (baby_step < 2) return prep && prep->dev ? FA_OK : fail(FA_E_INVAL, "%s: prep is null", fn);
  if ((rc = in_check(c, prep, fn, "prep", 2, (uint32_t)(baby_step - 1)))) return rc;
  if (prep->log_scale != q->log_scale)
    return fail(FA_E_SHAPE, "%s: prep is at scale 2^%d, the query at 2^%d", fn, prep->log_scale, q->log_scale);
  return FA_OK;
}

int fa_prepare_query(fa_ctx* c, const fa_buf* q, int baby_step, fa_buf* prep, void* ws, size_t ws_bytes,
                     void* stream) {
  if (!c) return fail(FA_E_INVAL, "fa_prepare_query: null context");
  if (baby_step < 1 || baby_step > c->n / 2) return fail(FA_E_INVAL, "baby_step %d out of range", baby_step);
  int rc = in_check(c, q, "fa_prepare_query", "q", 2, 1);
  if (rc || (rc = out_check(c, prep, "fa_prepare_query", "prep", (size_t)(baby_step - 1), 2))) return rc;
  const size_t need = baby_ws(c, baby_step);
  if (baby_step > 1 && (!ws || ws_bytes < need)) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  rc = baby_phase(c, (const double*)q->dev, baby_step, (double*)prep->dev, ar, (hipStream_t)stream);
  if (rc || (rc = check_launch("fa_prepare_query"))) return rc;
  out_set(c, prep, 2, (size_t)(baby_step - 1), q->log_scale);
  return FA_OK;
}

// queries whose baby steps are key-switched together: the per-launch item
// lists hold up to 32 key switches, so a group's steps per launch stay >= 2
constexpr int kBatchGroup = 16;

size_t fa_prepare_batch_workspace_bytes(const fa_ctx* c, int n_q, int baby_step) {
  if (!c || n_q < 1 || baby_step < 1) return 0;
  return baby_batch_ws(c, std::min(n_q, kBatchGroup), baby_step);
}

int fa_prepare_batch(fa_ctx* c, const fa_buf* qs, int n_q, int baby_step, fa_buf* preps, void* ws,
                     size_t ws_bytes, void* stream) {
  if (!c || !qs || !preps) return fail(FA_E_INVAL, "fa_prepare_batch: null argument");
  if (n_q < 1) return fail(FA_E_SHAPE, "n_q must be positive");
  if (baby_step < 1 || baby_step > c->n / 2) return fail(FA_E_INVAL, "baby_step %d out of range", baby_step);
  for (int j = 0; j < n_q; ++j) {
    int rc = in_check(c, &qs[j], "fa_prepare_batch", "a query", 2, 1);
    if (rc || (rc = out_check(c, &preps[j], "fa_prepare_batch", "a prepared buffer", (size_t)(baby_step - 1), 2)))
      return rc;
  }
  const size_t need = baby_batch_ws(c, std::min(n_q, kBatchGroup), baby_step);
  if (baby_step > 1 && (!ws || ws_bytes < need)) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  for (int j0 = 0; j0 < n_q; j0 += kBatchGroup) {
    const int m = std::min(kBatchGroup, n_q - j0);
    std::vector<const double*> qp(m);
    std::vector<double*> pp(m);
    for (int j = 0; j < m; ++j) {
      qp[j] = (const double*)qs[j0 + j].dev;
      pp[j] = (double*)preps[j0 + j].dev;
    }
    Arena ar{(char*)ws, ws_bytes, 0};
    int rc = baby_phase_batch(c, qp.data(), m, baby_step, pp.data(), ar, (hipStream_t)stream);
    if (rc) return rc;
  }
  for (int j = 0; j < n_q; ++j) out_set(c, &preps[j], 2, (size_t)(baby_step - 1), qs[j].log_scale);
  return FA_OK;
}

// Shape of a diagonal request (d a power of two <= S, baby step dividing d).
static int diag_shape(const fa_ctx* c, int d, int baby_step) {
  const int S = c->n / 2;
  if (d < 1 || (d & (d - 1)) || d > S) return fail(FA_E_SHAPE, "d=%d must be a power of two <= N/2", d);
  if (baby_step < 1 || d % baby_step) return fail(FA_E_INVAL, "baby_step %d must divide d=%d", baby_step, d);
  return FA_OK;
}

int fa_score_prepared(fa_ctx* c, const fa_buf* q, const fa_buf* prep, const fa_buf* blocks, int n_resident,
                      const int32_t* block_ids, int n_blocks, int d, int baby_step, fa_buf* out, void* ws,
                      size_t ws_bytes, void* stream) {
  const char* fn = "fa_score_prepared";
  if (!c) return fail(FA_E_INVAL, "%s: null context", fn);
  std::vector<const double*> bp;
  int32_t bls = 0;
  int rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, 1, 1, bp, &bls);
  if (rc || (rc = diag_shape(c, d, baby_step))) return rc;
  if ((rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, 1, (uint32_t)d, bp, &bls))) return rc;
  if ((rc = prep_check(c, fn, q, prep, baby_step))) return rc;
  if ((rc = scale_check(c, fn, (long)q->log_scale + bls))) return rc;
  if ((rc = out_check(c, out, fn, "out", n_blocks, 2))) return rc;
  const size_t need = giant_ws(c, n_blocks, d, baby_step);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  hipStream_t s = (hipStream_t)stream;
  if (c->prof) HIPCHK(hipEventRecord(c->ev[0], s));
  const double* qp = (const double*)q->dev;
  const double* pp = (const double*)prep->dev;
  double* op = (double*)out->dev;
  rc = mac_giant_phase(c, &qp, &pp, 1, bp.data(), n_blocks, d, baby_step, &op, ar, s);
  if (!rc) out_set(c, out, 2, n_blocks, q->log_scale + bls);
  return rc;
}

size_t fa_batch_workspace_bytes(const fa_ctx* c, int n_q, int n_blocks, int d, int baby_step) {
  if (!c || n_q < 1 || baby_step < 1 || d < baby_step) return 0;
  return giant_ws(c, std::max(1, n_blocks), d, baby_step, n_q);
}

int fa_score_batch(fa_ctx* c, const fa_buf* qs, const fa_buf* preps, int n_q, const fa_buf* blocks, int n_resident,
                   const int32_t* block_ids, int n_blocks, int d, int baby_step, fa_buf* outs, void* ws,
                   size_t ws_bytes, void* stream) {
  const char* fn = "fa_score_batch";
  if (!c || !qs || !preps || !outs) return fail(FA_E_INVAL, "%s: null argument", fn);
  if (n_q < 1) return fail(FA_E_SHAPE, "n_q must be positive");
  std::vector<const double*> bp;
  int32_t bls = 0;
  int rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, 1, 1, bp, &bls);
  if (rc || (rc = diag_shape(c, d, baby_step))) return rc;
  if ((rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, 1, (uint32_t)d, bp, &bls))) return rc;
  std::vector<const double*> qp(n_q), pp(n_q);
  std::vector<double*> op(n_q);
  for (int j = 0; j < n_q; ++j) {
    if ((rc = prep_check(c, fn, &qs[j], &preps[j], baby_step))) return rc;
    if ((rc = scale_check(c, fn, (long)qs[j].log_scale + bls))) return rc;
    if ((rc = out_check(c, &outs[j], fn, "an output", n_blocks, 2))) return rc;
    qp[j] = (const double*)qs[j].dev;
    pp[j] = (const double*)preps[j].dev;
    op[j] = (double*)outs[j].dev;
  }
  const size_t need = giant_ws(c, n_blocks, d, baby_step, n_q);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  hipStream_t s = (hipStream_t)stream;
  if (c->prof) HIPCHK(hipEventRecord(c->ev[0], s));
  rc = mac_giant_phase(c, qp.data(), pp.data(), n_q, bp.data(), n_blocks, d, baby_step, op.data(), ar, s);
  if (!rc)
    for (int j = 0; j < n_q; ++j) out_set(c, &outs[j], 2, n_blocks, qs[j].log_scale + bls);
  return rc;
}

int fa_score_block(fa_ctx* c, const fa_buf* q, const fa_buf* blocks, int n_resident, const int32_t* block_ids,
                   int n_blocks, int d, int layout, int baby_step, fa_buf* out, void* ws, size_t ws_bytes,
                   void* stream) {
  const char* fn = "fa_score_block";
  if (n_blocks < 1) return fail(FA_E_SHAPE, "n_blocks must be positive");
  if (!c) return fail(FA_E_INVAL, "%s: null context", fn);
  if (layout != FA_LAYOUT_ROW && layout != FA_LAYOUT_DIAG && layout != FA_LAYOUT_DIAG_ENC)
    return fail(FA_E_INVAL, "unknown layout %d", layout);
  const bool enc = layout == FA_LAYOUT_DIAG_ENC;
  const uint32_t kind = enc ? 2 : 1;
  std::vector<const double*> bp;
  int32_t bls = 0;
  int rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, kind, 1, bp, &bls);
  if (rc || (rc = in_check(c, q, fn, "q", 2, 1))) return rc;
  if (layout != FA_LAYOUT_ROW) {
    if ((rc = diag_shape(c, d, baby_step))) return rc;
    if ((rc = gather_blocks(c, fn, blocks, n_resident, block_ids, n_blocks, kind, (uint32_t)d, bp, &bls))) return rc;
  }
  if ((rc = scale_check(c, fn, (long)q->log_scale + bls))) return rc;
  if ((rc = out_check(c, out, fn, "out", n_blocks, 2))) return rc;
  hipStream_t s = (hipStream_t)stream;
  const double* qd = (const double*)q->dev;
  if (layout == FA_LAYOUT_ROW) {
    fa::mul_plain(c, qd, bp.data(), n_blocks, (double*)out->dev, s);
    if ((rc = check_launch("fa_score_block(row)"))) return rc;
    out_set(c, out, 2, n_blocks, q->log_scale + bls);
    return FA_OK;
  }
  const size_t need = enc ? score_enc_ws(c, n_blocks, d, baby_step) : score_ws(c, n_blocks, d, baby_step);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  rc = enc ? score_diag_enc(c, qd, bp.data(), n_blocks, d, baby_step, (double*)out->dev, ar, s)
           : score_diag(c, qd, bp.data(), n_blocks, d, baby_step, (double*)out->dev, ar, s);
  if (!rc) out_set(c, out, 2, n_blocks, q->log_scale + bls);
  return rc;
}

// ---- the membership path: rescale, ct x ct products, constants, polynomials ----

static bool chain_ok(const fa_ctx* hi, const fa_ctx* lo) {
  if (!hi || !lo || lo->L != hi->L - 1 || lo->K != hi->K || lo->n != hi->n) return false;
  for (int t = 0; t < lo->L; ++t)
    if (lo->primes[t] != hi->primes[t]) return false;
  for (int k = 0; k < hi->K; ++k)
    if (lo->primes[lo->L + k] != hi->primes[hi->L + k]) return false;
  return true;
}

size_t fa_chain_workspace_bytes(const fa_ctx* top, int degree) {
  if (!top || degree < 1) return 0;
  const size_t ctw = 2 * (size_t)top->L * top->n;
  const size_t gen = (size_t)std::max(1, degree / 2);  // the widest generation of Chebyshev terms
  // the terms, the sum and its rescale scratch; one generation's products (or a
  // sign step's: three ciphertexts and one product)
  return (size_t)(degree + 3) * rup(ctw) +
         std::max(gen * (2 * rup(ctw) + rup(3 * (size_t)top->L * top->n)), 4 * rup(ctw) + rup(3 * (size_t)top->L * top->n)) +
         relin_ws(top);
}

int fa_rescale(const fa_ctx* hi, const fa_ctx* lo, const void* ct, int n_polys, void* out, void* ws, size_t ws_bytes,
               void* stream) {
  if (!hi || !lo || !ct || !out) return fail(FA_E_INVAL, "fa_rescale: null argument");
  if (!chain_ok(hi, lo)) return fail(FA_E_SHAPE, "fa_rescale: the second context must be the first minus its last prime");
  if (n_polys < 1 || n_polys > 3) return fail(FA_E_SHAPE, "n_polys must be 1..3");
  const size_t need = rup((size_t)n_polys * hi->L * hi->n);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  fa::rescale(hi, (const double*)ct, n_polys, (double*)out, (double*)ws, (hipStream_t)stream);
  return check_launch("fa_rescale");
}

// relinearised products at one level, out_j = Relin(x_j (x) y_j) for count pairs:
// x_j = x + j*sx with xL limbs per polynomial (read as its drop to this level), likewise y;
// out [count][2][L][N]
static int mul_relin_n(fa_ctx* c, const double* x, int xL, size_t sx, const double* y, int yL, size_t sy, int count,
                       double* out, Arena& ar, hipStream_t s) {
  const size_t mark = ar.used;
  double* t3 = ar.take((size_t)count * 3 * c->L * c->n);
  if (!t3) return fail(FA_E_NOMEM, "workspace too small for a ciphertext product");
  fa::tensor(c, x, xL, sx, y, yL, sy, count, t3, s);
  const int rc = relin_batch(c, t3, count, out, ar, s);
  ar.used = mark;
  return rc;
}
static int mul_relin(fa_ctx* c, const double* x, const double* y, double* out, Arena& ar, hipStream_t s) {
  return mul_relin_n(c, x, c->L, 0, y, c->L, 0, 1, out, ar, s);
}

int fa_mul_ct(fa_ctx* c, const void* x, const void* y, void* out, void* ws, size_t ws_bytes, void* stream) {
  if (!c || !x || !y || !out) return fail(FA_E_INVAL, "fa_mul_ct: null argument");
  const size_t need = rup(3 * (size_t)c->L * c->n) + relin_ws(c);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  int rc = mul_relin(c, (const double*)x, (const double*)y, (double*)out, ar, (hipStream_t)stream);
  return rc ? rc : check_launch("fa_mul_ct");
}

// Residues mod each ciphertext prime of an integer-valued double v (|v| up to
// 2^1023): v = m * 2^e with m a 53-bit integer, so v mod q = (m mod q)(2^e mod q).
static std::vector<uint64_t> const_residues(const fa_ctx* c, double v) {
  std::vector<uint64_t> r(c->L);
  const bool neg = v < 0;
  const double a = std::fabs(v);
  int e = 0;
  const double fr = std::frexp(a, &e);  // a = fr * 2^e, fr in [0.5, 1)
  u64 m = 0;
  int sh = 0;
  if (e <= 53) {
    m = (u64)a;  // exact: a is an integer below 2^53
  } else {
    m = (u64)std::ldexp(fr, 53);  // 53-bit mantissa
    sh = e - 53;
  }
  for (int t = 0; t < c->L; ++t) {
    const u64 q = c->primes[t];
    u64 x = m % q;
    x = mulmod(x, powmod(2, (u64)sh, q), q);
    r[t] = neg && x ? q - x : x;
  }
  return r;
}
static std::vector<uint64_t> const_residues(const fa_ctx* c, int64_t k) {
  std::vector<uint64_t> r(c->L);
  for (int t = 0; t < c->L; ++t) {
    const int64_t q = (int64_t)c->primes[t];
    const int64_t x = k % q;
    r[t] = (uint64_t)(x < 0 ? x + q : x);
  }
  return r;
}

int fa_ct_add(fa_ctx* c, const void* x, const void* y, void* out, int subtract, void* stream) {
  if (!c || !x || !y || !out) return fail(FA_E_INVAL, "fa_ct_add: null argument");
  fa::ct_elem(c, (const double*)x, (const double*)y, (double*)out, 2, nullptr, subtract ? 3 : 2,
              (hipStream_t)stream);
  return check_launch("fa_ct_add");
}

int fa_ct_mul_const(fa_ctx* c, const void* x, int64_t k, void* out, void* stream) {
  if (!c || !x || !out) return fail(FA_E_INVAL, "fa_ct_mul_const: null argument");
  const auto r = const_residues(c, k);
  fa::ct_elem(c, (const double*)x, nullptr, (double*)out, 2, r.data(), 0, (hipStream_t)stream);
  return check_launch("fa_ct_mul_const");
}

int fa_ct_add_const(fa_ctx* c, const void* x, double k, void* out, void* stream) {
  if (!c || !x || !out) return fail(FA_E_INVAL, "fa_ct_add_const: null argument");
  if (!(std::fabs(k) < 0x1p1000) || k != std::nearbyint(k)) return fail(FA_E_INVAL, "k must be an integer value");
  const auto r = const_residues(c, k);
  fa::ct_elem(c, (const double*)x, nullptr, (double*)out, 2, r.data(), 1, (hipStream_t)stream);
  return check_launch("fa_ct_add_const");
}

namespace {
// A ciphertext in the chain: device words [2][L][N], its level and scale.
struct CtRef {
  double* p;
  int L;
  double s;
};
struct Chain {
  std::vector<fa_ctx*> by_L;  // index L -> context with L ciphertext primes
  fa_ctx* at(int L) const { return L >= 0 && L < (int)by_L.size() ? by_L[L] : nullptr; }
};
int make_chain(fa_ctx* const* levels, int n_levels, Chain& ch) {
  if (!levels || n_levels < 2) return fail(FA_E_INVAL, "a chain needs at least two levels");
  ch.by_L.assign(levels[0] ? levels[0]->L + 1 : 0, nullptr);
  for (int i = 0; i < n_levels; ++i) {
    if (!levels[i] || (i && !chain_ok(levels[i - 1], levels[i])))
      return fail(FA_E_SHAPE, "levels[%d] must hold the primes of levels[%d] minus its last ciphertext prime", i, i - 1);
    if (!levels[i]->d_rlk) return fail(FA_E_NOKEY, "level with %d primes has no relinearisation key", levels[i]->L);
    ch.by_L[levels[i]->L] = levels[i];
  }
  return FA_OK;
}
}  // namespace

// count products x_j * y_j of chain ciphertexts (x_j = x + j*sx at level Lx, y_j = y + j*sy
// at level Ly) at L = min(Lx, Ly), relinearised and rescaled into dst ([count][2][L-1][N]);
// scratch from ar
static int chain_mul_rescale_n(const Chain& ch, const double* x, int Lx, size_t sx, const double* y, int Ly,
                               size_t sy, int count, double* dst, Arena& ar, hipStream_t s) {
  const int L = std::min(Lx, Ly);
  fa_ctx* c = ch.at(L);
  if (!c || !ch.at(L - 1)) return fail(FA_E_SHAPE, "the chain has no level %d", L - 1);
  const size_t mark = ar.used, cw = (size_t)count * 2 * L * c->n;
  double* prod = ar.take(cw);
  double* scr = ar.take(cw);
  if (!prod || !scr) return fail(FA_E_NOMEM, "workspace too small for a chain product");
  int rc;
  if ((rc = mul_relin_n(c, x, Lx, sx, y, Ly, sy, count, prod, ar, s))) return rc;
  fa::rescale(c, prod, 2 * count, dst, scr, s);
  ar.used = mark;
  return FA_OK;
}
// workspace of chain_mul_rescale_n at level L (count pairs)
static size_t mul_rescale_ws(const fa_ctx* c, int count) {
  const size_t cw = (size_t)count * 2 * c->L * c->n;
  return 2 * rup(cw) + rup((size_t)count * 3 * c->L * c->n) + relin_ws(c);
}
static int chain_mul_rescale(const Chain& ch, const CtRef& a, const CtRef& b, double* dst, CtRef& out, Arena& ar,
                             hipStream_t s) {
  const int L = std::min(a.L, b.L);
  int rc = chain_mul_rescale_n(ch, a.p, a.L, 0, b.p, b.L, 0, 1, dst, ar, s);
  if (rc) return rc;
  out = {dst, L - 1, a.s * b.s / (double)ch.at(L)->primes[L - 1]};
  return FA_OK;
}

// sum_k coeffs[k] T_k(u) by the direct evaluator into out (scale u.s); the
// terms and their scratch come from ar and are released on return.  The terms
// are formed generation by generation (T_2; T_3, T_4; T_5 .. T_8; ...): every
// product of a generation reads terms of earlier generations only and sits at
// one level, so a generation is one batched product, one fix-up and one rescale.
static int cheb_core(const Chain& ch, const CtRef& u, const double* coeffs, int degree, double* out, CtRef& res,
                     Arena& ar, hipStream_t s) {
  const size_t mark = ar.used;
  std::vector<CtRef> T(degree + 1);
  T[1] = u;
  int rc;
  // T_k = Rescale(2 T_a T_b - T_{a-b}), with T_{a-b} brought to the product's
  // scale s_a s_b before the rescale: T_0 = 1 as the constant round(s_a s_b),
  // T_1 times the integer round(s_a s_b / s_1)
  for (int k0 = 2; k0 <= degree; k0 = 2 * k0 - 1) {
    const int k1 = std::min(degree, 2 * (k0 - 1));  // generation k0 .. k1
    const int count = k1 - k0 + 1;
    std::vector<const double*> xs(count), ys(count);
    std::vector<int> xLs(count), yLs(count), odd(count);
    std::vector<double> sp(count);
    int L = u.L;
    for (int j = 0; j < count; ++j) {
      const int k = k0 + j, a = (k + 1) / 2, b = k / 2;
      xs[j] = T[a].p;
      ys[j] = T[b].p;
      xLs[j] = T[a].L;
      yLs[j] = T[b].L;
      odd[j] = k & 1;
      sp[j] = T[a].s * T[b].s;
      L = std::min(L, std::min(T[a].L, T[b].L));
    }
    fa_ctx* c = ch.at(L);
    if (!c || !ch.at(L - 1)) return fail(FA_E_SHAPE, "the chain has no level %d", L - 1);
    const size_t cw = 2 * (size_t)L * c->n, cwo = 2 * (size_t)(L - 1) * c->n;
    double* gen = ar.take((size_t)count * cwo);
    if (!gen) return fail(FA_E_NOMEM, "workspace too small for the Chebyshev terms");
    const size_t mark_g = ar.used;
    double* prod = ar.take((size_t)count * cw);
    double* scr = ar.take((size_t)count * cw);
    double* t3 = ar.take((size_t)count * 3 * L * c->n);
    if (!prod || !scr || !t3) return fail(FA_E_NOMEM, "workspace too small for the Chebyshev terms");
    fa::tensor_list(c, xs.data(), xLs.data(), ys.data(), yLs.data(), count, t3, s);
    if ((rc = relin_batch(c, t3, count, prod, ar, s))) return rc;
    std::vector<std::vector<uint64_t>> cres(count);
    std::vector<const uint64_t*> cptr(count);
    for (int j = 0; j < count; ++j) {
      cres[j] = odd[j] ? const_residues(c, std::nearbyint(sp[j] / T[1].s)) : const_residues(c, -std::nearbyint(sp[j]));
      cptr[j] = cres[j].data();
    }
    fa::cheb_fix(c, prod, count, T[1].p, T[1].L, cptr.data(), odd.data(), s);
    fa::rescale(c, prod, 2 * count, gen, scr, s);
    for (int j = 0; j < count; ++j) T[k0 + j] = {gen + (size_t)j * cwo, L - 1, sp[j] / (double)c->primes[L - 1]};
    ar.used = mark_g;
  }
  int Lmin = u.L;
  for (int k = 1; k <= degree; ++k) Lmin = std::min(Lmin, T[k].L);
  fa_ctx* c = ch.at(Lmin);
  if (!ch.at(Lmin - 1)) return fail(FA_E_SHAPE, "the chain has no level %d", Lmin - 1);
  const double qn = (double)c->primes[Lmin - 1];
  const size_t cw = 2 * (size_t)Lmin * c->n;
  double* acc = ar.take(cw);
  double* scr = ar.take(cw);
  if (!acc || !scr) return fail(FA_E_NOMEM, "workspace too small for the Chebyshev sum");
  // every term is brought to the one scale u.s * qn: its constant carries u.s / T_k.s
  std::vector<std::vector<uint64_t>> ck(degree);
  std::vector<const uint64_t*> cptr(degree);
  std::vector<const double*> xs(degree);
  std::vector<int> xLs(degree);
  for (int k = 1; k <= degree; ++k) {
    ck[k - 1] = const_residues(c, std::nearbyint(coeffs[k] * qn * (u.s / T[k].s)));
    cptr[k - 1] = ck[k - 1].data();
    xs[k - 1] = T[k].p;
    xLs[k - 1] = T[k].L;
  }
  const double s_acc = u.s * qn;
  const auto c0 = const_residues(c, std::nearbyint(coeffs[0] * s_acc));
  fa::lincomb(c, acc, xs.data(), xLs.data(), cptr.data(), degree, c0.data(), s);
  fa::rescale(c, acc, 2, out, scr, s);
  res = {out, Lmin - 1, s_acc / qn};
  ar.used = mark;
  return FA_OK;
}

// iters sign steps on count ciphertexts at once: V_j = v + j*sv at level L (scale s_v,
// multiplier m), results at out + j*so; v is not written.  Returns the final level,
// scale and multiplier.
static int sign_core_n(const Chain& ch, const double* v, int L, size_t sv, int count, double s_v, int64_t m,
                       int iters, double* out, size_t so, CtRef& res, int64_t& m_out, Arena& ar, hipStream_t s) {
  const size_t mark = ar.used;
  const size_t cw = (size_t)count * 2 * L * ch.at(L)->n;
  double* zb = ar.take(cw);
  double* vb[2] = {ar.take(cw), ar.take(cw)};
  if (!zb || !vb[0] || !vb[1]) return fail(FA_E_NOMEM, "workspace too small for the sign iteration");
  int rc;
  const double* V = v;
  size_t stride = sv;
  for (int it = 0; it < iters; ++it) {
    const double mm = (double)m;
    // z = V^2, then 3 m^2 - z (at z's scale)
    if ((rc = chain_mul_rescale_n(ch, V, L, stride, V, L, stride, count, zb, ar, s))) return rc;
    fa_ctx* c = ch.at(L);
    const int Lz = L - 1;
    fa_ctx* cz = ch.at(Lz);
    const double sz = s_v * s_v / (double)c->primes[L - 1];
    const auto m1 = const_residues(cz, (int64_t)-1);
    const auto k3 = const_residues(cz, std::nearbyint(3.0 * mm * mm * sz));
    fa::ct_elem(cz, zb, nullptr, zb, 2 * count, m1.data(), 0, s);
    fa::ct_elem(cz, zb, nullptr, zb, 2 * count, k3.data(), 1, s);
    // V <- V (3 m^2 - V^2) at level Lz - 1
    const bool last = it == iters - 1;
    double* dst = last && (count == 1 || so == 2 * (size_t)(Lz - 1) * cz->n) ? out : vb[it & 1];
    if ((rc = chain_mul_rescale_n(ch, V, L, stride, zb, Lz, 2 * (size_t)Lz * cz->n, count, dst, ar, s))) return rc;
    s_v = s_v * sz / (double)cz->primes[Lz - 1];
    L = Lz - 1;
    V = dst;
    stride = 2 * (size_t)L * cz->n;
    m = 2 * m * m * m;
  }
  if (V != out) {
    const size_t words = 2 * (size_t)L * ch.at(L)->n;
    for (int j = 0; j < count; ++j)
      HIPCHK(hipMemcpyAsync(out + j * so, V + j * stride, words * 8, hipMemcpyDeviceToDevice, s));
  }
  res = {out, L, s_v};
  m_out = m;
  ar.used = mark;
  return FA_OK;
}
static size_t sign_ws(const fa_ctx* c, int count) {
  return 3 * rup((size_t)count * 2 * c->L * c->n) + mul_rescale_ws(c, count);
}

// levels the direct evaluator of this degree spends: ceil(log2 degree) product
// generations and the final rescale
static int cheb_depth(int degree) {
  int g = 0;
  while ((1 << g) < degree) ++g;
  return g + 1;
}
// every level from L down to L - depth is in the chain (checked before any launch)
static int chain_spans(const Chain& ch, int L, int depth) {
  for (int l = L; l >= L - depth; --l)
    if (!ch.at(l)) return fail(FA_E_SHAPE, "the chain has no level %d (%d levels needed below %d)", l, depth, L);
  return FA_OK;
}

static int sign_args_ok(int64_t m, int iters) {
  if (iters < 1 || iters > 8) return fail(FA_E_INVAL, "iters %d out of [1, 8]", iters);
  for (int64_t mm = m, it = 0; it < iters; ++it, mm = 2 * mm * mm * mm)
    if (mm < 1 || mm > (INT64_C(1) << 20)) return fail(FA_E_INVAL, "multiplier out of range at iteration %d", (int)it);
  return FA_OK;
}

int fa_cheb_eval(fa_ctx* const* levels, int n_levels, const void* u, int L_u, double s_u, const double* coeffs,
                 int degree, void* out, int* L_out, double* s_out, void* ws, size_t ws_bytes, void* stream) {
  if (!u || !coeffs || !out || !L_out || !s_out) return fail(FA_E_INVAL, "fa_cheb_eval: null argument");
  if (degree < 1 || degree > 64) return fail(FA_E_INVAL, "degree %d out of [1, 64]", degree);
  Chain ch;
  int rc = make_chain(levels, n_levels, ch);
  if (rc) return rc;
  if ((rc = chain_spans(ch, L_u, cheb_depth(degree)))) return rc;
  const size_t need = fa_chain_workspace_bytes(levels[0], degree);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  CtRef res;
  if ((rc = cheb_core(ch, {(double*)u, L_u, s_u}, coeffs, degree, (double*)out, res, ar, (hipStream_t)stream)))
    return rc;
  *L_out = res.L;
  *s_out = res.s;
  return check_launch("fa_cheb_eval");
}

int fa_sign_iter(fa_ctx* const* levels, int n_levels, const void* v, int L_v, double s_v, int64_t m, int iters,
                 void* out, int* L_out, double* s_out, int64_t* m_out, void* ws, size_t ws_bytes, void* stream) {
  if (!v || !out || !L_out || !s_out || !m_out) return fail(FA_E_INVAL, "fa_sign_iter: null argument");
  int rc = sign_args_ok(m, iters);
  if (rc) return rc;
  Chain ch;
  if ((rc = make_chain(levels, n_levels, ch))) return rc;
  if ((rc = chain_spans(ch, L_v, 2 * iters))) return rc;
  const size_t need = fa_chain_workspace_bytes(levels[0], 3);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  Arena ar{(char*)ws, ws_bytes, 0};
  CtRef res;
  if ((rc = sign_core_n(ch, (const double*)v, L_v, 0, 1, s_v, m, iters, (double*)out, 0, res, *m_out, ar,
                       (hipStream_t)stream)))
    return rc;
  *L_out = res.L;
  *s_out = res.s;
  return check_launch("fa_sign_iter");
}

int fa_cheb_fit_sqrt(double tau, double y_lo, double y_hi, int degree, double* coeffs) {
  if (!coeffs) return fail(FA_E_INVAL, "fa_cheb_fit_sqrt: null argument");
  if (degree < 1 || degree > 64) return fail(FA_E_INVAL, "degree %d out of [1, 64]", degree);
  if (!(y_lo > 0) || !(y_hi > y_lo)) return fail(FA_E_INVAL, "need 0 < y_lo < y_hi");
  // interpolation at the n = degree + 1 Chebyshev points of the first kind,
  // u_j = cos(pi (j + 1/2) / n):  c_k = (2/n) sum_j g(u_j) cos(k pi (j + 1/2) / n), c_0 halved
  const int n = degree + 1;
  const double pi = 3.14159265358979323846;
  const double half = 0.5 * (y_hi - y_lo), mid = 0.5 * (y_hi + y_lo);
  std::vector<double> g(n);
  for (int j = 0; j < n; ++j) g[j] = tau * std::sqrt(mid + half * std::cos(pi * (j + 0.5) / n));
  for (int k = 0; k < n; ++k) {
    double acc = 0;
    for (int j = 0; j < n; ++j) acc += g[j] * std::cos(pi * k * (j + 0.5) / n);
    coeffs[k] = (k ? 2.0 : 1.0) * acc / n;
  }
  return FA_OK;
}

static bool has_rotations(const fa_ctx* c, const std::vector<int>& steps) {
  for (int r : steps)
    if (!c->keys.count(r)) return false;
  return true;
}

// Workspace of the membership scan, in three regions: the rescaled scores;
// the threshold chain (y, t, fold scratch and the chain's products), which
// runs on the side stream while the scores are formed; the scoring (raw
// scores, the diagonal product, the rescale scratch), reused after both have
// joined for the differences and the batched sign steps.
static void membership_regions(const fa_ctx* cq, int n_blocks, int d, int baby_step, int degree, size_t r[3]) {
  const size_t ctw = 2 * (size_t)cq->L * cq->n;
  const size_t nb = (size_t)n_blocks;
  r[0] = rup(nb * ctw);
  r[1] = 3 * rup(ctw) + std::max(rotate_ws(cq, 1), fa_chain_workspace_bytes(cq, std::max(degree, 3)));
  r[1] = (r[1] + 255) & ~(size_t)255;  // the next region starts aligned
  r[2] = std::max(rup(nb * ctw) + std::max(score_ws(cq, n_blocks, d, baby_step), rup(nb * ctw)),
                  rup(nb * ctw) + sign_ws(cq, n_blocks));
}
size_t fa_membership_workspace_bytes(const fa_ctx* cq, int n_blocks, int d, int baby_step, int degree) {
  if (!cq || n_blocks < 1 || d < 1 || baby_step < 1 || d % baby_step || degree < 1) return 0;
  size_t r[3];
  membership_regions(cq, n_blocks, d, baby_step, degree, r);
  return r[0] + r[1] + r[2];
}

static int ensure_side(fa_ctx* c) {
  if (!c->side) HIPCHK(hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking));
  if (!c->side_fork) HIPCHK(hipEventCreateWithFlags(&c->side_fork, hipEventDisableTiming));
  if (!c->side_join) HIPCHK(hipEventCreateWithFlags(&c->side_join, hipEventDisableTiming));
  return FA_OK;
}

int fa_membership(fa_ctx* const* levels, int n_levels, const void* q_r, int L_q, double s_q,
                  const void* const* blocks, int n_blocks, int d, int baby_step, double y_lo, double y_hi,
                  const double* coeffs, int degree, int64_t m, int iters, void* out, int* L_out, double* s_out,
                  int64_t* m_out, void* ws, size_t ws_bytes, void* stream) {
  if (!q_r || !blocks || !coeffs || !out || !L_out || !s_out || !m_out)
    return fail(FA_E_INVAL, "fa_membership: null argument");
  if (n_blocks < 1) return fail(FA_E_SHAPE, "n_blocks must be positive");
  for (int i = 0; i < n_blocks; ++i)
    if (!blocks[i]) return fail(FA_E_INVAL, "block %d is null", i);
  if (degree < 1 || degree > 64) return fail(FA_E_INVAL, "degree %d out of [1, 64]", degree);
  if (!(y_hi > y_lo)) return fail(FA_E_INVAL, "need y_lo < y_hi");
  int rc = sign_args_ok(m, iters);
  if (rc) return rc;
  Chain ch;
  if ((rc = make_chain(levels, n_levels, ch))) return rc;
  fa_ctx* cq = ch.at(L_q);
  fa_ctx* cy = ch.at(L_q - 1);
  if (!cq || !cy) return fail(FA_E_SHAPE, "the chain has no level %d or %d", L_q, L_q - 1);
  const int S = cq->n / 2;
  if (d < 2 || (d & (d - 1)) || d > S) return fail(FA_E_SHAPE, "d=%d must be a power of two in [2, N/2]", d);
  if (baby_step < 1 || d % baby_step) return fail(FA_E_INVAL, "baby_step %d must divide d=%d", baby_step, d);
  std::vector<int> fold;
  for (int k = 1; k < d; k <<= 1) fold.push_back(k);
  if (!has_rotations(cy, fold)) return fail(FA_E_NOKEY, "level %d lacks a rotation key for the norm's fold", L_q - 1);
  if ((rc = chain_spans(ch, L_q, 1 + cheb_depth(degree) + 2 * iters))) return rc;
  for (int g = 1; g < d / baby_step; ++g)
    if (!cq->keys.count(g * baby_step)) return fail(FA_E_NOKEY, "no rotation key for giant step %d", g * baby_step);
  for (int b = 1; b < baby_step; ++b)
    if (!cq->keys.count(b)) return fail(FA_E_NOKEY, "no rotation key for baby step %d", b);
  size_t reg[3];
  membership_regions(cq, n_blocks, d, baby_step, degree, reg);
  const size_t need = reg[0] + reg[1] + reg[2];
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  if ((rc = ensure_side(cq))) return rc;
  hipStream_t s = (hipStream_t)stream, s2 = cq->side;
  char* base = (char*)ws;
  Arena ar_th{base + reg[0], reg[1], 0};           // threshold chain (side stream)
  Arena ar{base + reg[0] + reg[1], reg[2], 0};     // scoring, then differences and signs
  const size_t n = cq->n, ctw_q = 2 * (size_t)L_q * n, ctw_y = 2 * (size_t)(L_q - 1) * n;
  double* scores = (double*)base;

  // the threshold chain depends only on q_r: fork it onto the side stream
  const double s_sc = s_q * std::ldexp(1.0, cq->log_scale) / (double)cq->primes[L_q - 1];
  double* tb = ar_th.take(ctw_q);
  CtRef t;
  HIPCHK(hipEventRecord(cq->side_fork, s));
  HIPCHK(hipStreamWaitEvent(s2, cq->side_fork, 0));
  auto threshold = [&]() -> int {
    // y = |q_R|^2 in every slot: the rescaled square folded over d slots
    double* yb = ar_th.take(ctw_q);
    double* rb = ar_th.take(ctw_q);
    if (!yb || !tb || !rb) return fail(FA_E_NOMEM, "workspace too small for the threshold");
    CtRef q{(double*)q_r, L_q, s_q}, y;
    int e;
    if ((e = chain_mul_rescale(ch, q, q, yb, y, ar_th, s2))) return e;
    for (int r : fold) {
      if ((e = rotate_batch(cy, yb, 1, r, rb, ar_th, s2))) return e;
      fa::add_automorph(cy, yb, rb, 2, 1u, s2);
    }
    // u = alpha (y - mid) in [-1, 1]: the factor alpha costs nothing, it is taken
    // into the scale (u at scale y.s / alpha); the shift is an added constant
    const double alpha = 2.0 / (y_hi - y_lo), mid = 0.5 * (y_hi + y_lo);
    const auto cm = const_residues(cy, std::nearbyint(-mid * y.s));
    fa::ct_elem(cy, yb, nullptr, yb, 2, cm.data(), 1, s2);
    const CtRef u{yb, y.L, y.s / alpha};
    // t = tau |q_R| at the scores' scale: the coefficients carry s_sc / s_u
    std::vector<double> cf(degree + 1);
    const double ratio = s_sc / u.s;
    for (int k = 0; k <= degree; ++k) cf[k] = coeffs[k] * ratio;
    return cheb_core(ch, u, cf.data(), degree, tb, t, ar_th, s2);
  };
  // the scores <q_R, x_i> of every block on the caller's stream, rescaled
  // (level L_q - 1, scale s_sc), enqueued first: the threshold chain's many
  // small launches are enqueued after them and run beside them
  double* raw = ar.take((size_t)n_blocks * ctw_q);
  rc = raw ? score_diag(cq, (const double*)q_r, (const double* const*)blocks, n_blocks, d, baby_step, raw, ar, s)
           : fail(FA_E_NOMEM, "workspace too small for the scores");
  if (!rc) {
    ar.used = rup((size_t)n_blocks * ctw_q);
    double* scr = ar.take((size_t)n_blocks * ctw_q);
    if (scr) fa::rescale(cq, raw, 2 * n_blocks, scores, scr, s);
    else rc = fail(FA_E_NOMEM, "workspace too small for the scores' rescale");
  }
  if (!rc) rc = threshold();
  // joined back on every path, so that no side-stream work outlives the call's stream order
  HIPCHK(hipEventRecord(cq->side_join, s2));
  HIPCHK(hipStreamWaitEvent(s, cq->side_join, 0));
  if (rc) return rc;
  ar.used = 0;

  // every block at once: (score - t) at t's level, then the sign steps on all of them
  fa_ctx* ct = ch.at(t.L);
  const size_t ctw_t = 2 * (size_t)t.L * n;
  double* db = ar.take((size_t)n_blocks * ctw_t);
  if (!db) return fail(FA_E_NOMEM, "workspace too small for the differences");
  fa::ct_elem(ct, scores, tb, db, 2 * n_blocks, nullptr, 3, s, L_q - 1, ctw_y, 0, ctw_t);
  CtRef res{};
  int64_t mo = m;
  if ((rc = sign_core_n(ch, db, t.L, ctw_t, n_blocks, s_sc, m, iters, (double*)out, ctw_q, res, mo, ar, s)))
    return rc;
  *L_out = res.L;
  *s_out = res.s;
  *m_out = mo;
  return check_launch("fa_membership");
}

int fa_rotate(fa_ctx* c, const fa_buf* ct, int step, fa_buf* out, void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(FA_E_INVAL, "fa_rotate: null context");
  int rc = in_check(c, ct, "fa_rotate", "ct", 2, 1);
  if (rc || (rc = out_check(c, out, "fa_rotate", "out", 1, 2))) return rc;
  if (overlap(ct, out)) return fail(FA_E_INVAL, "fa_rotate: out overlaps ct (the rotation cannot run in place)");
  if (step < 1 || step >= c->n / 2) return fail(FA_E_INVAL, "step %d out of [1, N/2)", step);
  if (!c->keys.count(step)) return fail(FA_E_NOKEY, "no rotation key for step %d", step);
  if (!ws || ws_bytes < rotate_ws(c, 1)) return fail(FA_E_NOMEM, "workspace too small for rotation");
  Arena ar{(char*)ws, ws_bytes, 0};
  rc = rotate_batch(c, (const double*)ct->dev, 1, step, (double*)out->dev, ar, (hipStream_t)stream);
  if (!rc) out_set(c, out, 2, 1, ct->log_scale);
  return rc;
}

int fa_rotate_static(fa_ctx* c, const fa_buf* ct, int step, fa_buf* out, void* stream) {
  if (!c) return fail(FA_E_INVAL, "fa_rotate_static: null context");
  const size_t need = rotate_ws(c, 1);
  if (need > FA_STATIC_SCRATCH_BYTES)
    return fail(FA_E_NOMEM, "fa_rotate_static: this context's rotation needs %zu bytes of scratch, the fixed array "
                "holds %zu", need, (size_t)FA_STATIC_SCRATCH_BYTES);
  if (!c->static_scratch)
    return fail(FA_E_HIP, "fa_rotate_static: the fixed scratch array is not available on device %d: %s", c->device,
                hipGetErrorString(c->static_scratch_err));
  return fa_rotate(c, ct, step, out, c->static_scratch, FA_STATIC_SCRATCH_BYTES, stream);
}

int fa_rotate_sum(fa_ctx* c, fa_buf* cts_b, int first_shift, int n_steps, void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(FA_E_INVAL, "fa_rotate_sum: null context");
  if (int rc = in_check(c, cts_b, "fa_rotate_sum", "cts", 2, 1)) return rc;
  const int n_cts = (int)cts_b->count;
  void* cts = cts_b->dev;
  if (n_steps < 0 || first_shift < 1) return fail(FA_E_INVAL, "fa_rotate_sum: bad sizes");
  for (int k = 0; k < n_steps; ++k) {
    const long r = (long)first_shift << k;
    if (r >= c->n / 2) return fail(FA_E_INVAL, "rotation %ld out of [1, N/2)", r);
    if (!c->keys.count((int)r)) return fail(FA_E_NOKEY, "no rotation key for step %ld", r);
  }
  const size_t need = fa_workspace_bytes(c, FA_OP_ROTATE_SUM, n_cts, 0, 1);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  const size_t ctw = (fa_ct_bytes(c) / 8);
  Arena ar{(char*)ws, ws_bytes, 0};
  double* tmp = ar.take(ctw * kRotBatch);
  double* base = (double*)cts;
  for (int c0 = 0; c0 < n_cts; c0 += kRotBatch) {
    const int nb = std::min(kRotBatch, n_cts - c0);
    double* cur = base + (size_t)c0 * ctw;
    for (int k = 0; k < n_steps; ++k) {
      int rc = rotate_batch(c, cur, nb, first_shift << k, tmp, ar, s);
      if (rc) return rc;
      fa::add_automorph(c, cur, tmp, 2 * nb, 1u, s);
    }
  }
  return check_launch("fa_rotate_sum");
}

int fa_profile(fa_ctx* c, int enable) {
  if (!c) return fail(FA_E_INVAL, "fa_profile: null context");
  if (enable && !c->ev[0])
    for (auto& e : c->ev) HIPCHK(hipEventCreate(&e));
  c->prof = enable != 0;
  return FA_OK;
}

int fa_profile_read(fa_ctx* c, double* ms) {
  if (!c || !ms) return fail(FA_E_INVAL, "fa_profile_read: null argument");
  if (!c->prof_done) return fail(FA_E_INVAL, "fa_profile_read: no profiled call");
  HIPCHK(hipEventSynchronize(c->ev[3]));
  float t[4];
  HIPCHK(hipEventElapsedTime(&t[0], c->ev[0], c->ev[1]));
  HIPCHK(hipEventElapsedTime(&t[1], c->ev[1], c->ev[2]));
  HIPCHK(hipEventElapsedTime(&t[2], c->ev[2], c->ev[3]));
  HIPCHK(hipEventElapsedTime(&t[3], c->ev[0], c->ev[3]));
  for (int i = 0; i < 4; ++i) ms[i] = t[i];
  return FA_OK;
}

// The projection q_R = W^T q: the diagonal product of q with the r hybrid
// diagonals of W (plaintexts, or ciphertexts when enc), then the fold
// z += Rotate(z, r * 2^k) while r * 2^k < d_in.
static int project(fa_ctx* c, const fa_buf* qb, const fa_buf* wb, bool enc, int d_in, int r, int baby_step,
                   fa_buf* qrb, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = enc ? "fa_project_ct_enc" : "fa_project_ct";
  if (!c) return fail(FA_E_INVAL, "%s: null context", fn);
  if (r < 1 || (r & (r - 1)) || d_in < r || d_in % r || ((d_in / r) & (d_in / r - 1)) || d_in > c->n / 2)
    return fail(FA_E_SHAPE, "d_in=%d, r=%d: both powers of two with r <= d_in <= N/2", d_in, r);
  int rc0 = in_check(c, qb, fn, "q", 2, 1);
  if (rc0 || (rc0 = in_check(c, wb, fn, enc ? "w_cts" : "w_pts", enc ? 2 : 1, (uint32_t)r))) return rc0;
  if ((rc0 = scale_check(c, fn, (long)qb->log_scale + wb->log_scale))) return rc0;
  if ((rc0 = out_check(c, qrb, fn, "q_r", 1, 2))) return rc0;
  if (overlap(qb, qrb)) return fail(FA_E_INVAL, "%s: q_r overlaps q", fn);
  const void* q = qb->dev;
  const void* w = wb->dev;
  void* q_r = qrb->dev;
  if (baby_step < 1 || r % baby_step) return fail(FA_E_INVAL, "baby_step %d must divide r=%d", baby_step, r);
  const size_t need = fa_workspace_bytes(c, enc ? FA_OP_PROJECT_ENC : FA_OP_PROJECT, 1, r, baby_step);
  if (!ws || ws_bytes < need) return fail(FA_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, need);
  int steps = 0;
  while ((r << steps) < d_in) ++steps;
  for (int k = 0; k < steps; ++k)
    if (!c->keys.count(r << k)) return fail(FA_E_NOKEY, "no rotation key for fold step %d", r << k);
  hipStream_t s = (hipStream_t)stream;
  Arena ar{(char*)ws, ws_bytes, 0};
  const void* blocks[1] = {w};
  int rc = enc ? score_diag_enc(c, (const double*)q, (const double* const*)blocks, 1, r, baby_step, (double*)q_r, ar, s)
               : score_diag(c, (const double*)q, (const double* const*)blocks, 1, r, baby_step, (double*)q_r, ar, s);
  if (rc) return rc;
  for (int k = 0; k < steps; ++k) {
    Arena ar2{(char*)ws, ws_bytes, 0};
    double* tmp = ar2.take((fa_ct_bytes(c) / 8));
    rc = rotate_batch(c, (const double*)q_r, 1, r << k, tmp, ar2, s);
    if (rc) return rc;
    fa::add_automorph(c, (double*)q_r, tmp, 2, 1u, s);
  }
  if ((rc = check_launch(fn))) return rc;
  out_set(c, qrb, 2, 1, qb->log_scale + wb->log_scale);
  return FA_OK;
}

int fa_project_ct(fa_ctx* c, const fa_buf* q, const fa_buf* w_pts, int d_in, int r, int baby_step, fa_buf* q_r,
                  void* ws, size_t ws_bytes, void* stream) {
  return project(c, q, w_pts, false, d_in, r, baby_step, q_r, ws, ws_bytes, stream);
}

int fa_project_ct_enc(fa_ctx* c, const fa_buf* q, const fa_buf* w_cts, int d_in, int r, int baby_step, fa_buf* q_r,
                      void* ws, size_t ws_bytes, void* stream) {
  return project(c, q, w_cts, true, d_in, r, baby_step, q_r, ws, ws_bytes, stream);
}

}  // extern "C"
