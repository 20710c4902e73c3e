// Internal declarations of libfa (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "fa.h"

// Per-prime constants on the device.  Residues live in doubles: every prime
// is below 2^50, so a residue (and any lazily reduced value below 2^53) is
// an exactly represented integer.
struct DevPrime {
  double q;      // the prime
  double qinv;   // fl(1/q)
  double ninv;   // N^-1 mod q
  double pinv;   // P^-1 mod q  (ciphertext primes only; 0 for special primes)
  double pmod;   // P mod q     (ciphertext primes only; 0 for special primes)
};

// Up to FA_MAXL limbs (polynomials over one prime) processed by one launch.
#define FA_MAXL 64
struct LimbList {
  int n;
  int prime[FA_MAXL];
  double* ptr[FA_MAXL];
};

struct fa_ctx {
  int logn, n, L, K, np, alpha, dnum, log_scale, device;
  std::vector<uint64_t> primes;   // [np] q_0..q_{L-1}, p_0..p_{K-1}
  std::vector<uint64_t> psi;      // chosen primitive 2N-th roots
  // device tables
  DevPrime* d_pr = nullptr;       // [np]
  double* d_tw_fwd = nullptr;     // [np][N]  psi^{brev(k)}
  double* d_tw_inv = nullptr;     // [np][N]  psi^{-brev(k)}
  double* d_mu_inv = nullptr;     // [dnum][alpha]       (D_i/d_j)^-1 mod d_j
  double* d_mu_hat = nullptr;     // [dnum][alpha][np]   (D_i/d_j) mod prime t
  double* d_md_inv = nullptr;     // [K]                 (P/p_k)^-1 mod p_k
  double* d_md_hat = nullptr;     // [K][L]              (P/p_k) mod q_t
  // secret (NTT form over every prime), keys
  double* d_s = nullptr;          // [np][N]
  std::map<int, double*> keys;    // step -> [dnum][2][np][N] (b, a), NTT form
  std::vector<uint64_t> p_mod_q;  // [L] P mod q_t (gadget)
  // phase timing (fa_profile)
  bool prof = false, prof_done = false;
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
};

// --------------------------------------------------------------------------
// launchers (fa_kernels.hip)
// --------------------------------------------------------------------------
namespace fa {

void ntt_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s);
void ntt_inv(const fa_ctx* c, const LimbList& l, hipStream_t s);

// Batched forward / inverse over `count` polynomials laid out as
// base + i * stride (words) whose prime index is prime_of(i) = i % period
// + prime_off.  Splits into launches of at most FA_MAXL limbs.
void ntt_fwd_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s);
void ntt_inv_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s);

// ModUp basis conversion for `batch` ciphertext c1's in coefficient form:
// src[b] = c1c + b * src_stride ([L][N]); dst[b] = ext + b * dst_stride
// ([dnum][np][N]); writes every (digit i, prime t not in digit i) limb.
void conv_modup(const fa_ctx* c, const double* c1c, size_t src_stride, double* ext, size_t dst_stride, int batch,
                hipStream_t s);
// ModDown basis conversion P -> Q for `count` polynomials:
// src[i] = up + i * src_stride points at the K special-prime limbs (coefficient
// form, [K][N]); dst[i] = out + i * dst_stride ([L][N]).
void conv_moddown(const fa_ctx* c, const double* up, size_t src_stride, double* out, size_t dst_stride, int count,
                  hipStream_t s);

// ext[b][i][t][k] = c1[b][t][k] for every ciphertext prime t of digit i = t / alpha
// (the digit's own limbs, copied in NTT form), b < batch.
void scatter_own(const fa_ctx* c, const double* c1, size_t src_stride, double* ext, size_t dst_stride, int batch,
                 hipStream_t s);
// Forward NTT of every limb (digit i, prime t not in digit i) of `batch`
// extended digit sets ext + b * stride ([dnum][np][N]).
void ntt_fwd_ext(const fa_ctx* c, double* ext, size_t stride, int batch, hipStream_t s);

// Key-switch inner product with the automorphism folded in:
// u[j] (+)= sum_i sigma_{g_j}(ext[j or 0]_i) * key_j[i]  over all np primes.
struct KsItem {
  const double* ext;  // [dnum][np][N]
  const double* key;  // [dnum][2][np][N]
  double* u;          // [2][np][N]
  uint32_t gal;       // Galois element
};
void ks_inner(const fa_ctx* c, const KsItem* items, int count, bool accumulate, hipStream_t s);

// out[h][t][k] = base_h[t][pi_g(k)] + (u[h][t][k] - conv[h][t][k]) * P^-1   (canonical)
// for h = 0, 1; base_h may be null (treated as 0).
struct FinishItem {
  const double* u;      // [2][np][N]
  const double* conv;   // [2][L][N]
  const double* base0;  // [L][N] or null
  const double* base1;  // [L][N] or null
  double* out;          // [2][L][N]
  uint32_t gal;         // permutation applied to base0/base1 (1 = none)
};
void moddown_finish(const fa_ctx* c, const FinishItem* items, int count, hipStream_t s);

// acc[blk][g][2][L][N] = sum_b pts[blk][(g*B+b)][L][N] * qrot[b][2][L][N]
void mac_diag(const fa_ctx* c, const double* qrot, const double* const* blocks, int n_blocks, int B, int G,
              double* acc, hipStream_t s);

// out[w] = ct * pt[w] (both polys), w < count
void mul_plain(const fa_ctx* c, const double* ct, const double* const* pts, int count, double* out, hipStream_t s);
// dst[i] = dst[i] + sigma_g(src[i]) over `words` words of [.][L][N] data; g = 1 -> plain add
void add_automorph(const fa_ctx* c, double* dst, const double* src, int n_polys, uint32_t gal, hipStream_t s);
// residues of signed integers: dst[p][t][k] = src[p][k] mod prime t (t < nprimes)
void int_to_res(const fa_ctx* c, const int64_t* src, int n_polys, int nprimes, double* dst, hipStream_t s);
// u64 residues (already < prime) -> words
void u64_to_res(const uint64_t* src, size_t words, double* dst, hipStream_t s);
void res_to_u64(const double* src, size_t words, uint64_t* dst, hipStream_t s);
// keygen combine: for each digit i and prime t:
//   b = -a*s + e + gad[i][t] * s[pi_g(k)]   (all NTT form); a in place already NTT
void keygen_combine(const fa_ctx* c, double* key, const double* e_ntt, uint32_t gal, hipStream_t s);
// encryption combine: c0[t] = -c1[t]*s[t] + v[t]
void enc_combine(const fa_ctx* c, double* ct, const double* v, hipStream_t s);
// decryption: out[t] = c0[t] + c1[t]*s[t]
void dec_combine(const fa_ctx* c, const double* ct, double* out, hipStream_t s);

}  // namespace fa
