// Internal declarations of libfa (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <map>
#include <mutex>
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

// Up to FA_MAXL limbs (polynomials over one prime) processed by one launch:
// 128 covers one batch of 16 rotations' special-prime products (96 limbs) or
// one block's giant accumulators at 12 primes in a single launch, and keeps
// the list (passed by value) inside the 4 KiB of kernel arguments.
#define FA_MAXL 128
// Each limb is transformed from src[i] into ptr[i] (src[i] == ptr[i]: in place);
// the inverse transform ends with a multiply by scale[i] (N^-1, possibly times a
// basis-conversion constant).
struct LimbList {
  int n;
  int prime[FA_MAXL];
  double* ptr[FA_MAXL];
  const double* src[FA_MAXL];
  double scale[FA_MAXL];
};
static_assert(sizeof(LimbList) <= 4096, "LimbList is a kernel argument");

#define FA_MAXAUX 3

struct fa_ctx {
  int logn, n, L, K, np, alpha, dnum, log_scale, device;
  // the fixed scratch array's address on this context's device (fa_rotate_static)
  void* static_scratch = nullptr;
  hipError_t static_scratch_err = hipSuccess;
  std::vector<uint64_t> primes;   // [np] q_0..q_{L-1}, p_0..p_{K-1}
  std::vector<uint64_t> psi;      // chosen primitive 2N-th roots
  // device tables
  DevPrime* d_pr = nullptr;       // [np]
  // twiddles (see the transform in fa_kernels.hip): psi^{brev(k)} for k < 256,
  // the 256-entry table T and the per-row factors F of the second pass, and
  // the same three for psi^-1
  double* d_twa_fwd = nullptr;    // [np][256]
  double* d_twa_inv = nullptr;
  double* d_twt_fwd = nullptr;    // [np][256]
  double* d_twt_inv = nullptr;
  double* d_twr_fwd = nullptr;    // [np][N/256][8]
  double* d_twr_inv = nullptr;
  double* d_mu_hat = nullptr;     // [dnum][alpha][np]   (D_i/d_j) mod prime t
  double* d_md_hat = nullptr;     // [K][L]              (P/p_k) mod q_t
  double* d_mu_scale = nullptr;   // [L] device copy of h_mu_scale
  double* d_md_scale = nullptr;   // [K] device copy of h_md_scale
  // host copies used to build per-limb constants
  std::vector<double> h_ninv;     // [np] N^-1 mod prime
  std::vector<double> h_mu_scale; // [L] N^-1 (D_i/q_t)^-1 mod q_t, t in digit i
  std::vector<double> h_md_scale; // [K] N^-1 (P/p_k)^-1 mod p_k
  // secret (NTT form over every prime), keys
  double* d_s = nullptr;          // [np][N]
  std::map<int, double*> keys;    // step -> [dnum][2][np][N] (b, a), NTT form
  double* d_rlk = nullptr;        // relinearisation key (s^2 -> s), same layout
  std::vector<uint64_t> p_mod_q;  // [L] P mod q_t (gadget)
  // phase timing (fa_profile)
  bool prof = false, prof_done = false;
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
  // auxiliary streams (default priority) that independent key-switch batches
  // run on, forked from and joined back to the caller's stream with events
  int n_aux = 0;
  hipStream_t aux[FA_MAXAUX] = {};
  hipEvent_t fork_ev = nullptr;
  hipEvent_t join_ev[FA_MAXAUX] = {};
  // side stream (default priority) of the membership scan: the threshold chain
  // runs there while the scores run on the caller's stream
  hipStream_t side = nullptr;
  hipEvent_t side_fork = nullptr, side_join = nullptr;
  // device staging of fa_decrypt / fa_export_coeffs (client and test side),
  // grown on demand and reused; the mutex serialises callers on other threads
  std::mutex export_mu;
  double* d_export = nullptr;     // [2][words]: coefficient transform, then u64 residues
  size_t export_words = 0;
};

// --------------------------------------------------------------------------
// launchers (fa_kernels.hip)
// --------------------------------------------------------------------------
namespace fa {

// device address of the library's fixed scratch array on `device` (current)
void* static_scratch(int device, hipError_t* err);
void ntt_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s);
void ntt_inv(const fa_ctx* c, const LimbList& l, hipStream_t s);
// the first (row) pass of the inverse transform alone, src -> ptr
void ntt_inv_b(const fa_ctx* c, const LimbList& l, hipStream_t s);

// Batched forward / inverse over `count` polynomials laid out as
// base + i * stride (words) whose prime index is prime_of(i) = i % period
// + prime_off.  Splits into launches of at most FA_MAXL limbs.
void ntt_fwd_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s);
void ntt_inv_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s);

// ModUp: for each item, ext[i][t] = NTT(Conv_{digit i -> t}(y)) for every digit
// i and prime t outside the digit, where y ([L][N]) is c1 after the first
// (row) pass of its inverse transform.  One kernel finishes the inverse
// (column pass and the scaling by N^-1 (D_i/q_t)^-1, canonical), converts and
// runs the first forward pass of every converted limb, so the coefficients
// never reach HBM.  Own-digit limbs of ext are not written: the key-switch
// kernels read them from c1.
#define FA_MAXMU 16
struct MuItem {
  const double* y;  // [L][N], row pass of the inverse transform done
  double* ext;      // [dnum][np][N]
};
// pass_b false: only the first forward pass (the giant-step kernel finishes it)
void modup_fused(const fa_ctx* c, const MuItem* items, int count, hipStream_t s, bool pass_b = true);

// ModDown with its finish: out = base[pi_gal] + (uQ - NTT(Conv_{P->Q}(yP))) * P^-1,
// where yP ([K][N]) holds the special-prime limbs of the key-switch product
// after the first (row) pass of their inverse transform.  One kernel finishes
// the inverse (column pass and the scaling by N^-1 (P/p_k)^-1, canonical),
// converts and runs the first forward pass of every target limb into conv
// (scratch); a second finishes the forward transform and the formula.
#define FA_MAXMD 32
struct MdItem {
  const double* yP;    // [K][N], row pass of the inverse done
  double* conv;        // [L][N] scratch
  const double* uQ;    // [L][N] NTT form
  const double* base;  // [L][N] or null
  double* out;         // [L][N]
  uint32_t gal;        // permutation of base (1 = none)
};
// pass_b false: conversion and first forward pass only (conv is left for moddown_ks)
void moddown_fused(const fa_ctx* c, const MdItem* items, int count, hipStream_t s, bool pass_b = true);

// ModDown finish of rotations whose key-switch sum on the ciphertext primes is
// formed in the same kernel (ks_inner then only covers the special primes):
// out = (sigma(c0) + (u_Q,0 - conv0^) P^-1, b1 + (u_Q,1 - conv1^) P^-1) with
// u_Q,h = sum_i sigma(ext_i) key[i][h] and conv (from moddown with pass_b false)
// holding the first pass of Conv_{P->Q} of both polynomials.
struct MdKsItem {
  const double* conv;  // [2][L][N]
  const double* ext;   // [dnum][np][N]
  const double* c1;    // [L][N] the digits' own limbs
  const double* key;   // [dnum][2][np][N]
  const double* c0;    // [L][N]
  const double* b1;    // [L][N] or null: added to the second output polynomial
  double* out;         // [2][L][N]
  uint32_t gal;
  uint32_t inv_gal;    // gal^-1 mod 2N (set by the launcher)
};
// nq > 1: the items come in groups of nq (g*nq .. g*nq+nq-1) sharing one key
// (the same rotation of nq queries); their workgroups run back to back on one
// XCD so the key words are read from HBM once per group.  count % nq == 0.
void moddown_ks(const fa_ctx* c, const MdKsItem* items, int count, hipStream_t s, int nq = 1);

// Key-switch inner product with the automorphism folded in:
// u[j] (+)= sum_i sigma_{g_j}(ext[j or 0]_i) * key_j[i]  over all np primes.
struct KsItem {
  const double* ext;  // [dnum][np][N]
  const double* c1;   // [L][N] NTT form: the digits' own limbs
  const double* key;  // [dnum][2][np][N]
  double* u;          // [2][np][N]
  const double* c0;   // [L][N] or null: adds P * sigma(c0) to u0 on the ciphertext primes
  uint32_t gal;       // Galois element
  uint32_t inv_gal;   // gal^-1 mod 2N (set by the launcher)
};
// t0 > 0: only primes t0..np-1 (the special primes when t0 = L)
// nq > 1: items grouped by key as for moddown_ks (count % nq == 0)
void ks_inner(const fa_ctx* c, const KsItem* items, int count, bool accumulate, hipStream_t s, int t0 = 0,
              int nq = 1);
// The special-prime part of ks_inner (no c0 term, not accumulated) fused with
// the first pass of its inverse transform: it.u's special limbs leave holding
// what k_ntt_inv_b would produce from ks_inner's output (ntt_inv_a finishes).
// One-digit contexts (dnum == 1) only; does nothing otherwise.
void ks_inv_b(const fa_ctx* c, const KsItem* items, int count, hipStream_t s, int nq = 1);

// Fused giant steps of nb blocks: u[blk] = sum_{g=1..ng} sum_i sigma_g(NTT(ext)_i) key_g[i]
// + P sigma_g(acc_g.c0), with ext = [nb][ng][dnum][np][N] holding only the first
// forward pass of the extended digits of acc_g.c1 (acc_g = acc + blk*astride + g*2LN).
void giant_ks(const fa_ctx* c, const double* ext, const double* acc, size_t astride, const double* const* keys,
              const uint32_t* gals, int nb, int ng, double* u, hipStream_t s);


// For each query j < nq: acc[j][blk][g][2][L][N] = sum_b pts[blk][(g*B+b)][L][N] * rot_b[2][L][N]
// with rot_0 = q[j] and rot_b = qrot[j][b-1] for b >= 1.  Up to FA_MAXQ queries
// share each pass over the plaintexts.
#define FA_MAXQ 4
void mac_diag(const fa_ctx* c, const double* const* q, const double* const* qrot, int nq,
              const double* const* blocks, int n_blocks, int B, int G, double* const* acc, hipStream_t s);

// Encrypted blocks: acc[pair][3][L][N] = sum_b ct[blk][(g*B+b)] (x) rot_b, the
// three components of the tensor product (rot_0 = q, rot_b = qrot[b-1]).
void mac_diag_ct(const fa_ctx* c, const double* q, const double* qrot, const double* const* blocks, int n_blocks,
                 int B, int G, double* acc, hipStream_t s);

// Rescale n_polys polynomials [n_polys][L][N] (NTT form) by the last prime:
// out [n_polys][L-1][N] = round(x / q_last); scratch: n_polys * L * N words.
void rescale(const fa_ctx* c, const double* ct, int n_polys, double* out, double* scratch, hipStream_t s);
// out [count][3][L][N]: tensors of count ciphertext pairs (NTT form); pair j reads
// x + j*sx and y + j*sy (words), each with xL / yL limbs per polynomial of which the
// first L are used (a ciphertext above this level is read as its drop)
void tensor(const fa_ctx* c, const double* x, int xL, size_t sx, const double* y, int yL, size_t sy, int count,
            double* out, hipStream_t s);
// element-wise over n_polys polynomials: mode 0 out = x * cst, 1 out = x with cst added to
// the even polynomials (the first of each ciphertext), 2 out = x + y, 3 out = x - y (cst
// given by its residues cres[L], or null); x has xL limbs per polynomial (0: L), its
// first L read
// (ciphertext j of a batch at x + j*sx, y + j*sy, out + j*so words; by default
// consecutive ciphertexts)
void ct_elem(const fa_ctx* c, const double* x, const double* y, double* out, int n_polys, const uint64_t* cres,
             int mode, hipStream_t s, int xL = 0, size_t sx = (size_t)-1, size_t sy = (size_t)-1,
             size_t so = (size_t)-1);
// tensors of count ciphertext pairs (x_j, y_j) given by pointer, each with its own
// limbs per polynomial (xL[j], yL[j]; the first L read); out [count][3][L][N]
void tensor_list(const fa_ctx* c, const double* const* xs, const int* xLs, const double* const* ys, const int* yLs,
                 int count, double* out, hipStream_t s);
// in place over count ciphertexts prod [count][2][L][N]: p_j <- 2 p_j - c_j T1 when
// odd[j], else 2 p_j + c_j on polynomial 0 (c_j given by its residues cres[j][L];
// T1 with t1L limbs per polynomial)
void cheb_fix(const fa_ctx* c, double* prod, int count, const double* t1, int t1L, const uint64_t* const* cres,
              const int* odd, hipStream_t s);
// out [2][L][N] = sum_i x_i * c_i + c0 on polynomial 0 (x_i canonical, xL[i] limbs per
// polynomial; c_i by residues cres[i][L]; c0 by residues or null)
void lincomb(const fa_ctx* c, double* out, const double* const* xs, const int* xLs, const uint64_t* const* cres,
             int nterm, const uint64_t* c0res, hipStream_t s);

// out[w] = ct * pt[w] (both polys), w < count
void mul_plain(const fa_ctx* c, const double* ct, const double* const* pts, int count, double* out, hipStream_t s);
// dst[r] += src[r] for n_limbs limbs of N words, limb r over prime r % period
void add_limbs(const fa_ctx* c, double* dst, const double* src, int n_limbs, int period, hipStream_t s);
// dst[i] = dst[i] + sigma_g(src[i]) over `words` words of [.][L][N] data; g = 1 -> plain add
void add_automorph(const fa_ctx* c, double* dst, const double* src, int n_polys, uint32_t gal, hipStream_t s);
// residues of signed integers: dst[p][t][k] = src[p][k] mod prime t (t < nprimes)
void int_to_res(const fa_ctx* c, const int64_t* src, int n_polys, int nprimes, double* dst, hipStream_t s);
// u64 residues (already < prime) -> words
void u64_to_res(const uint64_t* src, size_t words, double* dst, hipStream_t s);
void res_to_u64(const double* src, size_t words, uint64_t* dst, hipStream_t s);
// keygen combine: for each digit i and prime t:
//   b = -a*s + e + gad[i][t] * s[pi_g(k)]   (all NTT form); a in place already NTT
// gal = 0 selects the relinearisation key: s^2 in place of s[pi_g(k)]
void keygen_combine(const fa_ctx* c, double* key, const double* e_ntt, uint32_t gal, hipStream_t s);
// encryption combine: c0[t] = -c1[t]*s[t] + v[t]
void enc_combine(const fa_ctx* c, double* ct, const double* v, hipStream_t s);
// decryption: out[t] = c0[t] + c1[t]*s[t]
void dec_combine(const fa_ctx* c, const double* ct, double* out, hipStream_t s);

// Collects limbs for batched transforms; launches every FA_MAXL limbs and on flush.
struct LimbBatch {
  const fa_ctx* c;
  hipStream_t s;
  bool fwd, b_only;  // inverse: b_only the first (row) pass alone, src -> ptr
  LimbList l;
  LimbBatch(const fa_ctx* c_, hipStream_t s_, bool fwd_, bool b_only_ = false)
      : c(c_), s(s_), fwd(fwd_), b_only(b_only_) {
    l.n = 0;
  }
  // scale < 0: N^-1 of the prime
  void add(double* dst, int prime, const double* src = nullptr, double scale = -1.0) {
    l.ptr[l.n] = dst;
    l.src[l.n] = src ? src : dst;
    l.prime[l.n] = prime;
    l.scale[l.n] = scale < 0.0 ? c->h_ninv[prime] : scale;
    if (++l.n == FA_MAXL) flush();
  }
  void flush() {
    if (l.n) {
      if (fwd) ntt_fwd(c, l, s);
      else if (b_only) ntt_inv_b(c, l, s);
      else ntt_inv(c, l, s);
      l.n = 0;
    }
  }
  ~LimbBatch() { flush(); }
};

}  // namespace fa
