// HIP kernels of libfa for gfx950 (CDNA4, wave64).
//
// Residue arithmetic in float64.  Every prime q is in (2^49, 2^50); residues
// and lazily reduced values are integers of magnitude < 2^53 held exactly in
// doubles.  A modular product uses the FMA to split a*b exactly into
// h = fl(a*b) and l = a*b - h, estimates the quotient t = rint(a*b/q) from a
// precomputed 1/q (or w/q), and forms a*b - t*q = fma(-t, q, h) + l, which is
// exact because the true value is an integer below 2^53.  fp64 FMA issues at
// full rate on CDNA while 32-bit integer multiplies issue at quarter rate,
// which is why the residues are doubles and not u64.
//
// Bounds used below (u = 2^-53, all q in (2^49, 2^50)):
//   mulc(a, w, w/q):  for |a| <= c*q the quotient estimate is off by at most
//     0.375c, so |result| <= (0.5 + 0.375c) q; exact for |a| <= 8q.
//   mul(a, b):        |a|, |b| <= q  ->  |result| <= 0.75 q.
//   reduce(x):        |x| < 2^52    ->  |result| <= q/2 (+ rounding slack).
// Forward NTT values stay within 5.82 q (stages alternate lazy and reduced
// butterflies, see ct_bfly), inverse NTT values within 2 q; every transform
// output that leaves a kernel is either canonicalised or feeds a mulc / mul
// whose operand stays within 8 q.

#include <hip/hip_runtime.h>

#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "fa_internal.h"

namespace {

__device__ __forceinline__ double reduce(double x, double q, double qinv) {
  return __fma_rn(-rint(x * qinv), q, x);
}
__device__ __forceinline__ double mulc(double a, double w, double wp, double q) {
  const double h = a * w;
  const double l = __fma_rn(a, w, -h);
  const double t = rint(a * wp);
  return __fma_rn(-t, q, h) + l;
}
__device__ __forceinline__ double mul(double a, double b, double q, double qinv) {
  const double h = a * b;
  const double l = __fma_rn(a, b, -h);
  const double t = rint(h * qinv);
  return __fma_rn(-t, q, h) + l;
}
// x in (-q, 2q) -> [0, q)
__device__ __forceinline__ double canon(double x, double q) {
  x = x < 0.0 ? x + q : x;
  return x >= q ? x - q : x;
}
// full canonical reduction of |x| < 2^52
__device__ __forceinline__ double canon_full(double x, double q, double qinv) {
  x = reduce(x, q, qinv);
  return x < 0.0 ? x + q : x;
}

// Index permutation of the Galois automorphism X -> X^gal in NTT order:
// output slot i of the forward transform holds a(psi^(2 brev(i) + 1)), so
// sigma(a)^[i] = a^[pi(i)] with 2 brev(pi(i)) + 1 = gal (2 brev(i) + 1) mod 2N.
__device__ __forceinline__ uint32_t perm(uint32_t i, uint32_t gal, int logn) {
  const uint32_t e = 2u * (__brev(i) >> (32 - logn)) + 1u;
  const uint32_t e2 = (gal * e) & ((2u << logn) - 1u);
  return __brev((e2 - 1u) >> 1) >> (32 - logn);
}

// Cooley-Tukey butterfly (forward): (x, y) -> (x + w y, x - w y).  With R
// false x is not reduced first: the passes below reduce on odd stages only.
// With c the bound (in units of q) of the stage's inputs, a reduced stage
// leaves 1 + 0.375c and a lazy one 1.375c + 0.5; alternating from c <= 1 the
// bound settles at 2.45 after reduced and 3.87 after lazy stages, and two lazy
// stages in a row (an odd first pass meeting the next pass's stage 0) reach
// 5.82: always inside the 8q of mulc's exactness and below 2^53.
template <bool R = true>
__device__ __forceinline__ void ct_bfly(double& x, double& y, double w, double q, double qinv) {
  const double u = R ? reduce(x, q, qinv) : x;
  const double t = mulc(y, w, w * qinv, q);
  x = u + t;
  y = u - t;
}
// Gentleman-Sande butterfly (inverse): (x, y) -> (x + y, (x - y) w^-1)
__device__ __forceinline__ void gs_bfly(double& x, double& y, double winv, double q, double qinv) {
  const double u = x + y;
  const double v = x - y;
  x = reduce(u, q, qinv);
  y = mulc(v, winv, winv * qinv, q);
}

// ---------------------------------------------------------------------------
// Negacyclic NTT, N = 2^logn = 2^SA * 256, natural order in, bit-reversed out.
// Stage s pairs elements j and j + N/2^(s+1) with twiddle
//   w(s, j) = psi^brev(2^s + (j >> (logn - s)))       (brev over logn bits).
// Pass A runs stages 0..SA-1 on columns (j mod 256 fixed): its twiddles are
// the first 2^SA table entries.  Pass B runs stages SA..SA+7 on contiguous
// rows of 256; for row r and stage SA + s' the twiddle factors as
//   w = f[r][s'] * T[2^s' + i'],  f[r][s'] = psi^((2 brev_SA(r) + 1) 2^(7-s')),
//   T[2^s' + i'] = psi^(brev_s'(i') N / 2^s'),
// so pass B reads 8 row factors and a 256-entry table instead of N entries.
// Each pass keeps a unit of elements in registers for half its stages,
// exchanges through LDS, then finishes.
// ---------------------------------------------------------------------------
template <int SA>
struct PassA {
  static constexpr int H = 1 << SA;
  static constexpr int S1 = (SA + 1) / 2;
  static constexpr int S2 = SA - S1;
  static constexpr int E1 = 1 << S1;
  static constexpr int E2 = 1 << S2;
  static constexpr int COLS = (4096 >> SA) < 256 ? (4096 >> SA) : 256;
  static constexpr int TILE = COLS * H;
};

// loaders for the first pass of the forward transform
struct PlainLd {
  const double* src;
  __device__ double operator()(size_t i) const { return src[i]; }
};
template <int SA, class Ld>
__device__ __forceinline__ void fwd_a_body(const Ld& ld, double* a, const double* __restrict__ w, double q,
                                           double qinv, int col0, double* sm) {
  using P = PassA<SA>;
  for (int u = threadIdx.x; u < P::TILE / P::E1; u += 256) {
    const int c = u % P::COLS, hl = u / P::COLS;
    double x[P::E1];
#pragma unroll
    for (int m = 0; m < P::E1; ++m) x[m] = ld(((size_t)(hl + (m << P::S2)) << 8) + col0 + c);
#pragma unroll
    for (int s = 0; s < P::S1; ++s) {
      const int half = P::E1 >> (s + 1);
#pragma unroll
      for (int m = 0; m < P::E1; ++m) {
        if (m & half) continue;
        if (s & 1) ct_bfly<true>(x[m], x[m + half], w[(1 << s) + (m >> (P::S1 - s))], q, qinv);
        else ct_bfly<false>(x[m], x[m + half], w[(1 << s) + (m >> (P::S1 - s))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < P::E1; ++m) sm[(hl + (m << P::S2)) * P::COLS + c] = x[m];
  }
  __syncthreads();
  for (int u = threadIdx.x; u < P::TILE / P::E2; u += 256) {
    const int c = u % P::COLS, hh = u / P::COLS;
    double x[P::E2];
#pragma unroll
    for (int m = 0; m < P::E2; ++m) x[m] = sm[((hh << P::S2) + m) * P::COLS + c];
#pragma unroll
    for (int s2 = 0; s2 < P::S2; ++s2) {
      const int s = P::S1 + s2, half = P::E2 >> (s2 + 1);
#pragma unroll
      for (int m = 0; m < P::E2; ++m) {
        if (m & half) continue;
        if (s & 1) ct_bfly<true>(x[m], x[m + half], w[(1 << s) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
        else ct_bfly<false>(x[m], x[m + half], w[(1 << s) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < P::E2; ++m) a[((size_t)((hh << P::S2) + m) << 8) + col0 + c] = x[m];
  }
}

template <int SA>
__global__ __launch_bounds__(256) void k_ntt_fwd_a(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ twa) {
  using P = PassA<SA>;
  __shared__ double sm[P::TILE];
  const int pi = ll.prime[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  fwd_a_body<SA>(PlainLd{ll.src[blockIdx.y]}, ll.ptr[blockIdx.y], twa + (size_t)pi * 256, q, qinv,
                 blockIdx.x * P::COLS, sm);
}

// ModUp, first pass: ext[i][t] = pass A of Conv_{digit i -> t}(y), for every
// digit i and prime t outside the digit.
struct MuArgs {
  fa::MuItem it[FA_MAXMU];
};

// Fused basis conversion from row-passed sources: a workgroup owns one column
// tile of one source group (a digit of c1 for ModUp, the special primes for
// ModDown).  It finishes the inverse transform of the group's limbs on that
// tile (column pass, then the scaling by N^-1 times the conversion factor,
// leaving canonical residues, exactly as k_ntt_inv_a does) and keeps the
// results in registers; then for every target prime it forms the fast basis
// conversion of the tile (as ConvLd does) and runs the first forward pass on
// it (as fwd_a_body does).  Each source word is read once and the
// coefficients never leave the chip.  With ngrp > 1 the targets are split
// into ngrp contiguous groups, one per workgroup (each group repeats the
// inverse pass): small launches get more workgroups.
//
// Src describes the group: nl source limbs src(j) over primes sprime(j) with
// scales scale(j); ntarget targets, the k-th over prime target(k), with
// conversion factors hat(j, t), written to out(t).
template <int SA, int NS, class Src>
__device__ __forceinline__ void conv_fused_body(const Src& sr, const DevPrime* __restrict__ pr,
                                                const double* __restrict__ twa_f, const double* __restrict__ twa_i,
                                                int grp, int ngrp, double* sm) {
  using P = PassA<SA>;
  constexpr int NU = P::TILE / P::E1 / 256;   // tile units per thread in the E1 layout
  constexpr int NU2 = P::TILE / P::E2 / 256;  // ... in the E2 layout
  static_assert(NU * P::E1 * 256 == P::TILE && NU2 * P::E2 * 256 == P::TILE, "whole units per thread");
  const int nl = sr.nl;
  const int col0 = blockIdx.x * P::COLS;
  double y[NS][NU][P::E1];
#pragma unroll
  for (int j = 0; j < NS; ++j) {
    if (j < nl) {
      const int pj = sr.sprime(j);
      const double q = pr[pj].q, qinv = pr[pj].qinv;
      const double* __restrict__ w = twa_i + (size_t)pj * 256;
      const double* __restrict__ a = sr.src(j);
#pragma unroll
      for (int v = 0; v < NU2; ++v) {
        const int u = threadIdx.x + 256 * v;
        const int c = u % P::COLS, hh = u / P::COLS;
        double x[P::E2];
#pragma unroll
        for (int m = 0; m < P::E2; ++m) x[m] = a[((size_t)((hh << P::S2) + m) << 8) + col0 + c];
#pragma unroll
        for (int s2 = P::S2 - 1; s2 >= 0; --s2) {
          const int st = P::S1 + s2, half = P::E2 >> (s2 + 1);
#pragma unroll
          for (int m = 0; m < P::E2; ++m) {
            if (m & half) continue;
            gs_bfly(x[m], x[m + half], w[(1 << st) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
          }
        }
#pragma unroll
        for (int m = 0; m < P::E2; ++m) sm[((hh << P::S2) + m) * P::COLS + c] = x[m];
      }
      __syncthreads();
      const double sc = sr.scale(j), scp = sc * qinv;
#pragma unroll
      for (int v = 0; v < NU; ++v) {
        const int u = threadIdx.x + 256 * v;
        const int c = u % P::COLS, hl = u / P::COLS;
        double x[P::E1];
#pragma unroll
        for (int m = 0; m < P::E1; ++m) x[m] = sm[(hl + (m << P::S2)) * P::COLS + c];
#pragma unroll
        for (int st = P::S1 - 1; st >= 0; --st) {
          const int half = P::E1 >> (st + 1);
#pragma unroll
          for (int m = 0; m < P::E1; ++m) {
            if (m & half) continue;
            gs_bfly(x[m], x[m + half], w[(1 << st) + (m >> (P::S1 - st))], q, qinv);
          }
        }
#pragma unroll
        for (int m = 0; m < P::E1; ++m) y[j][v][m] = canon_full(mulc(x[m], sc, scp, q), q, qinv);
      }
      __syncthreads();  // the next limb reuses the LDS tile
    } else {
#pragma unroll
      for (int v = 0; v < NU; ++v)
#pragma unroll
        for (int m = 0; m < P::E1; ++m) y[j][v][m] = 0.0;
    }
  }
  const int per = (sr.ntarget + ngrp - 1) / ngrp;  // targets of this group: k0 <= k < k0 + per
  const int k0 = grp * per;
#pragma unroll 1
  for (int k = k0; k < k0 + per && k < sr.ntarget; ++k) {
    const int t = sr.target(k);
    const double q = pr[t].q, qinv = pr[t].qinv;
    double h[NS], hp[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      h[j] = j < nl ? sr.hat(j, t) : 0.0;
      hp[j] = h[j] * qinv;
    }
    const double* __restrict__ w = twa_f + (size_t)t * 256;
    double* __restrict__ a = sr.out(t);
#pragma unroll
    for (int v = 0; v < NU; ++v) {
      const int u = threadIdx.x + 256 * v;
      const int c = u % P::COLS, hl = u / P::COLS;
      double x[P::E1];
#pragma unroll
      for (int m = 0; m < P::E1; ++m) {
        double acc = 0.0;
#pragma unroll
        for (int j = 0; j < NS; ++j) acc += mulc(y[j][v][m], h[j], hp[j], q);
        x[m] = reduce(acc, q, qinv);
      }
#pragma unroll
      for (int st = 0; st < P::S1; ++st) {
        const int half = P::E1 >> (st + 1);
#pragma unroll
        for (int m = 0; m < P::E1; ++m) {
          if (m & half) continue;
          if (st & 1) ct_bfly<true>(x[m], x[m + half], w[(1 << st) + (m >> (P::S1 - st))], q, qinv);
          else ct_bfly<false>(x[m], x[m + half], w[(1 << st) + (m >> (P::S1 - st))], q, qinv);
        }
      }
#pragma unroll
      for (int m = 0; m < P::E1; ++m) sm[(hl + (m << P::S2)) * P::COLS + c] = x[m];
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < NU2; ++v) {
      const int u = threadIdx.x + 256 * v;
      const int c = u % P::COLS, hh = u / P::COLS;
      double x[P::E2];
#pragma unroll
      for (int m = 0; m < P::E2; ++m) x[m] = sm[((hh << P::S2) + m) * P::COLS + c];
#pragma unroll
      for (int s2 = 0; s2 < P::S2; ++s2) {
        const int st = P::S1 + s2, half = P::E2 >> (s2 + 1);
#pragma unroll
        for (int m = 0; m < P::E2; ++m) {
          if (m & half) continue;
          if (st & 1) ct_bfly<true>(x[m], x[m + half], w[(1 << st) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
          else ct_bfly<false>(x[m], x[m + half], w[(1 << st) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
        }
      }
#pragma unroll
      for (int m = 0; m < P::E2; ++m) a[((size_t)((hh << P::S2) + m) << 8) + col0 + c] = x[m];
    }
    __syncthreads();  // the next target reuses the LDS tile
  }
}

// ModUp sources: digit i of c1, converted to every prime outside the digit
// (own limbs are read from c1 directly by the key-switch kernels)
struct MuSrc {
  const double* y;     // [L][N], row pass of the inverse done
  double* ext;         // [dnum][np][N]
  const double* hatt;  // [dnum][alpha][np]
  const double* sct;   // [L]
  int i, alpha, lo, nl, n, np, ntarget;
  __device__ const double* src(int j) const { return y + (size_t)(lo + j) * n; }
  __device__ int sprime(int j) const { return lo + j; }
  __device__ double scale(int j) const { return sct[lo + j]; }
  __device__ int target(int k) const { return k < lo ? k : k + nl; }
  __device__ double hat(int j, int t) const { return hatt[((size_t)i * alpha + j) * np + t]; }
  __device__ double* out(int t) const { return ext + ((size_t)i * np + t) * n; }
};
// ModDown sources: the K special-prime limbs, converted to the L ciphertext primes
struct MdSrc {
  const double* yP;    // [K][N], row pass of the inverse done
  double* conv;        // [L][N]
  const double* hatt;  // [K][L]
  const double* sct;   // [K]
  int L, nl, n, ntarget;
  __device__ const double* src(int j) const { return yP + (size_t)j * n; }
  __device__ int sprime(int j) const { return L + j; }
  __device__ double scale(int j) const { return sct[j]; }
  __device__ int target(int k) const { return k; }
  __device__ double hat(int j, int t) const { return hatt[(size_t)j * L + t]; }
  __device__ double* out(int t) const { return conv + (size_t)t * n; }
};

template <int SA, int ALPHA>
__global__ __launch_bounds__(256) void k_modup_fused(MuArgs args, const DevPrime* __restrict__ pr,
                                                     const double* __restrict__ twa_f,
                                                     const double* __restrict__ twa_i,
                                                     const double* __restrict__ hat,
                                                     const double* __restrict__ scale, int logn, int L, int np,
                                                     int ngrp) {
  __shared__ double sm[PassA<SA>::TILE];
  const fa::MuItem& it = args.it[blockIdx.z];
  MuSrc sr;
  sr.y = it.y;
  sr.ext = it.ext;
  sr.hatt = hat;
  sr.sct = scale;
  sr.i = blockIdx.y / ngrp;
  sr.alpha = ALPHA;
  sr.lo = sr.i * ALPHA;
  sr.nl = L - sr.lo < ALPHA ? L - sr.lo : ALPHA;  // a short last digit has fewer limbs
  sr.n = 1 << logn;
  sr.np = np;
  sr.ntarget = np - sr.nl;
  conv_fused_body<SA, ALPHA>(sr, pr, twa_f, twa_i, blockIdx.y % ngrp, ngrp, sm);
}

// ModDown, first pass: conv[t] = pass A of Conv_{P -> q_t}(y_P).
struct MdArgs {
  fa::MdItem it[FA_MAXMD];
};

template <int SA, int KP>
__global__ __launch_bounds__(256, 2) void k_moddown_fused(MdArgs args, const DevPrime* __restrict__ pr,
                                                       const double* __restrict__ twa_f,
                                                       const double* __restrict__ twa_i,
                                                       const double* __restrict__ hat,
                                                       const double* __restrict__ scale, int logn, int L,
                                                       int ngrp) {
  __shared__ double sm[PassA<SA>::TILE];
  const fa::MdItem& it = args.it[blockIdx.z];
  MdSrc sr;
  sr.yP = it.yP;
  sr.conv = it.conv;
  sr.hatt = hat;
  sr.sct = scale;
  sr.L = L;
  sr.nl = KP;
  sr.n = 1 << logn;
  sr.ntarget = L;
  conv_fused_body<SA, KP>(sr, pr, twa_f, twa_i, blockIdx.y, ngrp, sm);
}

// inverse pass A (the last pass of the inverse transform): columns; the final
// multiply uses a per-limb constant (N^-1, or N^-1 times a basis-conversion
// factor) and leaves canonical residues.
template <int SA>
__global__ __launch_bounds__(256) void k_ntt_inv_a(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ twa) {
  using P = PassA<SA>;
  __shared__ double sm[P::TILE];
  const int pi = ll.prime[blockIdx.y];
  double* __restrict__ a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ w = twa + (size_t)pi * 256;
  const int col0 = blockIdx.x * P::COLS;
  for (int u = threadIdx.x; u < P::TILE / P::E2; u += 256) {
    const int c = u % P::COLS, hh = u / P::COLS;
    double x[P::E2];
#pragma unroll
    for (int m = 0; m < P::E2; ++m) x[m] = a[((size_t)((hh << P::S2) + m) << 8) + col0 + c];
#pragma unroll
    for (int s2 = P::S2 - 1; s2 >= 0; --s2) {
      const int s = P::S1 + s2, half = P::E2 >> (s2 + 1);
#pragma unroll
      for (int m = 0; m < P::E2; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], w[(1 << s) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < P::E2; ++m) sm[((hh << P::S2) + m) * P::COLS + c] = x[m];
  }
  __syncthreads();
  const double sc = ll.scale[blockIdx.y], scp = sc * qinv;
  for (int u = threadIdx.x; u < P::TILE / P::E1; u += 256) {
    const int c = u % P::COLS, hl = u / P::COLS;
    double x[P::E1];
#pragma unroll
    for (int m = 0; m < P::E1; ++m) x[m] = sm[(hl + (m << P::S2)) * P::COLS + c];
#pragma unroll
    for (int s = P::S1 - 1; s >= 0; --s) {
      const int half = P::E1 >> (s + 1);
#pragma unroll
      for (int m = 0; m < P::E1; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], w[(1 << s) + (m >> (P::S1 - s))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < P::E1; ++m)
      a[((size_t)(hl + (m << P::S2)) << 8) + col0 + c] = canon_full(mulc(x[m], sc, scp, q), q, qinv);
  }
}

// Pass B: rows of 256 contiguous elements.  Row stride in LDS is 272 words
// (one pad word per 16) so that both access patterns spread over all banks.
#define ROWW 272
__device__ __forceinline__ int lds_row(int rl, int lo) { return rl * ROWW + lo + (lo >> 4); }

// twiddle of pass B for stage SA+s', row r, index i' (see the header above)
__device__ __forceinline__ double twb(const double* __restrict__ T, double f, int s1, int i1, double q, double qinv) {
  const double t = T[(1 << s1) + i1];
  return mulc(t, f, f * qinv, q);
}

// stores for the last pass of the forward transform, one element at a time
// (global index i, lazily reduced value x); the pass hands them out so that
// consecutive threads touch consecutive words.
struct CanonSt {
  double* a;
  double q, qinv;
  __device__ void operator()(size_t i, double x) const { a[i] = canon_full(x, q, qinv); }
};
// ModDown finish: out[k] = base[pi(k)] + (u_Q[k] - conv^[k]) * P^-1
struct FinishSt {
  const double* uQ;
  const double* base;
  double* out;
  uint32_t gal;
  int logn;
  double q, qinv, pv, pvp;
  __device__ void operator()(size_t i, double x) const {
    double r = mulc(uQ[i] - x, pv, pvp, q);
    if (base) r += base[gal == 1u ? (uint32_t)i : perm((uint32_t)i, gal, logn)];
    out[i] = canon_full(r, q, qinv);
  }
};

// The eight stages of pass B over `rows` rows row0.. of a; the results are
// left in LDS (lds_row layout) and the block is synchronised on return.
__device__ __forceinline__ void fwd_b_lds(const double* __restrict__ a, int row0, int rows,
                                          const double* __restrict__ T, const double* __restrict__ F, double q,
                                          double qinv, double* sm) {
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int l0 = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) x[m] = a[(size_t)r * 256 + l0 + 16 * m];
#pragma unroll
    for (int s1 = 0; s1 < 4; ++s1) {
      const int half = 8 >> s1;
      const double f = F[r * 8 + s1];
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        if (s1 & 1) ct_bfly<true>(x[m], x[m + half], twb(T, f, s1, m >> (4 - s1), q, qinv), q, qinv);
        else ct_bfly<false>(x[m], x[m + half], twb(T, f, s1, m >> (4 - s1), q, qinv), q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) sm[lds_row(rl, l0 + 16 * m)] = x[m];
  }
  __syncthreads();
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int lh = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) x[m] = sm[lds_row(rl, 16 * lh + m)];
#pragma unroll
    for (int s1 = 4; s1 < 8; ++s1) {
      const int half = 8 >> (s1 - 4);
      const double f = F[r * 8 + s1];
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        const double w = twb(T, f, s1, (lh << (s1 - 4)) + (m >> (8 - s1)), q, qinv);
        if (s1 & 1) ct_bfly<true>(x[m], x[m + half], w, q, qinv);
        else ct_bfly<false>(x[m], x[m + half], w, q, qinv);
      }
    }
    // back to LDS: each thread rewrites the words it read
#pragma unroll
    for (int m = 0; m < 16; ++m) sm[lds_row(rl, 16 * lh + m)] = x[m];
  }
  __syncthreads();
}

template <class St>
__device__ __forceinline__ void fwd_b_body(double* a, const St& st, const double* __restrict__ T,
                                           const double* __restrict__ F, double q, double qinv, int logn,
                                           double* sm) {
  const int n = 1 << logn;
  const int rows = (n >> 8) < 16 ? (n >> 8) : 16;
  const int row0 = blockIdx.x * rows;
  fwd_b_lds(a, row0, rows, T, F, q, qinv, sm);
  // out with consecutive threads on consecutive words
  for (int e = threadIdx.x; e < rows * 256; e += 256) st((size_t)row0 * 256 + e, sm[lds_row(e >> 8, e & 255)]);
}

__global__ __launch_bounds__(256) void k_ntt_fwd_b(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ twt, const double* __restrict__ twr,
                                                   int logn) {
  __shared__ double sm[16 * ROWW];
  const int pi = ll.prime[blockIdx.y];
  double* a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const int H = 1 << (logn - 8);
  fwd_b_body(a, CanonSt{a, q, qinv}, twt + (size_t)pi * 256, twr + (size_t)pi * H * 8, q, qinv, logn, sm);
}

__global__ __launch_bounds__(256) void k_moddown_b(MdArgs args, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ twt, const double* __restrict__ twr,
                                                   int logn) {
  __shared__ double sm[16 * ROWW];
  const int t = blockIdx.y;
  const fa::MdItem& it = args.it[blockIdx.z];
  const int n = 1 << logn;
  const double q = pr[t].q, qinv = pr[t].qinv, pv = pr[t].pinv;
  const size_t o = (size_t)t * n;
  FinishSt st{it.uQ + o, it.base ? it.base + o : nullptr, it.out + o, it.gal, logn, q, qinv, pv, pv * qinv};
  const int H = 1 << (logn - 8);
  fwd_b_body(it.conv + o, st, twt + (size_t)t * 256, twr + (size_t)t * H * 8, q, qinv, logn, sm);
}

// ModDown finish of a rotation with its key-switch sum on the ciphertext
// primes formed in place: for limb t < L and the tile's words k,
//   u_h[k] = sum_i sigma(ext_i)[k] * key_i[h][t][k]   (h = 0, 1; own limbs from c1)
//   out0[k] = c0[pi(k)] + (u_0[k] - conv0^[k]) * P^-1,
//   out1[k] = b1[k] + (u_1[k] - conv1^[k]) * P^-1       (b1 = 0 for a rotation)
// where conv_h^ is the forward transform of Conv_{P->Q} finished here (pass B).
// The sums never reach HBM; both polynomials of the rotation share one gather.
struct MdKsArgs {
  fa::MdKsItem it[FA_MAXMD];
};

// Work item decode shared by the key-switch kernels: `rest` runs over (x, y,
// key group) with x fastest; the nq items of a key group (the same rotation
// for nq queries, items g*nq .. g*nq+nq-1) use the same key words.  With
// nq > 1 the ids are decoded so that those nq workgroups run one after the
// other on one XCD (ids 8 apart) and share the key words in its L2.  Returns
// false for the padding ids of the last group of eight.
__device__ __forceinline__ bool ks_decode(unsigned W, int nx, int ny, int nq, int ngroup, int& x, int& y, int& item) {
  unsigned rest = W, qi = 0;
  if (nq > 1) {
    const unsigned j8 = W >> 3;
    qi = j8 % (unsigned)nq;
    rest = (j8 / (unsigned)nq) * 8u + (W & 7u);
  }
  if (rest >= (unsigned)(nx * ny * ngroup)) return false;
  x = (int)(rest % (unsigned)nx);
  y = (int)((rest / (unsigned)nx) % (unsigned)ny);
  item = (int)(rest / (unsigned)(nx * ny)) * nq + (int)qi;
  return true;
}

// One query's key switches (nq == 1): ids decoded source-tile-major with the
// items fastest within an XCD, so the workgroups one XCD runs back to back (ids
// 8 apart) take the same source tile x of prime y for every rotation of the
// launch; the digits and c0 words of that tile, which every rotation gathers
// (through its own automorphism, into its own output tile), are read from HBM
// once and from that XCD's L2 after.  Returns false for the padding ids.
__device__ __forceinline__ bool ks_decode_src(unsigned W, int nx, int ny, int m, int& x, int& y, int& item) {
  const unsigned j8 = W >> 3;
  item = (int)(j8 % (unsigned)m);
  const unsigned rest = (j8 / (unsigned)m) * 8u + (W & 7u);
  if (rest >= (unsigned)(nx * ny)) return false;
  x = (int)(rest % (unsigned)nx);
  y = (int)(rest / (unsigned)nx);
  return true;
}

template <int DNUM, int ROWS, bool NT>
__global__ __launch_bounds__(256) void k_moddown_ks_b(MdKsArgs args, const DevPrime* __restrict__ pr,
                                                      const double* __restrict__ twt, const double* __restrict__ twr,
                                                      int logn, int L, int np, int alpha, int nq, int ngroup) {
  __shared__ double sm[ROWS * ROWW];
  const int n = 1 << logn;
  int tile, t, item;
  if (nq == 1) {
    int src;
    if (!ks_decode_src(blockIdx.x, (n >> 8) / ROWS, L, ngroup, src, t, item)) return;
    // the output tile whose automorphism image is the source tile
    tile = (int)(perm((uint32_t)src * (ROWS * 256u), args.it[item].inv_gal, logn) / (ROWS * 256u));
  } else if (!ks_decode(blockIdx.x, (n >> 8) / ROWS, L, nq, ngroup, tile, t, item)) {
    return;
  }
  const fa::MdKsItem& it = args.it[item];
  const int row0 = tile * ROWS;
  const uint32_t k0 = (uint32_t)row0 * 256u + threadIdx.x;  // this thread's words: k0 + 256 j, j < ROWS
  const double q = pr[t].q, qinv = pr[t].qinv, pv = pr[t].pinv, pvp = pv * qinv;
  const int own = t / alpha;
  const double* __restrict__ T = twt + (size_t)t * 256;
  const double* __restrict__ F = twr + (size_t)t * (n >> 8) * 8;
  const size_t o = (size_t)t * n;
  double u0[ROWS], u1[ROWS];
#pragma unroll
  for (int j = 0; j < ROWS; ++j) u0[j] = u1[j] = 0.0;
#pragma unroll 1
  for (int i = 0; i < DNUM; ++i) {
    const double* __restrict__ src = i == own ? it.c1 + o : it.ext + ((size_t)i * np + t) * n;
    const double* __restrict__ kb = it.key + (((size_t)i * 2 + 0) * np + t) * n + k0;
    const double* __restrict__ ka = it.key + (((size_t)i * 2 + 1) * np + t) * n + k0;
#pragma unroll
    for (int j = 0; j < ROWS; ++j) {
      const double x = src[perm(k0 + 256u * j, it.gal, logn)];
      // NT (one query): each key word is used once, so it streams past the
      // caches; several queries share it through L2 (see ks_decode)
      const double b = NT ? __builtin_nontemporal_load(kb + 256 * j) : kb[256 * j];
      const double a = NT ? __builtin_nontemporal_load(ka + 256 * j) : ka[256 * j];
      u0[j] += mul(x, b, q, qinv);
      u1[j] += mul(x, a, q, qinv);
    }
  }
#pragma unroll
  for (int j = 0; j < ROWS; ++j) {
    u0[j] = reduce(u0[j], q, qinv);
    u1[j] = reduce(u1[j], q, qinv);
  }
  fwd_b_lds(it.conv + o, row0, ROWS, T, F, q, qinv, sm);
#pragma unroll
  for (int j = 0; j < ROWS; ++j) {
    const int e = threadIdx.x + 256 * j;
    const double r = mulc(u0[j] - sm[lds_row(e >> 8, e & 255)], pv, pvp, q) + it.c0[o + perm(k0 + 256u * j, it.gal, logn)];
    __builtin_nontemporal_store(canon_full(r, q, qinv), it.out + o + k0 + 256 * j);
  }
  __syncthreads();
  fwd_b_lds(it.conv + (size_t)L * n + o, row0, ROWS, T, F, q, qinv, sm);
#pragma unroll
  for (int j = 0; j < ROWS; ++j) {
    const int e = threadIdx.x + 256 * j;
    double r = mulc(u1[j] - sm[lds_row(e >> 8, e & 255)], pv, pvp, q);
    if (it.b1) r += it.b1[o + k0 + 256 * j];
    __builtin_nontemporal_store(canon_full(r, q, qinv), it.out + (size_t)L * n + o + k0 + 256 * j);
  }
}

// inverse pass B (the first pass of the inverse transform), src -> ptr
__global__ __launch_bounds__(256) void k_ntt_inv_b(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ twt, const double* __restrict__ twr,
                                                   int logn) {
  __shared__ double sm[16 * ROWW];
  const int n = 1 << logn;
  const int rows = (n >> 8) < 16 ? (n >> 8) : 16;
  const int row0 = blockIdx.x * rows;
  const int pi = ll.prime[blockIdx.y];
  double* a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ T = twt + (size_t)pi * 256;
  const double* __restrict__ F = twr + (size_t)pi * (n >> 8) * 8;
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int lh = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
    const double2* src = reinterpret_cast<const double2*>(ll.src[blockIdx.y] + (size_t)r * 256 + 16 * lh);
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const double2 v = src[m];
      x[2 * m] = v.x;
      x[2 * m + 1] = v.y;
    }
#pragma unroll
    for (int s1 = 7; s1 >= 4; --s1) {
      const int half = 8 >> (s1 - 4);
      const double f = F[r * 8 + s1];
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], twb(T, f, s1, (lh << (s1 - 4)) + (m >> (8 - s1)), q, qinv), q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) sm[lds_row(rl, 16 * lh + m)] = x[m];
  }
  __syncthreads();
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int l0 = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) x[m] = sm[lds_row(rl, l0 + 16 * m)];
#pragma unroll
    for (int s1 = 3; s1 >= 0; --s1) {
      const int half = 8 >> s1;
      const double f = F[r * 8 + s1];
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], twb(T, f, s1, m >> (4 - s1), q, qinv), q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) a[(size_t)r * 256 + l0 + 16 * m] = x[m];
  }
}

// ---------------------------------------------------------------------------
// key-switch inner product with the automorphism folded into the read of the
// extended digits; a digit's own limbs are read from c1 itself
// ---------------------------------------------------------------------------
#define FA_MAXKS 32
struct KsArgs {
  fa::KsItem it[FA_MAXKS];
};

template <int DNUM>
__global__ __launch_bounds__(256) void k_ks_inner(KsArgs args, const DevPrime* __restrict__ pr, int logn, int L,
                                                  int np, int alpha, int accumulate, int t0, int nq, int ngroup) {
  const int n = 1 << logn;
  int kx, tr, item;
  if (nq == 1) {
    int src;
    if (!ks_decode_src(blockIdx.x, n / 256, np - t0, ngroup, src, tr, item)) return;
    kx = (int)(perm((uint32_t)src * 256u, args.it[item].inv_gal, logn) / 256u);  // see k_moddown_ks_b
  } else if (!ks_decode(blockIdx.x, n / 256, np - t0, nq, ngroup, kx, tr, item)) {
    return;
  }
  const int k = kx * 256 + threadIdx.x;
  const int t = t0 + tr;
  const fa::KsItem& it = args.it[item];
  const double q = pr[t].q, qinv = pr[t].qinv;
  const uint32_t kk = perm((uint32_t)k, it.gal, logn);
  const int own = t < L ? t / alpha : -1;
  double x[DNUM], kb[DNUM], ka[DNUM];
#pragma unroll
  for (int i = 0; i < DNUM; ++i) {
    const double* src = i == own ? it.c1 + (size_t)t * n : it.ext + ((size_t)i * np + t) * n;
    x[i] = src[kk];
    kb[i] = __builtin_nontemporal_load(it.key + (((size_t)i * 2 + 0) * np + t) * n + k);
    ka[i] = __builtin_nontemporal_load(it.key + (((size_t)i * 2 + 1) * np + t) * n + k);
  }
  double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
  for (int i = 0; i < DNUM; ++i) {
    acc0 += mul(x[i], kb[i], q, qinv);
    acc1 += mul(x[i], ka[i], q, qinv);
  }
  // P * sigma(c0) on the ciphertext primes: ModDown of the sum then returns
  // ModDown(sum u0) + sigma(c0) exactly, so the giant-step c0 terms ride along.
  if (it.c0 && t < L) acc0 += mul(it.c0[(size_t)t * n + kk], pr[t].pmod, q, qinv);
  double* u0 = it.u + (size_t)t * n + k;
  double* u1 = it.u + ((size_t)np + t) * n + k;
  if (accumulate) {
    acc0 += *u0;
    acc1 += *u1;
  }
  *u0 = canon_full(acc0, q, qinv);
  *u1 = canon_full(acc1, q, qinv);
}

// Key-switch sum on the special primes fused with the first pass of its
// inverse transform: for special prime t and the workgroup's rows,
//   u_h = sum_i sigma(ext_i) * key_i[h]   (h = 0, 1; canonical residues)
// formed word by word, then the eight stages of inverse pass B in registers
// and LDS, written to it.u in place of k_ks_inner's output after
// k_ntt_inv_b.  Sixteen threads per row, sixteen consecutive words each.
template <int DNUM>
__global__ __launch_bounds__(256) void k_ks_inv_b(KsArgs args, const DevPrime* __restrict__ pr,
                                                  const double* __restrict__ twt, const double* __restrict__ twr,
                                                  int logn, int L, int np, int nq, int ngroup) {
  __shared__ double sm[16 * ROWW];
  const int n = 1 << logn;
  const int rows = (n >> 8) < 16 ? (n >> 8) : 16;
  int tile, tr, item;
  if (nq == 1) {
    int src;
    if (!ks_decode_src(blockIdx.x, (n >> 8) / rows, np - L, ngroup, src, tr, item)) return;
    tile = (int)(perm((uint32_t)src * (uint32_t)(rows * 256), args.it[item].inv_gal, logn) / (uint32_t)(rows * 256));
  } else if (!ks_decode(blockIdx.x, (n >> 8) / rows, np - L, nq, ngroup, tile, tr, item)) {
    return;
  }
  const int t = L + tr;
  const fa::KsItem& it = args.it[item];
  const double q = pr[t].q, qinv = pr[t].qinv;
  const double* __restrict__ T = twt + (size_t)t * 256;
  const double* __restrict__ F = twr + (size_t)t * (n >> 8) * 8;
  const int u = threadIdx.x, lh = u & 15, rl = u >> 4, r = tile * rows + rl;
  const bool active = u < rows * 16;
  double y0[16], y1[16];
  if (active) {
    const uint32_t k0 = (uint32_t)r * 256u + 16u * lh;
#pragma unroll
    for (int m = 0; m < 16; ++m) y0[m] = y1[m] = 0.0;
#pragma unroll 1
    for (int i = 0; i < DNUM; ++i) {
      const double* __restrict__ src = it.ext + ((size_t)i * np + t) * n;
      const double2* kb = reinterpret_cast<const double2*>(it.key + (((size_t)i * 2 + 0) * np + t) * n + k0);
      const double2* ka = reinterpret_cast<const double2*>(it.key + (((size_t)i * 2 + 1) * np + t) * n + k0);
#pragma unroll
      for (int m2 = 0; m2 < 8; ++m2) {
        const double2 b = kb[m2], a = ka[m2];
        const double x0 = src[perm(k0 + 2u * m2, it.gal, logn)];
        const double x1 = src[perm(k0 + 2u * m2 + 1u, it.gal, logn)];
        y0[2 * m2] += mul(x0, b.x, q, qinv);
        y1[2 * m2] += mul(x0, a.x, q, qinv);
        y0[2 * m2 + 1] += mul(x1, b.y, q, qinv);
        y1[2 * m2 + 1] += mul(x1, a.y, q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      y0[m] = canon_full(y0[m], q, qinv);
      y1[m] = canon_full(y1[m], q, qinv);
    }
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    double x[16];
    if (active) {
#pragma unroll
      for (int m = 0; m < 16; ++m) x[m] = h == 0 ? y0[m] : y1[m];
#pragma unroll
      for (int s1 = 7; s1 >= 4; --s1) {
        const int half = 8 >> (s1 - 4);
        const double f = F[r * 8 + s1];
#pragma unroll
        for (int m = 0; m < 16; ++m) {
          if (m & half) continue;
          gs_bfly(x[m], x[m + half], twb(T, f, s1, (lh << (s1 - 4)) + (m >> (8 - s1)), q, qinv), q, qinv);
        }
      }
#pragma unroll
      for (int m = 0; m < 16; ++m) sm[lds_row(rl, 16 * lh + m)] = x[m];
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int m = 0; m < 16; ++m) x[m] = sm[lds_row(rl, lh + 16 * m)];
#pragma unroll
      for (int s1 = 3; s1 >= 0; --s1) {
        const int half = 8 >> s1;
        const double f = F[r * 8 + s1];
#pragma unroll
        for (int m = 0; m < 16; ++m) {
          if (m & half) continue;
          gs_bfly(x[m], x[m + half], twb(T, f, s1, m >> (4 - s1), q, qinv), q, qinv);
        }
      }
      double* out = it.u + ((size_t)h * np + t) * n + (size_t)r * 256;
#pragma unroll
      for (int m = 0; m < 16; ++m) out[lh + 16 * m] = x[m];
    }
    __syncthreads();  // the second polynomial reuses the LDS rows
  }
}

// ---------------------------------------------------------------------------
// Giant steps of the diagonal scoring, fused: for every block and every
// ciphertext/special prime t,
//   u[blk] = sum_{g=1}^{G-1} ( sum_i sigma_g(ext[blk][g]_i) * key_g[i]  +  P * sigma_g(acc_g.c0) )
// where ext holds the first forward pass only of the extended digits of
// acc_g.c1.  A workgroup owns one tile of rows*256 output words of one prime:
// for each (g, digit) it runs the last eight NTT stages on the source tile
// (the automorphism maps an aligned tile onto an aligned tile) in LDS, then
// gathers through the permutation and multiplies by the key, so the digits in
// NTT form never reach HBM.  The digit's own limbs come from acc_g.c1 itself.
// Workgroup ids are decoded so that the nb blocks of one (tile, prime) land on
// the same XCD one after the other and share the key rows in its L2.
// ---------------------------------------------------------------------------
#define FA_MAXG 32
struct GiantArgs {
  const double* ext;  // [nb][ng][dnum][np][N], first pass only
  const double* acc;  // acc of block blk, giant g: acc + blk * astride + g * 2 L N
  const double* key[FA_MAXG];
  uint32_t gal[FA_MAXG];
  double* u;          // [nb][2][np][N]
  size_t astride;
  int nb, ng, ngs, g0, accumulate;  // ng giants in this launch; ngs: the giant stride of ext
};

template <int DNUM, int ROWS>
__global__ __launch_bounds__(256) void k_giant_ks(GiantArgs a, const DevPrime* __restrict__ pr,
                                                  const double* __restrict__ twt, const double* __restrict__ twr,
                                                  int logn, int L, int np, int alpha, int ntile) {
  __shared__ double sm[ROWS * ROWW];
  const unsigned W = blockIdx.x;
  const unsigned j8 = W >> 3;
  const int blk = (int)(j8 % (unsigned)a.nb);
  const unsigned rest = (j8 / (unsigned)a.nb) * 8u + (W & 7u);
  if (rest >= (unsigned)(ntile * np)) return;
  const int t = (int)(rest / (unsigned)ntile), tile = (int)(rest % (unsigned)ntile);
  const int n = 1 << logn;
  constexpr uint32_t TW = ROWS * 256u;  // words of a tile; ROWS words per thread
  const uint32_t k0 = (uint32_t)tile * TW;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const double* __restrict__ T = twt + (size_t)t * 256;
  const double* __restrict__ F = twr + (size_t)t * (n >> 8) * 8;
  const int own = t < L ? t / alpha : -1;
  const size_t ln = (size_t)L * n;
  double acc0[ROWS], acc1[ROWS];
#pragma unroll
  for (int j = 0; j < ROWS; ++j) acc0[j] = acc1[j] = 0.0;
#pragma unroll 1
  for (int g = 0; g < a.ng; ++g) {
    const uint32_t gal = a.gal[g];
    const uint32_t sbase = perm(k0, gal, logn) & ~(TW - 1u);
    const double* __restrict__ accg = a.acc + (size_t)blk * a.astride + (size_t)(a.g0 + g) * 2 * ln;
    const double* __restrict__ key = a.key[g];
#pragma unroll 1
    for (int i = 0; i < DNUM; ++i) {
      // opaque copies: recomputing the permutation per digit is cheaper than
      // keeping it (and the twiddle loads) live across the loop
      uint32_t galv = gal;
      const double* Tv = T;
      asm volatile("" : "+s"(galv), "+s"(Tv));
      const double* __restrict__ kb = key + (((size_t)i * 2 + 0) * np + t) * n + k0 + threadIdx.x;
      const double* __restrict__ ka = key + (((size_t)i * 2 + 1) * np + t) * n + k0 + threadIdx.x;
      double x[ROWS];
      if (i == own) {
        const double* __restrict__ c1 = accg + ln + (size_t)t * n;
#pragma unroll
        for (int j = 0; j < ROWS; ++j) x[j] = c1[perm(k0 + threadIdx.x + 256u * j, galv, logn)];
      } else {
        const double* src = a.ext + ((((size_t)blk * a.ngs + g) * DNUM + i) * np + t) * n;
        fwd_b_lds(src, (int)(sbase >> 8), ROWS, Tv, F, q, qinv, sm);
#pragma unroll
        for (int j = 0; j < ROWS; ++j) {
          const uint32_t sk = perm(k0 + threadIdx.x + 256u * j, galv, logn) - sbase;
          x[j] = sm[lds_row((int)(sk >> 8), (int)(sk & 255u))];
        }
        __syncthreads();  // the next digit's pass reuses the LDS tile
      }
#pragma unroll
      for (int j = 0; j < ROWS; ++j) {
        acc0[j] += mul(x[j], kb[256 * j], q, qinv);
        acc1[j] += mul(x[j], ka[256 * j], q, qinv);
      }
    }
    if (t < L) {
      const double* __restrict__ c0 = accg + (size_t)t * n;
      const double pm = pr[t].pmod;
#pragma unroll
      for (int j = 0; j < ROWS; ++j) acc0[j] += mul(c0[perm(k0 + threadIdx.x + 256u * j, gal, logn)], pm, q, qinv);
    }
#pragma unroll
    for (int j = 0; j < ROWS; ++j) {
      acc0[j] = reduce(acc0[j], q, qinv);
      acc1[j] = reduce(acc1[j], q, qinv);
    }
  }
  double* u0 = a.u + ((size_t)blk * 2 * np + t) * n + k0 + threadIdx.x;
  double* u1 = u0 + (size_t)np * n;
#pragma unroll
  for (int j = 0; j < ROWS; ++j) {
    double r0 = acc0[j], r1 = acc1[j];
    if (a.accumulate) {
      r0 += u0[256 * j];
      r1 += u1[256 * j];
    }
    u0[256 * j] = canon_full(r0, q, qinv);
    u1[256 * j] = canon_full(r1, q, qinv);
  }
}

// ---------------------------------------------------------------------------
// diagonal-layout multiply-accumulate: the HBM stream of the scoring path
//   acc_j[pair][h][t][k] = sum_b pts[blk][g*B+b][t][k] * qrot_j[b][h][t][k]
// for NQ queries j at once, pair = (blk, g).  Each wave owns 64 consecutive
// coefficients and keeps NACC pairs x NQ queries x 2 accumulators in
// registers; every plaintext word is read once per group of NQ queries.
//
// The operands of a step (NACC plaintext words and each query's two rotated
// words per coefficient) travel HBM -> LDS with direct-to-LDS loads into a
// ring of S per-wave slots: while step b is multiplied out of LDS, steps
// b+1..b+S-1 are in flight, and they occupy no registers.  A wave only reads
// its own slots, so the vector-memory counter (loads complete in order) is
// the only synchronisation: before step b, wait until at most the loads of
// the later steps are outstanding.  A reduction every 8 products keeps the
// lazy sums below 2^53.
//
// With several chunks of NACC pairs in one launch, workgroup ids are decoded
// so that the chunks of one coefficient tile run on one XCD back to back and
// read the rotated queries from that XCD's L2 after the first.
// ---------------------------------------------------------------------------
#define FA_MAXBLK 32
struct MacArgs {
  const double* q0[FA_MAXQ];    // per query: rotation 0 (the query itself)
  const double* qrot[FA_MAXQ];  // per query: rotations 1..B-1, [B-1][2][L][N]
  double* acc[FA_MAXQ];         // per query: [n_pairs][2][L][N]
  const double* blk[FA_MAXBLK];
  int n_pairs, pair0, B, logG, L;
  int nchunk, ntile;            // chunks of NACC pairs from pair0; tiles of 256 words
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_void_t;

// s_waitcnt immediate (gfx9 encoding): wait until at most n vector-memory
// operations are outstanding; the LDS and export counters are not waited on
#define FA_VMCNT(n) (0x0F70 | ((n) & 15) | (((n) >> 4) << 14))
#define FA_LGKMCNT0 0xC07F

template <int NQ, int NACC, int S>
__global__ __launch_bounds__(256) void k_mac_diag(MacArgs args, const DevPrime* __restrict__ pr, int logn) {
  constexpr int ROWS = NACC + 2 * NQ;    // 64-word rows of one step: plaintexts, then x0/x1 per query
  constexpr int GL = NACC / 2 + NQ;      // loads issued per step
  static_assert(S == 2 || S == 3, "ring of two or three slots");
  static_assert((S - 1) * GL <= 63, "vector-memory counter range");
  __shared__ double slab[4][S][ROWS][64];
  unsigned tile = blockIdx.x, chunk = 0;
  if (args.nchunk > 1) {
    const unsigned j = blockIdx.x >> 3;
    chunk = j % (unsigned)args.nchunk;
    tile = (j / (unsigned)args.nchunk) * 8u + (blockIdx.x & 7u);
    if (tile >= (unsigned)args.ntile) return;
  }
  const int n = 1 << logn;
  const size_t ln = (size_t)args.L * n;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const size_t c0 = (size_t)tile * 256 + (size_t)w * 64;  // first coefficient of this wave
  const size_t f = c0 + lane;
  const int t = (int)(c0 >> logn);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const int pair0 = args.pair0 + (int)chunk * NACC;
  const int last = args.n_pairs - 1;
  const int G = 1 << args.logG;
  const int B = args.B;
  const int hp = lane >> 5;                         // which of the two rows a lane's 16 bytes land in
  const size_t lo = c0 + 2 * (size_t)(lane & 31);   // its two coefficients
  // per-lane source of each load at step 0 (step b adds b * ln words): lanes
  // 0-31 read pair 2i, lanes 32-63 pair 2i+1 (pairs past the end re-read the
  // last pair, in bounds, and are never stored); the queries' x0 / x1 rows
  const double* src[NACC / 2];
#pragma unroll
  for (int i = 0; i < NACC / 2; ++i) {
    const int pa = min(pair0 + 2 * i, last), pb = min(pair0 + 2 * i + 1, last);
    const double* xa = args.blk[pa >> args.logG] + (size_t)((pa & (G - 1)) * B) * ln;
    const double* xb = args.blk[pb >> args.logG] + (size_t)((pb & (G - 1)) * B) * ln;
    src[i] = (hp ? xb : xa) + lo;
  }
  const double* qs0[NQ];
  const double* qsr[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    qs0[j] = args.q0[j] + (size_t)hp * ln + lo;
    qsr[j] = args.qrot[j] + (size_t)hp * ln + lo;
  }
  // one step's loads into slot sl: row 2i gets pair 2i, row 2i+1 pair 2i+1
  auto issue = [&](int sl, int b) {
#pragma unroll
    for (int i = 0; i < NACC / 2; ++i)
      __builtin_amdgcn_global_load_lds((gbl_void_t*)(src[i] + (size_t)b * ln), (lds_void_t*)&slab[w][sl][2 * i][0],
                                       16, 0, 0);
#pragma unroll
    for (int j = 0; j < NQ; ++j)
      __builtin_amdgcn_global_load_lds((gbl_void_t*)(b == 0 ? qs0[j] : qsr[j] + (size_t)(b - 1) * 2 * ln),
                                       (lds_void_t*)&slab[w][sl][NACC + 2 * j][0], 16, 0, 0);
  };
  double* accp[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) accp[j] = args.acc[j];
  const int cnt = min(NACC, args.n_pairs - pair0);
  double a0[NQ][NACC], a1[NQ][NACC];
#pragma unroll
  for (int j = 0; j < NQ; ++j)
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      a0[j][i] = 0.0;
      a1[j][i] = 0.0;
    }
#pragma unroll
  for (int sl = 0; sl < S; ++sl)
    if (sl < B) issue(sl, sl);
  // one step out of slot SL (a compile-time slot index lets the compiler's
  // tracking of pending direct-to-LDS loads tell the slots apart)
  auto step = [&](auto slc, int b) {
    constexpr int SL = decltype(slc)::value;
    // steps b+1 .. min(b+S-1, B-1) were issued after step b
    const int later = min(S - 1, B - 1 - b);
    __builtin_amdgcn_sched_barrier(0);
    if (later >= 2) __builtin_amdgcn_s_waitcnt(FA_VMCNT(2 * GL));
    else if (later == 1) __builtin_amdgcn_s_waitcnt(FA_VMCNT(GL));
    else __builtin_amdgcn_s_waitcnt(FA_VMCNT(0));
    __builtin_amdgcn_sched_barrier(0);
    double x0[NQ], x1[NQ], x0p[NQ], x1p[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      x0[j] = slab[w][SL][NACC + 2 * j][lane];
      x1[j] = slab[w][SL][NACC + 2 * j + 1][lane];
      x0p[j] = x0[j] * qinv;
      x1p[j] = x1[j] * qinv;
    }
#pragma unroll
    for (int i0 = 0; i0 < NACC; i0 += 8) {
      double p[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] = slab[w][SL][i0 + i][lane];
#pragma unroll
      for (int j = 0; j < NQ; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          a0[j][i0 + i] += mulc(p[i], x0[j], x0p[j], q);
          a1[j][i0 + i] += mulc(p[i], x1[j], x1p[j], q);
        }
    }
    if ((b & 7) == 7) {
#pragma unroll
      for (int j = 0; j < NQ; ++j)
#pragma unroll
        for (int i = 0; i < NACC; ++i) {
          a0[j][i] = reduce(a0[j][i], q, qinv);
          a1[j][i] = reduce(a1[j][i], q, qinv);
        }
    }
    // the slot is read out: refill it with step b+S
    __builtin_amdgcn_s_waitcnt(FA_LGKMCNT0);
    __builtin_amdgcn_sched_barrier(0);
    if (b + S < B) issue(SL, b + S);
  };
  for (int b0 = 0; b0 < B; b0 += S) {
    step(std::integral_constant<int, 0>{}, b0);
    if (b0 + 1 < B) step(std::integral_constant<int, 1>{}, b0 + 1);
    if constexpr (S > 2)
      if (b0 + 2 < B) step(std::integral_constant<int, 2>{}, b0 + 2);
  }
#pragma unroll
  for (int j = 0; j < NQ; ++j)
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      if (i < cnt) {
        double* o = accp[j] + (size_t)(pair0 + i) * 2 * ln + f;
        o[0] = canon_full(a0[j][i], q, qinv);
        o[ln] = canon_full(a1[j][i], q, qinv);
      }
    }
}

// One query, NACC pairs: the same product with three steps in flight per wave.
// Steps cycle through two LDS slots (direct-to-LDS loads of the NACC plaintext
// rows, the rotated query in registers) and one register stage (the NACC
// plaintext words and the rotated query loaded straight into registers), so a
// wave holds the loads of three steps while it multiplies one.  The LDS
// slots are synchronised by the vector-memory counter as in k_mac_diag (a
// slot's wait counts the loads issued after it); the register stage is waited
// on by the compiler.  Reductions every 6 steps (lazy sums below 6q + q/2).
template <int NACC>
__global__ __launch_bounds__(256) void k_mac_diag3(MacArgs args, const DevPrime* __restrict__ pr, int logn) {
  constexpr int ROWS = NACC + 2;    // an LDS step: the plaintext rows, then the rotated query's x0 / x1
  constexpr int GL = NACC / 2 + 1;  // vector-memory operations of an LDS step
  constexpr int GR = NACC + 2;      // of a register step
  static_assert(GL + GR <= 63, "vector-memory counter range");
  __shared__ double slab[4][2][ROWS][64];
  unsigned tile = blockIdx.x, chunk = 0;
  if (args.nchunk > 1) {
    const unsigned j = blockIdx.x >> 3;
    chunk = j % (unsigned)args.nchunk;
    tile = (j / (unsigned)args.nchunk) * 8u + (blockIdx.x & 7u);
    if (tile >= (unsigned)args.ntile) return;
  }
  const int n = 1 << logn;
  const size_t ln = (size_t)args.L * n;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const size_t c0 = (size_t)tile * 256 + (size_t)w * 64;
  const size_t f = c0 + lane;
  const int t = (int)(c0 >> logn);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const int pair0 = args.pair0 + (int)chunk * NACC;
  const int last = args.n_pairs - 1;
  const int G = 1 << args.logG;
  const int B = args.B;
  const int hp = lane >> 5;
  const size_t lo = c0 + 2 * (size_t)(lane & 31);
  // plaintext row of pair i at step 0 (pairs past the end re-read the last pair)
  auto row = [&](int i) -> const double* {
    const int pa = min(pair0 + i, last);
    return args.blk[pa >> args.logG] + (size_t)((pa & (G - 1)) * B) * ln;
  };
  const double* src[NACC / 2];  // direct-to-LDS source of load i (pairs 2i, 2i+1)
#pragma unroll
  for (int i = 0; i < NACC / 2; ++i) src[i] = (hp ? row(2 * i + 1) : row(2 * i)) + lo;
  const double* qd0 = args.q0[0] + (size_t)hp * ln + lo;    // direct-to-LDS: x0 row (lanes 0-31), x1 row
  const double* qdr = args.qrot[0] + (size_t)hp * ln + lo;
  const double* qv0 = args.q0[0] + f;                       // into registers
  const double* qvr = args.qrot[0] + f;
  double a0[NACC], a1[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    a0[i] = 0.0;
    a1[i] = 0.0;
  }
  auto dma = [&](auto slc, int b) {
    constexpr int SL = decltype(slc)::value;
#pragma unroll
    for (int i = 0; i < NACC / 2; ++i)
      __builtin_amdgcn_global_load_lds((gbl_void_t*)(src[i] + (size_t)b * ln), (lds_void_t*)&slab[w][SL][2 * i][0],
                                       16, 0, 0);
    __builtin_amdgcn_global_load_lds((gbl_void_t*)(b == 0 ? qd0 : qdr + (size_t)(b - 1) * 2 * ln),
                                     (lds_void_t*)&slab[w][SL][NACC][0], 16, 0, 0);
  };
  double pv[NACC], xr0, xr1;
  auto rld = [&](int b) {
#pragma unroll
    for (int i = 0; i < NACC; ++i) pv[i] = __builtin_nontemporal_load(row(i) + (size_t)b * ln + f);
    const double* x = b == 0 ? qv0 : qvr + (size_t)(b - 1) * 2 * ln;
    xr0 = x[0];
    xr1 = x[ln];
  };
  auto mac_lds = [&](auto slc) {
    constexpr int SL = decltype(slc)::value;
    const double x0 = slab[w][SL][NACC][lane], x1 = slab[w][SL][NACC + 1][lane];
    const double x0p = x0 * qinv, x1p = x1 * qinv;
#pragma unroll
    for (int c = 0; c < NACC; c += 8) {
      double pc[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) pc[i] = slab[w][SL][c + i][lane];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a0[c + i] += mulc(pc[i], x0, x0p, q);
        a1[c + i] += mulc(pc[i], x1, x1p, q);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  dma(S0{}, 0);
  if (B > 1) dma(S1{}, 1);
  if (B > 2) rld(2);
  int red = 0;
  for (int b = 0; b < B; b += 3) {
    // step b out of slot 0: issued after its loads are slot 1's step (if any)
    // and the register step (if any), in that order
    __builtin_amdgcn_sched_barrier(0);
    if (b + 2 < B) __builtin_amdgcn_s_waitcnt(FA_VMCNT(GL + GR));
    else if (b + 1 < B) __builtin_amdgcn_s_waitcnt(FA_VMCNT(GL));
    else __builtin_amdgcn_s_waitcnt(FA_VMCNT(0));
    __builtin_amdgcn_sched_barrier(0);
    mac_lds(S0{});
    __builtin_amdgcn_s_waitcnt(FA_LGKMCNT0);
    __builtin_amdgcn_sched_barrier(0);
    const bool n0 = b + 3 < B, n1 = b + 4 < B, n2 = b + 5 < B;
    if (n0) dma(S0{}, b + 3);
    if (b + 1 < B) {
      // step b+1 out of slot 1: issued after it are the register step (when
      // b+2 < B) and slot 0's refill (when b+3 < B)
      __builtin_amdgcn_sched_barrier(0);
      if (n0) __builtin_amdgcn_s_waitcnt(FA_VMCNT(GR + GL));
      else if (b + 2 < B) __builtin_amdgcn_s_waitcnt(FA_VMCNT(GR));
      else __builtin_amdgcn_s_waitcnt(FA_VMCNT(0));
      __builtin_amdgcn_sched_barrier(0);
      mac_lds(S1{});
      __builtin_amdgcn_s_waitcnt(FA_LGKMCNT0);
      __builtin_amdgcn_sched_barrier(0);
      if (n1) dma(S1{}, b + 4);
    }
    if (b + 2 < B) {
      // step b+2 out of registers (the compiler waits for them)
      const double x0p = xr0 * qinv, x1p = xr1 * qinv;
#pragma unroll
      for (int i = 0; i < NACC; ++i) {
        a0[i] += mulc(pv[i], xr0, x0p, q);
        a1[i] += mulc(pv[i], xr1, x1p, q);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (n2) rld(b + 5);
    }
    if (++red == 2) {
      red = 0;
#pragma unroll
      for (int i = 0; i < NACC; ++i) {
        a0[i] = reduce(a0[i], q, qinv);
        a1[i] = reduce(a1[i], q, qinv);
      }
    }
  }
  const int cnt = min(NACC, args.n_pairs - pair0);
  double* accp = args.acc[0];
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    if (i < cnt) {
      double* o = accp + (size_t)(pair0 + i) * 2 * ln + f;
      o[0] = canon_full(a0[i], q, qinv);
      o[ln] = canon_full(a1[i], q, qinv);
    }
  }
}

// ---------------------------------------------------------------------------
// multiply-accumulate against an encrypted block (ct x ct, three components)
//   acc[pair][0] += c0 q0,  acc[pair][1] += c0 q1 + c1 q0,  acc[pair][2] += c1 q1
// with (c0, c1) = ct[blk][g*B+b] and (q0, q1) = rot_b.  One thread per
// coefficient, NACC pairs per chunk; several chunks in one launch share the
// rotated query through one XCD's L2 as in k_mac_diag.  A reduction every 4
// steps keeps the lazy sums below 2^53 (the middle component gains two
// products per step).
// ---------------------------------------------------------------------------
struct MacCtArgs {
  const double* q0;
  const double* qrot;
  double* acc;  // [n_pairs][3][L][N]
  const double* blk[FA_MAXBLK];
  int n_pairs, pair0, B, logG, L;
  int nchunk, ntile;
};

template <int NACC>
__global__ __launch_bounds__(256) void k_mac_diag_ct(MacCtArgs args, const DevPrime* __restrict__ pr, int logn) {
  unsigned tile = blockIdx.x, chunk = 0;
  if (args.nchunk > 1) {
    const unsigned j = blockIdx.x >> 3;
    chunk = j % (unsigned)args.nchunk;
    tile = (j / (unsigned)args.nchunk) * 8u + (blockIdx.x & 7u);
    if (tile >= (unsigned)args.ntile) return;
  }
  const int n = 1 << logn;
  const size_t ln = (size_t)args.L * n;
  const size_t f = (size_t)tile * 256 + threadIdx.x;
  const int t = (int)(f >> logn);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const int pair0 = args.pair0 + (int)chunk * NACC;
  const int last = args.n_pairs - 1;
  const int G = 1 << args.logG;
  const double* src[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    const int pair = min(pair0 + i, last);
    src[i] = args.blk[pair >> args.logG] + (size_t)((pair & (G - 1)) * args.B) * 2 * ln + f;
  }
  double a0[NACC], a1[NACC], a2[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) a0[i] = a1[i] = a2[i] = 0.0;
  for (int b = 0; b < args.B; ++b) {
    const double* __restrict__ qb = b == 0 ? args.q0 : args.qrot + (size_t)(b - 1) * 2 * ln;
    const double x0 = qb[f], x1 = qb[ln + f];
    double p0[NACC], p1[NACC];
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      p0[i] = __builtin_nontemporal_load(src[i] + (size_t)b * 2 * ln);
      p1[i] = __builtin_nontemporal_load(src[i] + (size_t)b * 2 * ln + ln);
    }
    const double x0p = x0 * qinv, x1p = x1 * qinv;
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      a0[i] += mulc(p0[i], x0, x0p, q);
      a1[i] += mulc(p0[i], x1, x1p, q) + mulc(p1[i], x0, x0p, q);
      a2[i] += mulc(p1[i], x1, x1p, q);
    }
    if ((b & 3) == 3) {
#pragma unroll
      for (int i = 0; i < NACC; ++i) {
        a0[i] = reduce(a0[i], q, qinv);
        a1[i] = reduce(a1[i], q, qinv);
        a2[i] = reduce(a2[i], q, qinv);
      }
    }
  }
  const int cnt = min(NACC, args.n_pairs - pair0);
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    if (i < cnt) {
      double* o = args.acc + (size_t)(pair0 + i) * 3 * ln + f;
      o[0] = canon_full(a0[i], q, qinv);
      o[ln] = canon_full(a1[i], q, qinv);
      o[2 * ln] = canon_full(a2[i], q, qinv);
    }
  }
}

// ---------------------------------------------------------------------------
// small element-wise kernels
// ---------------------------------------------------------------------------
#define FA_MAXPT 32
struct PtArgs {
  const double* pt[FA_MAXPT];
};

__global__ __launch_bounds__(256) void k_mul_plain(const double* __restrict__ ct, PtArgs pts, double* out,
                                                   const DevPrime* __restrict__ pr, int logn, int L) {
  const int n = 1 << logn;
  const size_t ln = (size_t)L * n;
  const size_t f = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int w = blockIdx.y;
  const int t = (int)(f >> logn);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const double p = pts.pt[w][f];
  double* o = out + (size_t)w * 2 * ln;
  o[f] = canon(mul(ct[f], p, q, qinv), q);
  o[ln + f] = canon(mul(ct[ln + f], p, q, qinv), q);
}

__global__ __launch_bounds__(256) void k_add_automorph(double* __restrict__ dst, const double* __restrict__ src,
                                                       const DevPrime* __restrict__ pr, int logn, int L,
                                                       uint32_t gal) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int row = blockIdx.y;  // poly * L + t
  const int t = row % L;
  const double q = pr[t].q;
  const uint32_t kk = gal == 1u ? (uint32_t)k : perm((uint32_t)k, gal, logn);
  const size_t o = (size_t)row * n;
  dst[o + k] = canon(dst[o + k] + src[o + kk], q);
}

__global__ __launch_bounds__(256) void k_add_limbs(double* __restrict__ dst, const double* __restrict__ src,
                                                   const DevPrime* __restrict__ pr, int logn, int period) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int row = blockIdx.y;
  const double q = pr[row % period].q;
  const size_t o = (size_t)row * n + k;
  dst[o] = canon(dst[o] + src[o], q);
}

// --- the membership path: rescale, ct x ct tensor, constants -------------
// Rescale, lift: lift[h][t][k] = the centred value of last[h][k] (residues of
// the last prime, coefficient form, canonical) reduced mod q_t, t < L-1.
#define FA_MAXLIMB 16
struct ResArgs {
  double c[FA_MAXLIMB];   // per limb: q_last^-1 mod q_t (rescale) or a constant mod q_t
  double cp[FA_MAXLIMB];  // c * (1/q_t)
};
#define FA_MAXTERM 8
struct TensorList {
  const double* x[FA_MAXTERM];
  const double* y[FA_MAXTERM];
  int xL[FA_MAXTERM], yL[FA_MAXTERM];
};
struct ChebFixArgs {
  double c[FA_MAXTERM][FA_MAXLIMB];
  double cp[FA_MAXTERM][FA_MAXLIMB];
  int odd[FA_MAXTERM];
};
struct LinArgs {
  const double* x[FA_MAXTERM];
  int xL[FA_MAXTERM];
  double c[FA_MAXTERM][FA_MAXLIMB];
  double cp[FA_MAXTERM][FA_MAXLIMB];
  double c0[FA_MAXLIMB];
  int nterm, accumulate;
};
__global__ __launch_bounds__(256) void k_rescale_lift(const double* __restrict__ last, double* __restrict__ lift,
                                                      const DevPrime* __restrict__ pr, int logn, int Lm1,
                                                      double ql) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, h = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  double v = last[(size_t)h * n + k];
  if (v > 0.5 * (ql - 1.0)) v -= ql;  // centred, |v| < q_last / 2, exact
  lift[((size_t)h * Lm1 + t) * n + k] = canon_full(v, q, qinv);
}
// out[h][t] = (c[h][t] - lift^[h][t]) * q_last^-1  (NTT form), t < L-1; c has L limbs per poly
__global__ __launch_bounds__(256) void k_rescale_combine(const double* __restrict__ ct, const double* __restrict__ lift,
                                                         double* __restrict__ out, ResArgs a,
                                                         const DevPrime* __restrict__ pr, int logn, int L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, h = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const double x = ct[((size_t)h * L + t) * n + k] - lift[((size_t)h * (L - 1) + t) * n + k];
  out[((size_t)h * (L - 1) + t) * n + k] = canon_full(mulc(x, a.c[t], a.cp[t], q), q, qinv);
}
// out = (x0 y0, x0 y1 + x1 y0, x1 y1) over the L primes (NTT form)
// ciphertext j = blockIdx.z: x_j = x + j*sx with xL limbs per polynomial (its first L
// limbs read: the drop to L is free), likewise y; out_j = out + j*3LN
__global__ __launch_bounds__(256) void k_tensor(const double* __restrict__ x, const double* __restrict__ y,
                                                double* __restrict__ out, const DevPrime* __restrict__ pr, int logn,
                                                int L, int xL, int yL, size_t sx, size_t sy) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const size_t j = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = (size_t)t * n + k, ln = (size_t)L * n;
  x += j * sx;
  y += j * sy;
  out += j * 3 * ln;
  const double x0 = x[o], x1 = x[(size_t)xL * n + o], y0 = y[o], y1 = y[(size_t)yL * n + o];
  out[o] = canon_full(mul(x0, y0, q, qinv), q, qinv);
  out[ln + o] = canon_full(mul(x0, y1, q, qinv) + mul(x1, y0, q, qinv), q, qinv);
  out[2 * ln + o] = canon_full(mul(x1, y1, q, qinv), q, qinv);
}
// tensors of count ciphertext pairs given by pointer (pair j = blockIdx.z): x_j with
// xL[j] limbs per polynomial (its first L read), likewise y_j; out_j = out + j*3LN
__global__ __launch_bounds__(256) void k_tensor_list(TensorList a, double* __restrict__ out,
                                                     const DevPrime* __restrict__ pr, int logn, int L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, j = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = (size_t)t * n + k, ln = (size_t)L * n;
  const double* __restrict__ x = a.x[j];
  const double* __restrict__ y = a.y[j];
  const double x0 = x[o], x1 = x[(size_t)a.xL[j] * n + o], y0 = y[o], y1 = y[(size_t)a.yL[j] * n + o];
  out += (size_t)j * 3 * ln;
  out[o] = canon_full(mul(x0, y0, q, qinv), q, qinv);
  out[ln + o] = canon_full(mul(x0, y1, q, qinv) + mul(x1, y0, q, qinv), q, qinv);
  out[2 * ln + o] = canon_full(mul(x1, y1, q, qinv), q, qinv);
}
// Chebyshev products, in place over count ciphertexts (pair j = blockIdx.z >> 1,
// polynomial h = blockIdx.z & 1): p_j <- 2 p_j - c_j T1 (odd[j]; T1 with t1L limbs per
// polynomial, its first L read) or 2 p_j + c_j on polynomial 0 (even)
__global__ __launch_bounds__(256) void k_cheb_fix(double* __restrict__ prod, const double* __restrict__ t1,
                                                  ChebFixArgs a, const DevPrime* __restrict__ pr, int logn, int L,
                                                  int t1L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, j = blockIdx.z >> 1, h = blockIdx.z & 1;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = ((size_t)(2 * j + h) * L + t) * n + k;
  double v = prod[o];
  v = v + v;
  if (a.odd[j]) v -= mulc(t1[((size_t)h * t1L + t) * n + k], a.c[j][t], a.cp[j][t], q);
  else if (h == 0) v += a.c[j][t];
  prod[o] = canon_full(v, q, qinv);
}
// out = (accumulate ? out : 0) + sum_i x_i * c_i (+ c0 on polynomial 0), one ciphertext;
// x_i canonical with xL[i] limbs per polynomial (its first L read); a reduction after
// every four terms keeps the lazy sum below 5q
__global__ __launch_bounds__(256) void k_lincomb(double* __restrict__ out, LinArgs a, const DevPrime* __restrict__ pr,
                                                 int logn, int L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, h = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = ((size_t)h * L + t) * n + k;
  double v = a.accumulate ? out[o] : 0.0;
  for (int i = 0; i < a.nterm; ++i) {
    v += mulc(a.x[i][((size_t)h * a.xL[i] + t) * n + k], a.c[i][t], a.cp[i][t], q);
    if ((i & 3) == 3) v = reduce(v, q, qinv);
  }
  if (h == 0) v += a.c0[t];
  out[o] = canon_full(v, q, qinv);
}
// out[h][t] = x[h][t] * c_t (mode 0), or out = x with c_t added to the first polynomial of
// every ciphertext (even h, mode 1), or out[h][t] = x[h][t] +/- y[h][t] (mode 2 add, mode 3
// subtract); x has xL limbs per polynomial (its first L read), y and out L
__global__ __launch_bounds__(256) void k_ct_elem(const double* __restrict__ x, const double* __restrict__ y,
                                                 double* __restrict__ out, ResArgs a,
                                                 const DevPrime* __restrict__ pr, int logn, int L, int xL, int mode,
                                                 size_t sx, size_t sy, size_t so) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y, h = blockIdx.z;
  const size_t ct = (size_t)(h >> 1), p = (size_t)(h & 1);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = ct * so + (p * L + t) * n + k;
  double v = x[ct * sx + (p * xL + t) * n + k];
  if (mode == 0) v = mulc(v, a.c[t], a.cp[t], q);
  else if (mode == 1) v = p == 0 ? v + a.c[t] : v;
  else if (mode == 2) v = v + y[ct * sy + (p * L + t) * n + k];
  else v = v - y[ct * sy + (p * L + t) * n + k];
  out[o] = canon_full(v, q, qinv);
}

__global__ __launch_bounds__(256) void k_int_to_res(const int64_t* __restrict__ src, double* __restrict__ dst,
                                                    const DevPrime* __restrict__ pr, int logn, int nprimes) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const int p = blockIdx.z;
  const int64_t q = (int64_t)pr[t].q;
  int64_t v = src[(size_t)p * n + k] % q;
  if (v < 0) v += q;
  dst[((size_t)p * nprimes + t) * n + k] = (double)v;
}

__global__ __launch_bounds__(256) void k_u64_to_res(const uint64_t* __restrict__ src, size_t words,
                                                    double* __restrict__ dst) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < words) dst[i] = (double)src[i];
}

__global__ __launch_bounds__(256) void k_res_to_u64(const double* __restrict__ src, size_t words,
                                                    uint64_t* __restrict__ dst) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < words) dst[i] = (uint64_t)src[i];
}

__global__ __launch_bounds__(256) void k_keygen_combine(double* __restrict__ key, const double* __restrict__ e,
                                                        const double* __restrict__ s,
                                                        const DevPrime* __restrict__ pr, int logn, int L, int np,
                                                        int alpha, uint32_t gal) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const int i = blockIdx.z;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const int lo = i * alpha, hi = min(lo + alpha, L);
  const double gad = (t >= lo && t < hi) ? pr[t].pmod : 0.0;
  const double a = key[(((size_t)i * 2 + 1) * np + t) * n + k];
  const double st = s[(size_t)t * n + k];
  const double sg = gal == 0u ? mul(st, st, q, qinv) : s[(size_t)t * n + perm((uint32_t)k, gal, logn)];
  const double ev = e[((size_t)i * np + t) * n + k];
  const double v = -mul(a, st, q, qinv) + ev + mul(gad, sg, q, qinv);
  key[(((size_t)i * 2 + 0) * np + t) * n + k] = canon_full(v, q, qinv);
}

__global__ __launch_bounds__(256) void k_enc_combine(double* __restrict__ ct, const double* __restrict__ v,
                                                     const double* __restrict__ s,
                                                     const DevPrime* __restrict__ pr, int logn, int L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = (size_t)t * n + k;
  const double c1 = ct[(size_t)L * n + o];
  ct[o] = canon_full(v[o] - mul(c1, s[o], q, qinv), q, qinv);
}

__global__ __launch_bounds__(256) void k_dec_combine(const double* __restrict__ ct, double* __restrict__ out,
                                                     const double* __restrict__ s,
                                                     const DevPrime* __restrict__ pr, int logn, int L) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const double q = pr[t].q, qinv = pr[t].qinv;
  const size_t o = (size_t)t * n + k;
  out[o] = canon_full(ct[o] + mul(ct[(size_t)L * n + o], s[o], q, qinv), q, qinv);
}

}  // namespace

// ===========================================================================
// launchers
// ===========================================================================
// The library's fixed scratch array (fa_rotate_static): every GPU that loads
// the library holds its own copy.  The host refers to it only through the
// device address hipGetSymbolAddress returns on that GPU.
static __device__ __align__(256) double scratch[FA_STATIC_SCRATCH_BYTES / 8];

namespace fa {

// The address of `scratch` on `device` (which must be current), looked up once
// per device and kept; nullptr (with the HIP error in *err) if the lookup fails.
void* static_scratch(int device, hipError_t* err) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static void* ptr[kMaxDev] = {};
  static hipError_t res[kMaxDev] = {};
  static bool done[kMaxDev] = {};
  if (device < 0 || device >= kMaxDev) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!done[device]) {
    void* p = nullptr;
    res[device] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    ptr[device] = res[device] == hipSuccess ? p : nullptr;
    done[device] = true;
  }
  *err = res[device];
  return ptr[device];
}

template <int SA>
static void launch_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  using P = PassA<SA>;
  dim3 ga(c->n / P::TILE, l.n);
  hipLaunchKernelGGL(k_ntt_fwd_a<SA>, ga, dim3(256), 0, s, l, c->d_pr, c->d_twa_fwd);
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, l.n);
  hipLaunchKernelGGL(k_ntt_fwd_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn);
}

template <int SA>
static void launch_inv(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  using P = PassA<SA>;
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, l.n);
  hipLaunchKernelGGL(k_ntt_inv_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_twt_inv, c->d_twr_inv, c->logn);
  dim3 ga(c->n / P::TILE, l.n);
  hipLaunchKernelGGL(k_ntt_inv_a<SA>, ga, dim3(256), 0, s, l, c->d_pr, c->d_twa_inv);
}

#define FA_SA_SWITCH(fn, ...)            \
  switch (c->logn - 8) {                  \
    case 2: fn<2>(__VA_ARGS__); break;    \
    case 3: fn<3>(__VA_ARGS__); break;    \
    case 4: fn<4>(__VA_ARGS__); break;    \
    case 5: fn<5>(__VA_ARGS__); break;    \
    case 6: fn<6>(__VA_ARGS__); break;    \
    case 7: fn<7>(__VA_ARGS__); break;    \
    case 8: fn<8>(__VA_ARGS__); break;    \
    default: break;                       \
  }

void ntt_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  if (l.n == 0) return;
  FA_SA_SWITCH(launch_fwd, c, l, s)
}

void ntt_inv(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  if (l.n == 0) return;
  FA_SA_SWITCH(launch_inv, c, l, s)
}

void ntt_inv_b(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  if (l.n == 0) return;
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, l.n);
  hipLaunchKernelGGL(k_ntt_inv_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_twt_inv, c->d_twr_inv, c->logn);
}

static void strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                    hipStream_t s, bool fwd) {
  LimbBatch b(c, s, fwd);
  for (int i = 0; i < count; ++i) b.add(base + (size_t)i * stride, i % period + prime_off);
}

void ntt_fwd_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s) {
  strided(c, base, stride, count, period, prime_off, s, true);
}
void ntt_inv_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s) {
  strided(c, base, stride, count, period, prime_off, s, false);
}

// target groups of a fused ModUp launch: a launch of at least 256 workgroups
// keeps one group per digit (the repeated inverse passes of more groups cost
// more than they gain there); a smaller one (one ciphertext) is split to about
// FA_MU_WGS (default 512) workgroups, at most one group per target
static int modup_groups(int wgs, int targets) {
  static const int want = [] {
    const char* e = getenv("FA_MU_WGS");
    return e && atoi(e) > 0 ? atoi(e) : 512;
  }();
  if (wgs >= 256) return 1;
  const int g = (want + wgs - 1) / wgs;
  return g < 1 ? 1 : g > targets ? targets : g;
}
template <int SA, int ALPHA>
static void launch_modup_fused(const fa_ctx* c, const MuArgs& a, int count, hipStream_t s) {
  using P = PassA<SA>;
  const int ngrp = modup_groups(c->n / P::TILE * c->dnum * count, c->np - ALPHA);
  dim3 g(c->n / P::TILE, c->dnum * ngrp, count);
  hipLaunchKernelGGL((k_modup_fused<SA, ALPHA>), g, dim3(256), 0, s, a, c->d_pr, c->d_twa_fwd, c->d_twa_inv,
                     c->d_mu_hat, c->d_mu_scale, c->logn, c->L, c->np, ngrp);
}
template <int SA>
static void launch_modup_fused_sa(const fa_ctx* c, const MuArgs& a, int count, hipStream_t s) {
  switch (c->alpha) {
    case 1: launch_modup_fused<SA, 1>(c, a, count, s); break;
    case 2: launch_modup_fused<SA, 2>(c, a, count, s); break;
    case 3: launch_modup_fused<SA, 3>(c, a, count, s); break;
    case 4: launch_modup_fused<SA, 4>(c, a, count, s); break;
    default: break;
  }
}

static void modup_pass_b(const fa_ctx* c, const MuItem* items, int count, hipStream_t s);

void modup_fused(const fa_ctx* c, const MuItem* items, int count, hipStream_t s, bool pass_b) {
  for (int off = 0; off < count; off += FA_MAXMU) {
    const int m = count - off < FA_MAXMU ? count - off : FA_MAXMU;
    MuArgs a;
    for (int i = 0; i < m; ++i) a.it[i] = items[off + i];
    FA_SA_SWITCH(launch_modup_fused_sa, c, a, m, s)
  }
  if (pass_b) modup_pass_b(c, items, count, s);
}

static void modup_pass_b(const fa_ctx* c, const MuItem* items, int count, hipStream_t s) {
  // second pass over every converted limb
  LimbList l;
  l.n = 0;
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, 0);
  auto flush = [&]() {
    if (!l.n) return;
    gb.y = l.n;
    hipLaunchKernelGGL(k_ntt_fwd_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn);
    l.n = 0;
  };
  for (int b = 0; b < count; ++b)
    for (int i = 0; i < c->dnum; ++i) {
      const int lo = i * c->alpha, hi = lo + c->alpha < c->L ? lo + c->alpha : c->L;
      for (int t = 0; t < c->np; ++t) {
        if (t >= lo && t < hi) continue;
        l.ptr[l.n] = items[b].ext + ((size_t)i * c->np + t) * c->n;
        l.src[l.n] = l.ptr[l.n];
        l.prime[l.n] = t;
        l.scale[l.n] = 0.0;
        if (++l.n == FA_MAXL) flush();
      }
    }
  flush();
}

template <int SA, int KP>
static void launch_moddown_fused(const fa_ctx* c, const MdArgs& a, int count, hipStream_t s) {
  using P = PassA<SA>;
  const int ngrp = modup_groups(c->n / P::TILE * count, c->L);
  dim3 g(c->n / P::TILE, ngrp, count);
  hipLaunchKernelGGL((k_moddown_fused<SA, KP>), g, dim3(256), 0, s, a, c->d_pr, c->d_twa_fwd, c->d_twa_inv,
                     c->d_md_hat, c->d_md_scale, c->logn, c->L, ngrp);
}
template <int SA>
static void launch_moddown_fused_sa(const fa_ctx* c, const MdArgs& a, int count, hipStream_t s) {
  switch (c->K) {
    case 1: launch_moddown_fused<SA, 1>(c, a, count, s); break;
    case 2: launch_moddown_fused<SA, 2>(c, a, count, s); break;
    case 3: launch_moddown_fused<SA, 3>(c, a, count, s); break;
    case 4: launch_moddown_fused<SA, 4>(c, a, count, s); break;
    default: break;
  }
}

void moddown_fused(const fa_ctx* c, const MdItem* items, int count, hipStream_t s, bool pass_b) {
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  for (int off = 0; off < count; off += FA_MAXMD) {
    const int m = count - off < FA_MAXMD ? count - off : FA_MAXMD;
    MdArgs a;
    for (int i = 0; i < m; ++i) a.it[i] = items[off + i];
    FA_SA_SWITCH(launch_moddown_fused_sa, c, a, m, s)
    if (!pass_b) continue;
    dim3 gb((c->n >> 8) / rows, c->L, m);
    hipLaunchKernelGGL(k_moddown_b, gb, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn);
  }
}


// 1-D grid of the key-switch kernels: nx * ny * ngroup work units, padded to
// whole groups of eight per query when nq > 1 (see ks_decode)
static unsigned ks_grid(int nx, int ny, int nq, int ngroup) {
  if (nq == 1) return 8u * ngroup * (((unsigned)nx * ny + 7) / 8);  // ks_decode_src
  const unsigned units = (unsigned)nx * ny * ngroup;
  return 8u * nq * ((units + 7) / 8);
}

// inverse of an odd Galois element modulo 2N (Newton's iteration modulo 2^32)
static uint32_t inv_galois(uint32_t g, int logn) {
  uint32_t x = g;
  for (int i = 0; i < 5; ++i) x *= 2u - g * x;
  return x & ((2u << logn) - 1u);
}

template <int DNUM>
static void launch_moddown_ks(const fa_ctx* c, const MdKsArgs& a, int m, int nq, hipStream_t s) {
  // eight 256-word rows per workgroup (four on a ring of 2^10, the smallest
  // accepted): twice the workgroups of sixteen-row tiles, measured faster at
  // 8 and 12 primes and even at 3
  const int rows = (c->n >> 8) < 8 ? (c->n >> 8) : 8;
  const int ngroup = m / nq;
  dim3 gb(ks_grid((c->n >> 8) / rows, c->L, nq, ngroup));
  if (rows == 8 && nq == 1)
    hipLaunchKernelGGL((k_moddown_ks_b<DNUM, 8, true>), gb, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd, c->d_twr_fwd,
                       c->logn, c->L, c->np, c->alpha, nq, ngroup);
  else if (rows == 8)
    hipLaunchKernelGGL((k_moddown_ks_b<DNUM, 8, false>), gb, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd,
                       c->d_twr_fwd, c->logn, c->L, c->np, c->alpha, nq, ngroup);
  else
    hipLaunchKernelGGL((k_moddown_ks_b<DNUM, 4, false>), gb, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd,
                       c->d_twr_fwd, c->logn, c->L, c->np, c->alpha, nq, ngroup);
}

void moddown_ks(const fa_ctx* c, const MdKsItem* items, int count, hipStream_t s, int nq) {
  const int chunk = (FA_MAXMD / nq) * nq;
  for (int off = 0; off < count; off += chunk) {
    const int m = count - off < chunk ? count - off : chunk;
    MdKsArgs a;
    for (int i = 0; i < m; ++i) {
      a.it[i] = items[off + i];
      a.it[i].inv_gal = inv_galois(a.it[i].gal, c->logn);
    }
    switch (c->dnum) {
      case 1: launch_moddown_ks<1>(c, a, m, nq, s); break;
      case 2: launch_moddown_ks<2>(c, a, m, nq, s); break;
      case 3: launch_moddown_ks<3>(c, a, m, nq, s); break;
      case 4: launch_moddown_ks<4>(c, a, m, nq, s); break;
      case 5: launch_moddown_ks<5>(c, a, m, nq, s); break;
      case 6: launch_moddown_ks<6>(c, a, m, nq, s); break;
      case 7: launch_moddown_ks<7>(c, a, m, nq, s); break;
      case 8: launch_moddown_ks<8>(c, a, m, nq, s); break;
      default: break;
    }
  }
}

template <int DNUM>
static void launch_ks(const fa_ctx* c, const KsArgs& a, int m, bool accumulate, hipStream_t s, int t0, int nq) {
  const int ngroup = m / nq;
  dim3 g(ks_grid(c->n / 256, c->np - t0, nq, ngroup));
  hipLaunchKernelGGL(k_ks_inner<DNUM>, g, dim3(256), 0, s, a, c->d_pr, c->logn, c->L, c->np, c->alpha,
                     accumulate ? 1 : 0, t0, nq, ngroup);
}

void ks_inner(const fa_ctx* c, const KsItem* items, int count, bool accumulate, hipStream_t s, int t0, int nq) {
  const int chunk = (FA_MAXKS / nq) * nq;
  for (int off = 0; off < count; off += chunk) {
    KsArgs a;
    const int m = count - off < chunk ? count - off : chunk;
    for (int i = 0; i < m; ++i) {
      a.it[i] = items[off + i];
      a.it[i].inv_gal = inv_galois(a.it[i].gal, c->logn);
    }
    switch (c->dnum) {
      case 1: launch_ks<1>(c, a, m, accumulate, s, t0, nq); break;
      case 2: launch_ks<2>(c, a, m, accumulate, s, t0, nq); break;
      case 3: launch_ks<3>(c, a, m, accumulate, s, t0, nq); break;
      case 4: launch_ks<4>(c, a, m, accumulate, s, t0, nq); break;
      case 5: launch_ks<5>(c, a, m, accumulate, s, t0, nq); break;
      case 6: launch_ks<6>(c, a, m, accumulate, s, t0, nq); break;
      case 7: launch_ks<7>(c, a, m, accumulate, s, t0, nq); break;
      case 8: launch_ks<8>(c, a, m, accumulate, s, t0, nq); break;
      default: break;
    }
  }
}

template <int DNUM>
static void launch_ks_inv_b(const fa_ctx* c, const KsArgs& a, int m, hipStream_t s, int nq) {
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  const int ngroup = m / nq;
  dim3 g(ks_grid((c->n >> 8) / rows, c->K, nq, ngroup));
  hipLaunchKernelGGL(k_ks_inv_b<DNUM>, g, dim3(256), 0, s, a, c->d_pr, c->d_twt_inv, c->d_twr_inv, c->logn, c->L,
                     c->np, nq, ngroup);
}

void ks_inv_b(const fa_ctx* c, const KsItem* items, int count, hipStream_t s, int nq) {
  if (c->dnum != 1) return;  // the host calls it for one-digit contexts only
  const int chunk = (FA_MAXKS / nq) * nq;
  for (int off = 0; off < count; off += chunk) {
    KsArgs a;
    const int m = count - off < chunk ? count - off : chunk;
    for (int i = 0; i < m; ++i) {
      a.it[i] = items[off + i];
      a.it[i].inv_gal = inv_galois(a.it[i].gal, c->logn);
    }
    launch_ks_inv_b<1>(c, a, m, s, nq);
  }
}

template <int DNUM>
static void launch_giant(const fa_ctx* c, const GiantArgs& a, hipStream_t s) {
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  const int ntile = (c->n >> 8) / rows;
  const int rest8 = (ntile * c->np + 7) / 8;
  dim3 g((unsigned)(8 * a.nb * rest8));
  if (rows == 16)
    hipLaunchKernelGGL((k_giant_ks<DNUM, 16>), g, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn,
                       c->L, c->np, c->alpha, ntile);
  else if (rows == 8)
    hipLaunchKernelGGL((k_giant_ks<DNUM, 8>), g, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn,
                       c->L, c->np, c->alpha, ntile);
  else
    hipLaunchKernelGGL((k_giant_ks<DNUM, 4>), g, dim3(256), 0, s, a, c->d_pr, c->d_twt_fwd, c->d_twr_fwd, c->logn,
                       c->L, c->np, c->alpha, ntile);
}

void giant_ks(const fa_ctx* c, const double* ext, const double* acc, size_t astride, const double* const* keys,
              const uint32_t* gals, int nb, int ng, double* u, hipStream_t s) {
  const size_t ext_g = (size_t)c->dnum * c->np * c->n;
  for (int g0 = 0; g0 < ng; g0 += FA_MAXG) {
    GiantArgs a;
    const int m = ng - g0 < FA_MAXG ? ng - g0 : FA_MAXG;
    // chunks of giant indices: ext of chunk g0 is [nb][m] laid out inside [nb][ng]
    a.ext = ext + (size_t)g0 * ext_g;
    a.acc = acc;
    for (int g = 0; g < m; ++g) {
      a.key[g] = keys[g0 + g];
      a.gal[g] = gals[g0 + g];
    }
    a.u = u;
    a.astride = astride;
    a.nb = nb;
    a.ng = m;
    a.ngs = ng;
    a.g0 = 1 + g0;
    a.accumulate = g0 > 0;
    switch (c->dnum) {
      case 1: launch_giant<1>(c, a, s); break;
      case 2: launch_giant<2>(c, a, s); break;
      case 3: launch_giant<3>(c, a, s); break;
      case 4: launch_giant<4>(c, a, s); break;
      case 5: launch_giant<5>(c, a, s); break;
      case 6: launch_giant<6>(c, a, s); break;
      case 7: launch_giant<7>(c, a, s); break;
      case 8: launch_giant<8>(c, a, s); break;
      default: break;
    }
  }
}

// Most (block, giant) accumulator pairs one pass keeps in registers for one
// query: 32 (default), 16 or 8; FA_MAC_PAIRS overrides it for tuning.  With
// NQ queries per pass the pairs per pass drop to 32 / NQ.
// the three-stage single-query kernel (FA_MAC_STAGES=2 selects the two-slot one)
// 17..31 pairs left: one padded 32-pair launch (FA_MAC_PAD=0: 16 + 16 / 8)
static bool mac_pad_wide() {
  static const bool v = [] {
    const char* e = getenv("FA_MAC_PAD");
    return !e || atoi(e) != 0;
  }();
  return v;
}
static bool mac_three_stages() {
  static const bool v = [] {
    const char* e = getenv("FA_MAC_STAGES");
    return !(e && atoi(e) == 2);
  }();
  return v;
}

// pairs per pass of a four-query group: 8 (default) or 16 (FA_MAC_Q4_PAIRS)
static int mac_q4_pairs() {
  static const int v = [] {
    const char* e = getenv("FA_MAC_Q4_PAIRS");
    return e && atoi(e) == 16 ? 16 : 8;
  }();
  return v;
}

static int mac_pairs_max() {
  static const int v = [] {
    const char* e = getenv("FA_MAC_PAIRS");
    const int r = e ? atoi(e) : 32;
    return (r == 8 || r == 16) ? r : 32;
  }();
  return v;
}

// ring depth of the staged loads: as many slots as fit beside the other
// workgroup sharing a CU's 160 KB of LDS (two slots at one query x 32 pairs)
template <int NQ, int NACC>
struct MacStages {
  static constexpr int BYTES = 4 * (NACC + 2 * NQ) * 64 * 8;
  static constexpr int S = BYTES * 3 <= 80 * 1024 ? 3 : 2;
};

template <int NQ, int NACC>
static void launch_mac(MacArgs a, int nchunk, const fa_ctx* c, hipStream_t s) {
  a.ntile = (int)((size_t)c->L * c->n / 256);
  a.nchunk = nchunk;
  const unsigned grid = nchunk == 1 ? (unsigned)a.ntile : 8u * nchunk * ((a.ntile + 7) / 8);
  if constexpr (NQ == 1) {
    if (mac_three_stages())
      hipLaunchKernelGGL((k_mac_diag3<NACC>), dim3(grid), dim3(256), 0, s, a, c->d_pr, c->logn);
    else
      hipLaunchKernelGGL((k_mac_diag<NQ, NACC, MacStages<NQ, NACC>::S>), dim3(grid), dim3(256), 0, s, a, c->d_pr,
                         c->logn);
  } else {
    hipLaunchKernelGGL((k_mac_diag<NQ, NACC, MacStages<NQ, NACC>::S>), dim3(grid), dim3(256), 0, s, a, c->d_pr,
                       c->logn);
  }
}

// pairs p0.. of the current query group: all full chunks of the group's widest
// pass in one launch, then one narrower launch for the rest
template <int NQ, int WIDE>
static int mac_chunks(MacArgs& a, int p0, const fa_ctx* c, hipStream_t s) {
  const int left = a.n_pairs - p0;
  a.pair0 = p0;
  if (left >= WIDE) {
    launch_mac<NQ, WIDE>(a, left / WIDE, c, s);
    return p0 + (left / WIDE) * WIDE;
  }
  if (NQ == 1 && WIDE == 32 && left > 16 && mac_pad_wide()) {
    // one padded launch: the missing pairs re-read the last pair's rows (cache
    // hits) instead of a second launch re-reading every rotated query
    launch_mac<NQ, WIDE>(a, 1, c, s);
    return p0 + WIDE;
  }
  if (WIDE > 16 && left > 8) {
    launch_mac<NQ, (WIDE > 16 ? 16 : WIDE)>(a, 1, c, s);
    return p0 + 16;
  }
  launch_mac<NQ, 8>(a, 1, c, s);
  return p0 + 8;
}

void mac_diag(const fa_ctx* c, const double* const* q, const double* const* qrot, int nq,
              const double* const* blocks, int n_blocks, int B, int G, double* const* acc, hipStream_t s) {
  const int pmax = mac_pairs_max();
  int logG = 0;
  while ((1 << logG) < G) ++logG;
  const size_t ctw = (size_t)2 * c->L * c->n;
  for (int j0 = 0; j0 < nq;) {
    const int m = nq - j0 >= 4 ? 4 : nq - j0 >= 2 ? 2 : 1;  // queries sharing this plaintext pass
    for (int b0 = 0; b0 < n_blocks; b0 += FA_MAXBLK) {
      const int nb = n_blocks - b0 < FA_MAXBLK ? n_blocks - b0 : FA_MAXBLK;
      MacArgs a;
      for (int j = 0; j < m; ++j) {
        a.q0[j] = q[j0 + j];
        a.qrot[j] = qrot[j0 + j];
        a.acc[j] = acc[j0 + j] + (size_t)b0 * G * ctw;
      }
      for (int i = 0; i < nb; ++i) a.blk[i] = blocks[b0 + i];
      a.n_pairs = nb * G;
      a.B = B;
      a.logG = logG;
      a.L = c->L;
      for (int p0 = 0; p0 < a.n_pairs;) {
        if (m == 4) p0 = mac_q4_pairs() == 16 ? mac_chunks<4, 16>(a, p0, c, s) : mac_chunks<4, 8>(a, p0, c, s);
        else if (m == 2) p0 = pmax >= 32 ? mac_chunks<2, 16>(a, p0, c, s) : mac_chunks<2, 8>(a, p0, c, s);
        else if (pmax >= 32) p0 = mac_chunks<1, 32>(a, p0, c, s);
        else if (pmax >= 16) p0 = mac_chunks<1, 16>(a, p0, c, s);
        else p0 = mac_chunks<1, 8>(a, p0, c, s);
      }
    }
    j0 += m;
  }
}

template <int NACC>
static void launch_mac_ct(MacCtArgs a, int nchunk, const fa_ctx* c, hipStream_t s) {
  a.ntile = (int)((size_t)c->L * c->n / 256);
  a.nchunk = nchunk;
  const unsigned grid = nchunk == 1 ? (unsigned)a.ntile : 8u * nchunk * ((a.ntile + 7) / 8);
  hipLaunchKernelGGL((k_mac_diag_ct<NACC>), dim3(grid), dim3(256), 0, s, a, c->d_pr, c->logn);
}

void mac_diag_ct(const fa_ctx* c, const double* q, const double* qrot, const double* const* blocks, int n_blocks,
                 int B, int G, double* acc, hipStream_t s) {
  int logG = 0;
  while ((1 << logG) < G) ++logG;
  const size_t ln = (size_t)c->L * c->n;
  for (int b0 = 0; b0 < n_blocks; b0 += FA_MAXBLK) {
    const int nb = n_blocks - b0 < FA_MAXBLK ? n_blocks - b0 : FA_MAXBLK;
    MacCtArgs a;
    a.q0 = q;
    a.qrot = qrot;
    a.acc = acc + (size_t)b0 * G * 3 * ln;
    for (int i = 0; i < nb; ++i) a.blk[i] = blocks[b0 + i];
    a.n_pairs = nb * G;
    a.B = B;
    a.logG = logG;
    a.L = c->L;
    for (int p0 = 0; p0 < a.n_pairs;) {
      const int left = a.n_pairs - p0;
      a.pair0 = p0;
      if (left >= 16) {
        launch_mac_ct<16>(a, left / 16, c, s);
        p0 += (left / 16) * 16;
      } else {
        launch_mac_ct<8>(a, 1, c, s);
        p0 += 8;
      }
    }
  }
}

void mul_plain(const fa_ctx* c, const double* ct, const double* const* pts, int count, double* out, hipStream_t s) {
  for (int off = 0; off < count; off += FA_MAXPT) {
    PtArgs a;
    const int m = count - off < FA_MAXPT ? count - off : FA_MAXPT;
    for (int i = 0; i < m; ++i) a.pt[i] = pts[off + i];
    dim3 g((unsigned)((size_t)c->L * c->n / 256), m);
    hipLaunchKernelGGL(k_mul_plain, g, dim3(256), 0, s, ct, a, out + (size_t)off * 2 * c->L * c->n, c->d_pr,
                       c->logn, c->L);
  }
}

void add_automorph(const fa_ctx* c, double* dst, const double* src, int n_polys, uint32_t gal, hipStream_t s) {
  dim3 g(c->n / 256, n_polys * c->L);
  hipLaunchKernelGGL(k_add_automorph, g, dim3(256), 0, s, dst, src, c->d_pr, c->logn, c->L, gal);
}

static ResArgs res_args(const fa_ctx* c, const uint64_t* cres, int L) {
  ResArgs a;
  for (int t = 0; t < FA_MAXLIMB; ++t) {
    a.c[t] = t < L ? (double)cres[t] : 0.0;
    a.cp[t] = t < L ? a.c[t] / (double)c->primes[t] : 0.0;
  }
  return a;
}

void rescale(const fa_ctx* c, const double* ct, int n_polys, double* out, double* scratch, hipStream_t s) {
  const size_t n = c->n;
  const int L = c->L;
  double* last = scratch;                        // [n_polys][N]
  double* lift = scratch + (size_t)n_polys * n;  // [n_polys][L-1][N]
  {
    LimbBatch inv(c, s, false);
    for (int h = 0; h < n_polys; ++h) inv.add(last + (size_t)h * n, L - 1, ct + ((size_t)h * L + L - 1) * n);
  }
  const double ql = (double)c->primes[L - 1];
  hipLaunchKernelGGL(k_rescale_lift, dim3(c->n / 256, L - 1, n_polys), dim3(256), 0, s, last, lift, c->d_pr, c->logn,
                     L - 1, ql);
  ntt_fwd_strided(c, lift, n, n_polys * (L - 1), L - 1, 0, s);
  std::vector<uint64_t> inv(L - 1);
  const uint64_t qlast = c->primes[L - 1];
  for (int t = 0; t < L - 1; ++t) {
    const uint64_t q = c->primes[t];
    // (q_last mod q)^(q-2) mod q
    unsigned __int128 b = qlast % q, r = 1;
    for (uint64_t e = q - 2; e; e >>= 1) {
      if (e & 1) r = r * b % q;
      b = b * b % q;
    }
    inv[t] = (uint64_t)r;
  }
  hipLaunchKernelGGL(k_rescale_combine, dim3(c->n / 256, L - 1, n_polys), dim3(256), 0, s, ct, lift, out,
                     res_args(c, inv.data(), L - 1), c->d_pr, c->logn, L);
}

void tensor(const fa_ctx* c, const double* x, int xL, size_t sx, const double* y, int yL, size_t sy, int count,
            double* out, hipStream_t s) {
  hipLaunchKernelGGL(k_tensor, dim3(c->n / 256, c->L, count), dim3(256), 0, s, x, y, out, c->d_pr, c->logn, c->L,
                     xL, yL, sx, sy);
}

void tensor_list(const fa_ctx* c, const double* const* xs, const int* xLs, const double* const* ys, const int* yLs,
                 int count, double* out, hipStream_t s) {
  const size_t step = (size_t)3 * c->L * c->n;
  for (int j0 = 0; j0 < count; j0 += FA_MAXTERM) {
    const int m = std::min(FA_MAXTERM, count - j0);
    TensorList a{};
    for (int j = 0; j < m; ++j) {
      a.x[j] = xs[j0 + j];
      a.y[j] = ys[j0 + j];
      a.xL[j] = xLs[j0 + j];
      a.yL[j] = yLs[j0 + j];
    }
    hipLaunchKernelGGL(k_tensor_list, dim3(c->n / 256, c->L, m), dim3(256), 0, s, a, out + (size_t)j0 * step,
                       c->d_pr, c->logn, c->L);
  }
}

void cheb_fix(const fa_ctx* c, double* prod, int count, const double* t1, int t1L, const uint64_t* const* cres,
              const int* odd, hipStream_t s) {
  const size_t step = (size_t)2 * c->L * c->n;
  for (int j0 = 0; j0 < count; j0 += FA_MAXTERM) {
    const int m = std::min(FA_MAXTERM, count - j0);
    ChebFixArgs a{};
    for (int j = 0; j < m; ++j) {
      const ResArgs r = res_args(c, cres[j0 + j], c->L);
      for (int t = 0; t < FA_MAXLIMB; ++t) {
        a.c[j][t] = r.c[t];
        a.cp[j][t] = r.cp[t];
      }
      a.odd[j] = odd[j0 + j];
    }
    hipLaunchKernelGGL(k_cheb_fix, dim3(c->n / 256, c->L, 2 * m), dim3(256), 0, s, prod + (size_t)j0 * step,
                       t1, a, c->d_pr, c->logn, c->L, t1L);
  }
}

void lincomb(const fa_ctx* c, double* out, const double* const* xs, const int* xLs, const uint64_t* const* cres,
             int nterm, const uint64_t* c0res, hipStream_t s) {
  for (int i0 = 0; i0 < nterm; i0 += FA_MAXTERM) {
    const int m = std::min(FA_MAXTERM, nterm - i0);
    LinArgs a{};
    for (int i = 0; i < m; ++i) {
      const ResArgs r = res_args(c, cres[i0 + i], c->L);
      a.x[i] = xs[i0 + i];
      a.xL[i] = xLs[i0 + i];
      for (int t = 0; t < FA_MAXLIMB; ++t) {
        a.c[i][t] = r.c[t];
        a.cp[i][t] = r.cp[t];
      }
    }
    if (i0 == 0 && c0res)
      for (int t = 0; t < c->L; ++t) a.c0[t] = (double)c0res[t];
    a.nterm = m;
    a.accumulate = i0 > 0;
    hipLaunchKernelGGL(k_lincomb, dim3(c->n / 256, c->L, 2), dim3(256), 0, s, out, a, c->d_pr, c->logn, c->L);
  }
}

void ct_elem(const fa_ctx* c, const double* x, const double* y, double* out, int n_polys, const uint64_t* cres,
             int mode, hipStream_t s, int xL, size_t sx, size_t sy, size_t so) {
  std::vector<uint64_t> zero(c->L, 0);
  const int xl = xL ? xL : c->L;
  const size_t n = c->n, ctw = 2 * (size_t)c->L * n;
  // the defaults: consecutive ciphertexts (x with xl limbs per polynomial)
  if (sx == (size_t)-1) sx = 2 * (size_t)xl * n;
  if (sy == (size_t)-1) sy = ctw;
  if (so == (size_t)-1) so = ctw;
  hipLaunchKernelGGL(k_ct_elem, dim3(c->n / 256, c->L, n_polys), dim3(256), 0, s, x, y, out,
                     res_args(c, cres ? cres : zero.data(), c->L), c->d_pr, c->logn, c->L, xl, mode, sx, sy, so);
}

void add_limbs(const fa_ctx* c, double* dst, const double* src, int n_limbs, int period, hipStream_t s) {
  dim3 g(c->n / 256, n_limbs);
  hipLaunchKernelGGL(k_add_limbs, g, dim3(256), 0, s, dst, src, c->d_pr, c->logn, period);
}

void int_to_res(const fa_ctx* c, const int64_t* src, int n_polys, int nprimes, double* dst, hipStream_t s) {
  for (int p0 = 0; p0 < n_polys; p0 += 65535) {
    const int m = n_polys - p0 < 65535 ? n_polys - p0 : 65535;
    dim3 g(c->n / 256, nprimes, m);
    hipLaunchKernelGGL(k_int_to_res, g, dim3(256), 0, s, src + (size_t)p0 * c->n,
                       dst + (size_t)p0 * nprimes * c->n, c->d_pr, c->logn, nprimes);
  }
}

void u64_to_res(const uint64_t* src, size_t words, double* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_u64_to_res, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, s, src, words, dst);
}

void res_to_u64(const double* src, size_t words, uint64_t* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_res_to_u64, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, s, src, words, dst);
}

void keygen_combine(const fa_ctx* c, double* key, const double* e_ntt, uint32_t gal, hipStream_t s) {
  dim3 g(c->n / 256, c->np, c->dnum);
  hipLaunchKernelGGL(k_keygen_combine, g, dim3(256), 0, s, key, e_ntt, c->d_s, c->d_pr, c->logn, c->L, c->np,
                     c->alpha, gal);
}

void enc_combine(const fa_ctx* c, double* ct, const double* v, hipStream_t s) {
  dim3 g(c->n / 256, c->L);
  hipLaunchKernelGGL(k_enc_combine, g, dim3(256), 0, s, ct, v, c->d_s, c->d_pr, c->logn, c->L);
}

void dec_combine(const fa_ctx* c, const double* ct, double* out, hipStream_t s) {
  dim3 g(c->n / 256, c->L);
  hipLaunchKernelGGL(k_dec_combine, g, dim3(256), 0, s, ct, out, c->d_s, c->d_pr, c->logn, c->L);
}

}  // namespace fa
