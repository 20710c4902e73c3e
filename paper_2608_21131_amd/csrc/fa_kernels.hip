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
// Forward NTT values stay within 1.6 q, inverse NTT values within 2 q.

#include <hip/hip_runtime.h>

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

// Cooley-Tukey butterfly (forward): (x, y) -> (x + w y, x - w y)
__device__ __forceinline__ void ct_bfly(double& x, double& y, double w, double q, double qinv) {
  const double u = reduce(x, q, qinv);
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
// Stage s pairs elements j and j + N/2^(s+1) with twiddle psi_rev[2^s + (j >> (logn - s))].
// Pass A runs stages 0..SA-1 on columns (j mod 256 fixed), pass B stages
// SA..logn-1 on contiguous rows of 256.  Each pass keeps a unit of elements
// in registers for half its stages, exchanges through LDS, then finishes.
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

template <int SA>
__global__ __launch_bounds__(256) void k_ntt_fwd_a(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ tw, int logn) {
  using P = PassA<SA>;
  __shared__ double sm[P::TILE];
  const int n = 1 << logn;
  const int pi = ll.prime[blockIdx.y];
  double* __restrict__ a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ w = tw + (size_t)pi * n;
  const int col0 = blockIdx.x * P::COLS;
  for (int u = threadIdx.x; u < P::TILE / P::E1; u += 256) {
    const int c = u % P::COLS, hl = u / P::COLS;
    double x[P::E1];
#pragma unroll
    for (int m = 0; m < P::E1; ++m) x[m] = a[((size_t)(hl + (m << P::S2)) << 8) + col0 + c];
#pragma unroll
    for (int s = 0; s < P::S1; ++s) {
      const int half = P::E1 >> (s + 1);
#pragma unroll
      for (int m = 0; m < P::E1; ++m) {
        if (m & half) continue;
        ct_bfly(x[m], x[m + half], w[(1 << s) + (m >> (P::S1 - s))], q, qinv);
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
        ct_bfly(x[m], x[m + half], w[(1 << s) + (hh << s2) + (m >> (P::S2 - s2))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < P::E2; ++m) a[((size_t)((hh << P::S2) + m) << 8) + col0 + c] = x[m];
  }
}

template <int SA>
__global__ __launch_bounds__(256) void k_ntt_inv_a(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ tw, int logn) {
  using P = PassA<SA>;
  __shared__ double sm[P::TILE];
  const int n = 1 << logn;
  const int pi = ll.prime[blockIdx.y];
  double* __restrict__ a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ w = tw + (size_t)pi * n;
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
  const double ninv = pr[pi].ninv, ninvp = ninv * qinv;
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
      a[((size_t)(hl + (m << P::S2)) << 8) + col0 + c] = canon_full(mulc(x[m], ninv, ninvp, q), q, qinv);
  }
}

// Pass B: rows of 256 contiguous elements, stages SA..SA+7.  Row stride in
// LDS is 272 words (one pad word per 16) so that both access patterns spread
// over all banks.
#define ROWW 272
__device__ __forceinline__ int lds_row(int rl, int lo) { return rl * ROWW + lo + (lo >> 4); }

__global__ __launch_bounds__(256) void k_ntt_fwd_b(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ tw, int logn) {
  __shared__ double sm[16 * ROWW];
  const int n = 1 << logn, SA = logn - 8;
  const int rows = (n >> 8) < 16 ? (n >> 8) : 16;
  const int row0 = blockIdx.x * rows;
  const int pi = ll.prime[blockIdx.y];
  double* __restrict__ a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ w = tw + (size_t)pi * n;
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int l0 = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) x[m] = a[(size_t)r * 256 + l0 + 16 * m];
#pragma unroll
    for (int s1 = 0; s1 < 4; ++s1) {
      const int half = 8 >> s1;
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        ct_bfly(x[m], x[m + half], w[(1 << (SA + s1)) + (r << s1) + (m >> (4 - s1))], q, qinv);
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
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        ct_bfly(x[m], x[m + half], w[(1 << (SA + s1)) + (r << s1) + (lh << (s1 - 4)) + (m >> (8 - s1))], q, qinv);
      }
    }
    double2* dst = reinterpret_cast<double2*>(a + (size_t)r * 256 + 16 * lh);
#pragma unroll
    for (int m = 0; m < 8; ++m)
      dst[m] = make_double2(canon_full(x[2 * m], q, qinv), canon_full(x[2 * m + 1], q, qinv));
  }
}

__global__ __launch_bounds__(256) void k_ntt_inv_b(LimbList ll, const DevPrime* __restrict__ pr,
                                                   const double* __restrict__ tw, int logn) {
  __shared__ double sm[16 * ROWW];
  const int n = 1 << logn, SA = logn - 8;
  const int rows = (n >> 8) < 16 ? (n >> 8) : 16;
  const int row0 = blockIdx.x * rows;
  const int pi = ll.prime[blockIdx.y];
  double* __restrict__ a = ll.ptr[blockIdx.y];
  const double q = pr[pi].q, qinv = pr[pi].qinv;
  const double* __restrict__ w = tw + (size_t)pi * n;
  for (int u = threadIdx.x; u < rows * 16; u += 256) {
    const int lh = u & 15, rl = u >> 4, r = row0 + rl;
    double x[16];
    const double2* src = reinterpret_cast<const double2*>(a + (size_t)r * 256 + 16 * lh);
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const double2 v = src[m];
      x[2 * m] = v.x;
      x[2 * m + 1] = v.y;
    }
#pragma unroll
    for (int s1 = 7; s1 >= 4; --s1) {
      const int half = 8 >> (s1 - 4);
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], w[(1 << (SA + s1)) + (r << s1) + (lh << (s1 - 4)) + (m >> (8 - s1))], q, qinv);
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
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        if (m & half) continue;
        gs_bfly(x[m], x[m + half], w[(1 << (SA + s1)) + (r << s1) + (m >> (4 - s1))], q, qinv);
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) a[(size_t)r * 256 + l0 + 16 * m] = x[m];
  }
}

// ---------------------------------------------------------------------------
// fast basis conversion (no correction term):
//   Conv_{S->t}(x) = sum_j [x_j * (S/s_j)^-1]_{s_j} * ((S/s_j) mod t)  mod t
// The bracket is taken canonical in [0, s_j), as the definition requires.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_conv_modup(const double* __restrict__ c1c, size_t src_stride,
                                                    double* __restrict__ ext, size_t dst_stride,
                                                    const DevPrime* __restrict__ pr,
                                                    const double* __restrict__ inv, const double* __restrict__ hat,
                                                    int logn, int L, int np, int alpha) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int i = blockIdx.y;
  const int b = blockIdx.z;
  const int lo = i * alpha;
  const int hi = min(lo + alpha, L);
  const double* __restrict__ src = c1c + (size_t)b * src_stride;
  double* __restrict__ dst = ext + (size_t)b * dst_stride + (size_t)i * np * n;
  double y[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (lo + j < hi) {
      const double q = pr[lo + j].q, qinv = pr[lo + j].qinv, iv = inv[i * alpha + j];
      y[j] = canon(mulc(src[(size_t)(lo + j) * n + k], iv, iv * qinv, q), q);
    } else {
      y[j] = 0.0;
    }
  }
  for (int t = 0; t < np; ++t) {
    if (t >= lo && t < hi) continue;
    const double q = pr[t].q, qinv = pr[t].qinv;
    double acc = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (lo + j < hi) {
        const double hv = hat[((size_t)i * alpha + j) * np + t];
        acc += mulc(y[j], hv, hv * qinv, q);
      }
    }
    dst[(size_t)t * n + k] = reduce(acc, q, qinv);
  }
}

__global__ __launch_bounds__(256) void k_conv_moddown(const double* __restrict__ up, size_t src_stride,
                                                      double* __restrict__ out, size_t dst_stride,
                                                      const DevPrime* __restrict__ pr,
                                                      const double* __restrict__ inv,
                                                      const double* __restrict__ hat, int logn, int L, int K) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int b = blockIdx.y;
  const double* __restrict__ src = up + (size_t)b * src_stride;
  double* __restrict__ dst = out + (size_t)b * dst_stride;
  double y[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j < K) {
      const double q = pr[L + j].q, qinv = pr[L + j].qinv, iv = inv[j];
      y[j] = canon(mulc(src[(size_t)j * n + k], iv, iv * qinv, q), q);
    } else {
      y[j] = 0.0;
    }
  }
  for (int t = 0; t < L; ++t) {
    const double q = pr[t].q, qinv = pr[t].qinv;
    double acc = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j < K) {
        const double hv = hat[(size_t)j * L + t];
        acc += mulc(y[j], hv, hv * qinv, q);
      }
    }
    dst[(size_t)t * n + k] = reduce(acc, q, qinv);
  }
}

__global__ __launch_bounds__(256) void k_scatter_own(const double* __restrict__ c1, size_t src_stride,
                                                     double* __restrict__ ext, size_t dst_stride, int logn,
                                                     int L, int np, int alpha) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const int b = blockIdx.z;
  const int i = t / alpha;
  ext[(size_t)b * dst_stride + ((size_t)i * np + t) * n + k] = c1[(size_t)b * src_stride + (size_t)t * n + k];
}

// ---------------------------------------------------------------------------
// key-switch inner product with the automorphism folded into the read of ext
// ---------------------------------------------------------------------------
#define FA_MAXKS 32
struct KsArgs {
  int count;
  fa::KsItem it[FA_MAXKS];
};

__global__ __launch_bounds__(256) void k_ks_inner(KsArgs args, const DevPrime* __restrict__ pr, int logn, int np,
                                                  int dnum, int accumulate) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const fa::KsItem& it = args.it[blockIdx.z];
  const double q = pr[t].q, qinv = pr[t].qinv;
  const uint32_t kk = perm((uint32_t)k, it.gal, logn);
  double acc0 = 0.0, acc1 = 0.0;
  for (int i = 0; i < dnum; ++i) {
    const double x = it.ext[((size_t)i * np + t) * n + kk];
    const double kb = it.key[(((size_t)i * 2 + 0) * np + t) * n + k];
    const double ka = it.key[(((size_t)i * 2 + 1) * np + t) * n + k];
    acc0 += mul(x, kb, q, qinv);
    acc1 += mul(x, ka, q, qinv);
  }
  double* u0 = it.u + (size_t)t * n + k;
  double* u1 = it.u + ((size_t)np + t) * n + k;
  if (accumulate) {
    acc0 += *u0;
    acc1 += *u1;
  }
  *u0 = canon_full(acc0, q, qinv);
  *u1 = canon_full(acc1, q, qinv);
}

#define FA_MAXFIN 32
struct FinArgs {
  int count;
  fa::FinishItem it[FA_MAXFIN];
};

__global__ __launch_bounds__(256) void k_moddown_finish(FinArgs args, const DevPrime* __restrict__ pr, int logn,
                                                        int L, int np) {
  const int n = 1 << logn;
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int t = blockIdx.y;
  const fa::FinishItem& it = args.it[blockIdx.z];
  const double q = pr[t].q, qinv = pr[t].qinv, pv = pr[t].pinv, pvp = pv * qinv;
  const uint32_t kk = it.gal == 1u ? (uint32_t)k : perm((uint32_t)k, it.gal, logn);
  const size_t o = (size_t)t * n + k;
  for (int h = 0; h < 2; ++h) {
    const double* base = h == 0 ? it.base0 : it.base1;
    const double v = it.u[(size_t)h * np * n + o] - it.conv[(size_t)h * L * n + o];
    double r = mulc(v, pv, pvp, q);
    if (base) r += base[(size_t)t * n + kk];
    it.out[(size_t)h * L * n + o] = canon_full(r, q, qinv);
  }
}

// ---------------------------------------------------------------------------
// diagonal-layout multiply-accumulate: the HBM stream of the scoring path
//   acc[blk][g][h][t][k] = sum_b pts[blk][g*B+b][t][k] * qrot[b][h][t][k]
// One thread per coefficient (t, k); up to NACC (block, g) pairs per pass so
// every baby rotation of the query is read once per pass; a reduction every
// 8 products keeps the lazy sums below 2^53.
// ---------------------------------------------------------------------------
#define FA_MAXBLK 32
struct MacArgs {
  const double* qrot;
  const double* blk[FA_MAXBLK];
  double* acc;
  int n_pairs, pair0, B, G, L;
};

template <int NACC>
__global__ __launch_bounds__(256) void k_mac_diag(MacArgs args, const DevPrime* __restrict__ pr, int logn) {
  const int n = 1 << logn;
  const size_t ln = (size_t)args.L * n;
  const size_t f = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int t = (int)(f >> logn);
  const double q = pr[t].q, qinv = pr[t].qinv;
  const int cnt = min(NACC, args.n_pairs - args.pair0);
  const double* __restrict__ pbase[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    const int pair = args.pair0 + (i < cnt ? i : 0);
    const int blk = pair / args.G, g = pair % args.G;
    pbase[i] = args.blk[blk] + (size_t)g * args.B * ln + f;
  }
  double a0[NACC], a1[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    a0[i] = 0.0;
    a1[i] = 0.0;
  }
  const double* __restrict__ qr = args.qrot + f;
  for (int b = 0; b < args.B; ++b) {
    const double x0 = qr[(size_t)(2 * b) * ln];
    const double x1 = qr[(size_t)(2 * b + 1) * ln];
    const double x0p = x0 * qinv, x1p = x1 * qinv;
#pragma unroll
    for (int i = 0; i < NACC; ++i) {
      if (i < cnt) {
        const double p = pbase[i][(size_t)b * ln];
        a0[i] += mulc(p, x0, x0p, q);
        a1[i] += mulc(p, x1, x1p, q);
      }
    }
    if ((b & 7) == 7) {
#pragma unroll
      for (int i = 0; i < NACC; ++i) {
        a0[i] = reduce(a0[i], q, qinv);
        a1[i] = reduce(a1[i], q, qinv);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NACC; ++i) {
    if (i < cnt) {
      double* o = args.acc + (size_t)(args.pair0 + i) * 2 * ln + f;
      o[0] = canon_full(a0[i], q, qinv);
      o[ln] = canon_full(a1[i], q, qinv);
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
  const double sg = s[(size_t)t * n + perm((uint32_t)k, gal, logn)];
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
namespace fa {

template <int SA>
static void launch_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  using P = PassA<SA>;
  dim3 ga(c->n / P::TILE, l.n);
  hipLaunchKernelGGL(k_ntt_fwd_a<SA>, ga, dim3(256), 0, s, l, c->d_pr, c->d_tw_fwd, c->logn);
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, l.n);
  hipLaunchKernelGGL(k_ntt_fwd_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_tw_fwd, c->logn);
}

template <int SA>
static void launch_inv(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  using P = PassA<SA>;
  const int rows = (c->n >> 8) < 16 ? (c->n >> 8) : 16;
  dim3 gb((c->n >> 8) / rows, l.n);
  hipLaunchKernelGGL(k_ntt_inv_b, gb, dim3(256), 0, s, l, c->d_pr, c->d_tw_inv, c->logn);
  dim3 ga(c->n / P::TILE, l.n);
  hipLaunchKernelGGL(k_ntt_inv_a<SA>, ga, dim3(256), 0, s, l, c->d_pr, c->d_tw_inv, c->logn);
}

void ntt_fwd(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  if (l.n == 0) return;
  switch (c->logn - 8) {
    case 2: launch_fwd<2>(c, l, s); break;
    case 3: launch_fwd<3>(c, l, s); break;
    case 4: launch_fwd<4>(c, l, s); break;
    case 5: launch_fwd<5>(c, l, s); break;
    case 6: launch_fwd<6>(c, l, s); break;
    case 7: launch_fwd<7>(c, l, s); break;
    case 8: launch_fwd<8>(c, l, s); break;
    default: break;
  }
}

void ntt_inv(const fa_ctx* c, const LimbList& l, hipStream_t s) {
  if (l.n == 0) return;
  switch (c->logn - 8) {
    case 2: launch_inv<2>(c, l, s); break;
    case 3: launch_inv<3>(c, l, s); break;
    case 4: launch_inv<4>(c, l, s); break;
    case 5: launch_inv<5>(c, l, s); break;
    case 6: launch_inv<6>(c, l, s); break;
    case 7: launch_inv<7>(c, l, s); break;
    case 8: launch_inv<8>(c, l, s); break;
    default: break;
  }
}

static void strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                    hipStream_t s, bool fwd) {
  LimbList l;
  l.n = 0;
  for (int i = 0; i < count; ++i) {
    l.ptr[l.n] = base + (size_t)i * stride;
    l.prime[l.n] = i % period + prime_off;
    if (++l.n == FA_MAXL) {
      fwd ? ntt_fwd(c, l, s) : ntt_inv(c, l, s);
      l.n = 0;
    }
  }
  if (l.n) fwd ? ntt_fwd(c, l, s) : ntt_inv(c, l, s);
}

void ntt_fwd_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s) {
  strided(c, base, stride, count, period, prime_off, s, true);
}
void ntt_inv_strided(const fa_ctx* c, double* base, size_t stride, int count, int period, int prime_off,
                     hipStream_t s) {
  strided(c, base, stride, count, period, prime_off, s, false);
}

void ntt_fwd_ext(const fa_ctx* c, double* ext, size_t stride, int batch, hipStream_t s) {
  LimbList l;
  l.n = 0;
  const size_t n = c->n;
  for (int b = 0; b < batch; ++b)
    for (int i = 0; i < c->dnum; ++i) {
      const int lo = i * c->alpha, hi = lo + c->alpha < c->L ? lo + c->alpha : c->L;
      for (int t = 0; t < c->np; ++t) {
        if (t >= lo && t < hi) continue;
        l.ptr[l.n] = ext + (size_t)b * stride + ((size_t)i * c->np + t) * n;
        l.prime[l.n] = t;
        if (++l.n == FA_MAXL) {
          ntt_fwd(c, l, s);
          l.n = 0;
        }
      }
    }
  if (l.n) ntt_fwd(c, l, s);
}

void conv_modup(const fa_ctx* c, const double* c1c, size_t src_stride, double* ext, size_t dst_stride, int batch,
                hipStream_t s) {
  dim3 g(c->n / 256, c->dnum, batch);
  hipLaunchKernelGGL(k_conv_modup, g, dim3(256), 0, s, c1c, src_stride, ext, dst_stride, c->d_pr, c->d_mu_inv,
                     c->d_mu_hat, c->logn, c->L, c->np, c->alpha);
}

void conv_moddown(const fa_ctx* c, const double* up, size_t src_stride, double* out, size_t dst_stride, int count,
                  hipStream_t s) {
  dim3 g(c->n / 256, count);
  hipLaunchKernelGGL(k_conv_moddown, g, dim3(256), 0, s, up, src_stride, out, dst_stride, c->d_pr, c->d_md_inv,
                     c->d_md_hat, c->logn, c->L, c->K);
}

void scatter_own(const fa_ctx* c, const double* c1, size_t src_stride, double* ext, size_t dst_stride, int batch,
                 hipStream_t s) {
  dim3 g(c->n / 256, c->L, batch);
  hipLaunchKernelGGL(k_scatter_own, g, dim3(256), 0, s, c1, src_stride, ext, dst_stride, c->logn, c->L, c->np,
                     c->alpha);
}

void ks_inner(const fa_ctx* c, const KsItem* items, int count, bool accumulate, hipStream_t s) {
  for (int off = 0; off < count; off += FA_MAXKS) {
    KsArgs a;
    a.count = count - off < FA_MAXKS ? count - off : FA_MAXKS;
    for (int i = 0; i < a.count; ++i) a.it[i] = items[off + i];
    dim3 g(c->n / 256, c->np, a.count);
    hipLaunchKernelGGL(k_ks_inner, g, dim3(256), 0, s, a, c->d_pr, c->logn, c->np, c->dnum, accumulate ? 1 : 0);
  }
}

void moddown_finish(const fa_ctx* c, const FinishItem* items, int count, hipStream_t s) {
  for (int off = 0; off < count; off += FA_MAXFIN) {
    FinArgs a;
    a.count = count - off < FA_MAXFIN ? count - off : FA_MAXFIN;
    for (int i = 0; i < a.count; ++i) a.it[i] = items[off + i];
    dim3 g(c->n / 256, c->L, a.count);
    hipLaunchKernelGGL(k_moddown_finish, g, dim3(256), 0, s, a, c->d_pr, c->logn, c->L, c->np);
  }
}

void mac_diag(const fa_ctx* c, const double* qrot, const double* const* blocks, int n_blocks, int B, int G,
              double* acc, hipStream_t s) {
  for (int b0 = 0; b0 < n_blocks; b0 += FA_MAXBLK) {
    const int nb = n_blocks - b0 < FA_MAXBLK ? n_blocks - b0 : FA_MAXBLK;
    MacArgs a;
    a.qrot = qrot;
    for (int i = 0; i < nb; ++i) a.blk[i] = blocks[b0 + i];
    a.acc = acc + (size_t)b0 * G * 2 * c->L * c->n;
    a.n_pairs = nb * G;
    a.B = B;
    a.G = G;
    a.L = c->L;
    dim3 g((unsigned)((size_t)c->L * c->n / 256));
    for (int p0 = 0; p0 < a.n_pairs;) {
      a.pair0 = p0;
      const int left = a.n_pairs - p0;
      if (left > 8) {
        hipLaunchKernelGGL(k_mac_diag<32>, g, dim3(256), 0, s, a, c->d_pr, c->logn);
        p0 += 32;
      } else {
        hipLaunchKernelGGL(k_mac_diag<8>, g, dim3(256), 0, s, a, c->d_pr, c->logn);
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
