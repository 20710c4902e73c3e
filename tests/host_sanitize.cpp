// Host-side check of libfa's client code (encode, decode) built with
// AddressSanitizer and UndefinedBehaviorSanitizer, no GPU needed.
// tests/test_host_sanitizers.py compiles this file with the library's host
// source, then feeds parameter sets on stdin, one per line:
//     log_n L q_0 ... q_{L-1}
// For each set it encodes random slot vectors, reduces the integer
// coefficients to residues (also after multiplying them by 2^40, the scale of
// a score), decodes them with fa_decode and prints
//     ok log_n L max_err
// or exits non-zero.  The context is filled in by hand: encode and decode read
// only the ring degree, the prime count and the primes.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "fa_internal.h"

using u64 = uint64_t;
using u128 = unsigned __int128;
using i128 = __int128;

static u64 mod_i128(i128 x, u64 q) {
  i128 r = x % (i128)q;
  return (u64)(r < 0 ? r + (i128)q : r);
}

int main() {
  int logn, L;
  std::mt19937_64 g(7);
  std::uniform_real_distribution<double> uni(-1.0, 1.0);
  while (std::scanf("%d %d", &logn, &L) == 2) {
    fa_ctx c;
    c.logn = logn;
    c.n = 1 << logn;
    c.L = L;
    c.np = L;
    c.primes.resize(L);
    for (int t = 0; t < L; ++t)
      if (std::scanf("%llu", (unsigned long long*)&c.primes[t]) != 1) return 2;
    const int n = c.n, S = n / 2;
    double worst = 0.0;
    for (int extra : {0, 40}) {
      // a short vector (the rest of the slots zero) and a full one
      for (int ns : {S / 3 + 1, S}) {
        std::vector<double> v(S, 0.0);
        for (int j = 0; j < ns; ++j) v[j] = uni(g);
        std::vector<int64_t> m(n);
        if (fa_encode(&c, v.data(), ns, 40, m.data()) != FA_OK) return 3;
        std::vector<u64> res((size_t)L * n);
        for (int t = 0; t < L; ++t)
          for (int k = 0; k < n; ++k) {
            const i128 x = (i128)m[k] * ((i128)1 << extra) + (i128)((k % 7) - 3);  // plus a little noise
            res[(size_t)t * n + k] = mod_i128(x, c.primes[t]);
          }
        std::vector<double> z(S);
        if (fa_decode(&c, res.data(), 40 + extra, z.data(), S) != FA_OK) return 4;
        for (int j = 0; j < S; ++j) worst = std::fmax(worst, std::fabs(z[j] - v[j]));
        // the first slots only
        std::vector<double> z5(5);
        if (fa_decode(&c, res.data(), 40 + extra, z5.data(), 5) != FA_OK) return 5;
        for (int j = 0; j < 5; ++j)
          if (z5[j] != z[j]) return 6;
      }
    }
    // argument checks return errors without touching the buffers
    std::vector<u64> r1(1);
    std::vector<double> z1(1);
    if (fa_decode(&c, nullptr, 40, z1.data(), 1) == FA_OK) return 7;
    if (fa_decode(&c, r1.data(), 40, z1.data(), S + 1) == FA_OK) return 8;
    std::printf("ok %d %d %.3e\n", logn, L, worst);
    if (!(worst < 1e-6)) return 9;
  }
  return 0;
}
