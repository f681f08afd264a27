// fastdiv.h -- division of non-negative 31-bit integers by a divisor fixed at
// launch time, as a multiply-high, an add and a shift (the round-up
// "magic number" method of Granlund and Montgomery, "Division by invariant
// integers using multiplication", PLDI 1994, with the 33-bit multiplier
// folded into an add).
//
// For a divisor d >= 1 let l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1
// (m < 2^32).  Then for every 0 <= n < 2^31
//     n / d == (umulhi(m, n) + n) >> l
// (umulhi(m, n) <= n, so the 32-bit sum cannot overflow).  Host code builds
// the constants; device code evaluates them.  Plain C++ so that a host-only
// test can check the identity exhaustively on small divisors.
#pragma once

#include <stdint.h>

namespace cf {

struct FastDiv {
  uint32_t mul;   // m
  uint32_t shift; // l
  uint32_t div;   // d (for the remainder)
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  uint32_t l = 0;
  while (l < 32 && (1ull << l) < d) ++l;
  f.shift = l;
  f.mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  f.div = d;
  return f;
}

#if defined(__HIPCC__)
__device__ __forceinline__ int fdiv(int n, const FastDiv &f) {
  const uint32_t hi = __umulhi(f.mul, (uint32_t)n);
  return (int)((hi + (uint32_t)n) >> f.shift);
}
#endif

inline int fdiv_host(int n, const FastDiv &f) {
  const uint32_t hi = (uint32_t)(((uint64_t)f.mul * (uint32_t)n) >> 32);
  return (int)((hi + (uint32_t)n) >> f.shift);
}

}  // namespace cf
