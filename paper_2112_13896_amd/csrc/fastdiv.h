// Division of unsigned 32-bit numbers by a divisor fixed at launch: one
// multiply-high, one add and one shift instead of the ~30-instruction
// software division the GPU otherwise runs.  This is the round-up reciprocal
// method for division by invariant integers of T. Granlund and P. L.
// Montgomery, "Division by Invariant Integers using Multiplication", PLDI
// 1994 (Section 4): m = floor(2^32 (2^s - d) / d) + 1 with s = ceil(log2 d),
// then floor(n / d) = (mulhi(n, m) + n) >> s, the add done in 64 bits.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

struct FastDiv {
  uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f{d, 0u, 0u};
  if (d > 1) {
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    f.s = s;
    f.m = (uint32_t)((((1ull << 32) * ((1ull << s) - d)) / d) + 1);
  }
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  return (uint32_t)(((uint64_t)__umulhi(n, f.m) + n) >> f.s);
}

}  // namespace cs
