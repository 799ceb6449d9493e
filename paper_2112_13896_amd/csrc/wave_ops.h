// Wavefront-wide scans and reductions with DPP (data-parallel primitives:
// row shifts and row broadcasts read another lane's register directly, no
// LDS round trip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

// Inclusive scan over the 64 lanes of a wavefront: shifts by 1, 2, 4, 8
// inside each row of 16 lanes, then the last lane of rows 0 and 2 to rows 1
// and 3, then lane 31 to rows 2 and 3.  Lanes without a source take the
// identity.  Every lane of the wavefront must be active.
template <typename Op>
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, uint32_t id, Op op) {
  const int iv = (int)id;
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x111, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x112, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x114, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x118, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x142, 0xa, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(iv, (int)v, 0x143, 0xc, 0xf, false));
  return v;
}

struct OpAdd {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; }
};
struct OpMin {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a < b ? a : b; }
};
struct OpMax {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a > b ? a : b; }
};

// Compiler-only ordering of a wavefront's LDS accesses: the LDS runs one
// wavefront's instructions in issue order, so a write by one lane is seen by a
// later read of another lane of the same wavefront once the compiler keeps
// the two in order.
__device__ __forceinline__ void wave_lds_order() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_wave_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Wavefront minimum / maximum, the same in every lane (all lanes active).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(v, 0xFFFFFFFFu, OpMin{}), 63);
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(v, 0u, OpMax{}), 63);
}

// Within rows of 16 lanes (DPP row operations; every lane active):
// butterfly reductions whose result every lane of the row holds - xor 1 and
// xor 2 inside quads, then the half-row and row mirrors - and an inclusive
// prefix sum by row shifts of 1, 2, 4, 8.
template <typename Op>
__device__ __forceinline__ uint32_t row16_reduce(uint32_t v, Op op) {
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xf, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xf, 0xf, false));
  return v;
}
__device__ __forceinline__ int row16_incl_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);
  return v;
}

// A value the compiler must treat as unknown where it is used: keeps it from
// hoisting per-slot copies of a lane constant out of a loop, or (a lane's
// own zero) makes a wavefront-uniform address a vector one.
__device__ __forceinline__ int opaque_int(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

}  // namespace cs
