// Multiply, Route and Sum (Section 3.2 steps 3-5; Sections 3.3.1-3.3.2) of a
// sparse-sparse convolution whose input pixels are already compacted into
// (index, value) lists.  A linear layer is the 1x1 convolution of 1x1 images.
//
// gfx950 mapping
//  * one lane per (output pixel, packed set g); consecutive lanes take
//    consecutive sets of the same pixel, so the G packed weights of slot i
//    (row i of val/kid) are read as one contiguous run, and the pixel's list
//    entries are the same address for those lanes (a broadcast);
//  * Multiply: the lane multiplies each non-zero activation v at slot i by
//    val[i][g] (the "column at a predefined location" of Section 3.2);
//  * Route: the product goes to accumulator kid[i][g] of the lane.  The n
//    accumulators of a lane live in LDS at acc[kid][lane] (a bank is a
//    function of the lane only, so a wavefront's 64 routed adds never
//    conflict, whatever the kernel ids are).  Integer products use the LDS
//    integer atomic add (no return value, pipelined); fp32 products use a
//    lane-private read-add-write (the LDS float atomic is a slow path on
//    this chip).  With n == 1 the single accumulator is a register;
//  * Sum: bias, the optional 2x2 max-pool over the four conv outputs the lane
//    computes in turn, then the n contiguous outputs g*n .. g*n+n-1 of the
//    pixel are stored.  Nothing but the final outputs is written to HBM and
//    no HBM atomics are used; each accumulator adds in list order, so results
//    are bitwise reproducible.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "count_products.h"
#include "phase_stamps.h"

namespace cs {

struct ConvGeom {
  int B, H, W, C;          // input NHWC
  int KH, KW, S, P;        // kernel, stride, pad
  int Ho, Wo;              // conv output size
  int pool;                // 1 or 2
  int G, n, c_out;         // packed sets, kernels per set, output channels
  int cap;                 // list row stride
};

// Entry of the augmented packed tensor (Section 3.3.1): value + Kernel ID.
// int8: one 16-bit word (uint8 value | kid << 8); fp32: (value bits, kid).
template <typename T>
struct Aug;
template <>
struct Aug<int8_t> {
  using type = uint16_t;
  static __device__ __forceinline__ int32_t value(uint16_t e) { return (int32_t)(int8_t)(e & 0xFFu); }
  static __device__ __forceinline__ int kid(uint16_t e) { return (int)(e >> 8); }
};
template <>
struct Aug<float> {
  using type = uint2;
  static __device__ __forceinline__ float value(uint2 e) { return __uint_as_float(e.x); }
  static __device__ __forceinline__ int kid(uint2 e) { return (int)e.y; }
};

template <typename A>
__device__ __forceinline__ void route_add(A* p, A v);

template <>
__device__ __forceinline__ void route_add<int32_t>(int32_t* p, int32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <>
__device__ __forceinline__ void route_add<float>(float* p, float v) {
  *p = *p + v;   // lane-private slot: a plain read-add-write is race free
}

// T: list/weight element type (int8_t or float); A: accumulator (int32_t or float).
template <typename T, typename A, bool ONE>
__global__ __launch_bounds__(256) void mrs_conv(const uint16_t* __restrict__ lidx,
                                                const T* __restrict__ lval,
                                                const int32_t* __restrict__ lcnt,
                                                const typename Aug<T>::type* __restrict__ aug,
                                                const A* __restrict__ bias, A* __restrict__ y,
                                                ConvGeom geo, int64_t total) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int bd = blockDim.x;
  const int tid = threadIdx.x;
  A* acc = reinterpret_cast<A*>(smem);               // [n][bd]
  A* mx = acc + (ONE ? 1 : geo.n) * bd;              // [n][bd] running pool max

  const int64_t t = (int64_t)blockIdx.x * bd + tid;
  if (t >= total) return;                             // no block-level sync below
  const int G = geo.G;
  const int g = (int)(t % G);
  const int64_t opix = t / G;
  const int Hp = geo.Ho / geo.pool, Wp = geo.Wo / geo.pool;
  const int wp = (int)(opix % Wp);
  const int64_t tmp = opix / Wp;
  const int hp = (int)(tmp % Hp);
  const int bb = (int)(tmp / Hp);
  const int n = ONE ? 1 : geo.n;

  A accr = A(0);
  const int nq = geo.pool * geo.pool;
  for (int q = 0; q < nq; ++q) {
    const int ho = hp * geo.pool + q / geo.pool;
    const int wo = wp * geo.pool + q % geo.pool;
    if (ONE) {
      accr = A(0);
    } else {
      for (int k = 0; k < n; ++k) acc[k * bd + tid] = A(0);
    }
    for (int ky = 0; ky < geo.KH; ++ky) {
      const int hy = ho * geo.S + ky - geo.P;
      if (hy < 0 || hy >= geo.H) continue;
      for (int kx = 0; kx < geo.KW; ++kx) {
        const int wx = wo * geo.S + kx - geo.P;
        if (wx < 0 || wx >= geo.W) continue;
        const int64_t pix = ((int64_t)bb * geo.H + hy) * geo.W + wx;
        const int m = min(lcnt[pix], geo.cap);      // never read past a list row
        const uint16_t* li = lidx + pix * geo.cap;
        const T* lv = lval + pix * geo.cap;
        const int64_t sbase = (int64_t)(ky * geo.KW + kx) * geo.C;
        for (int j = 0; j < m; ++j) {
          const int64_t i = sbase + li[j];
          const auto e = aug[i * G + g];
          const A prod = (A)lv[j] * (A)Aug<T>::value(e);       // Multiply
          if (ONE) {
            accr += prod;                                       // Sum
          } else {
            route_add<A>(&acc[Aug<T>::kid(e) * bd + tid], prod);  // Route + Sum
          }
        }
      }
    }
    // Sum epilogue for this conv output: bias, running max for the pool
    for (int k = 0; k < n; ++k) {
      A a = ONE ? accr : acc[k * bd + tid];
      if (bias) a += bias[g * n + k];
      if (nq == 1) {
        y[opix * geo.c_out + g * n + k] = a;
      } else if (q == 0) {
        mx[k * bd + tid] = a;
      } else {
        const A b = mx[k * bd + tid];
        mx[k * bd + tid] = a > b ? a : b;
      }
    }
  }
  if (nq > 1) {
    for (int k = 0; k < n; ++k) y[opix * geo.c_out + g * n + k] = mx[k * bd + tid];
  }
}

}  // namespace cs
