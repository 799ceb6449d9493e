// Select step, sparse representation (Section 3.2 step 2; Figure 10 passes
// the surviving activations "along with their indices").  A row of c values
// becomes the ascending list of its non-zero (index, value) pairs plus a count.
//
// gfx950 mapping: each 64-lane wavefront reads 64 consecutive elements, takes
// a ballot of the non-zero lanes and gives every non-zero lane its output slot
// as the popcount of the ballot bits below it (the prefix-sum arbitration of
// Section 3.3.2, done by the wave's mask hardware).  No atomics, no LDS, and
// the list order is the index order.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

constexpr int COMPACT_BATCH = 8;   // 64-element chunks of a row in flight together

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

template <typename T>
__device__ __forceinline__ bool is_nonzero(T v) {
  return v != T(0);  // -0.0f != 0.0f is false: a signed zero is a zero
}

// Rows of c >= 64: one wavefront per row, 64-element chunks.
template <typename T>
__global__ __launch_bounds__(256) void compact_wide(const T* __restrict__ x, int64_t rows, int c,
                                                    uint16_t* __restrict__ idx,
                                                    T* __restrict__ val,
                                                    int32_t* __restrict__ cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const uint64_t below = lanemask_lt(lane);
  for (int64_t row = wave; row < rows; row += nwaves) {
    const T* xr = x + row * c;
    uint16_t* ir = idx + row * c;
    T* vr = val + row * c;
    int run = 0;
    // COMPACT_BATCH chunks of 64 are loaded before any is used
    for (int b0 = 0; b0 < c; b0 += 64 * COMPACT_BATCH) {
      T v[COMPACT_BATCH];
#pragma unroll
      for (int u = 0; u < COMPACT_BATCH; ++u) {
        const int j = b0 + u * 64 + lane;
        v[u] = j < c ? xr[j] : T(0);
      }
#pragma unroll
      for (int u = 0; u < COMPACT_BATCH; ++u) {
        const int j = b0 + u * 64 + lane;
        const bool nz = j < c && is_nonzero(v[u]);
        const uint64_t m = __ballot(nz);
        if (nz) {
          const int pos = run + __popcll(m & below);
          ir[pos] = (uint16_t)j;
          vr[pos] = v[u];
        }
        run += __popcll(m);
      }
    }
    if (lane == 0) cnt[row] = run;
  }
}

// Rows of c < 64: a wavefront holds 64 >> s_log2 rows in segments of
// S = 2^s_log2 >= c lanes; ranks are counted inside the segment.
template <typename T>
__global__ __launch_bounds__(256) void compact_narrow(const T* __restrict__ x, int64_t rows, int c,
                                                      int s_log2, uint16_t* __restrict__ idx,
                                                      T* __restrict__ val,
                                                      int32_t* __restrict__ cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int rows_per_wave = 64 >> s_log2;
  const int sub = lane >> s_log2;
  const int j = lane & ((1 << s_log2) - 1);
  const uint64_t seg = (s_log2 == 6) ? ~0ull
                                     : (((1ull << (1 << s_log2)) - 1ull) << (sub << s_log2));
  const uint64_t below = lanemask_lt(lane);
  for (int64_t r0 = wave * rows_per_wave; r0 < rows; r0 += nwaves * rows_per_wave) {
    const int64_t row = r0 + sub;
    const bool valid = row < rows && j < c;
    const T v = valid ? x[row * c + j] : T(0);
    const bool nz = valid && is_nonzero(v);
    const uint64_t m = __ballot(nz) & seg;
    if (nz) {
      const int pos = __popcll(m & below);
      idx[row * c + pos] = (uint16_t)j;
      val[row * c + pos] = v;
    }
    if (j == 0 && row < rows) cnt[row] = __popcll(m);
  }
}

}  // namespace cs
