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

#include "wave_ops.h"

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

// Rows whose length is a multiple of E = 16 / sizeof(T) elements (16-byte
// rows, 16-byte aligned base): each lane loads E consecutive elements with one
// 16-byte load.  A row takes NL = c / E lanes; rows of NL <= 16 lanes are
// packed 64 / L to a wavefront in aligned groups of L = NL rounded up to a
// power of two, longer rows take a whole wavefront each and go through the
// row 64 vectors at a time.  A lane loads only when its row exists and its
// vector lies inside the row (v < NL), so every address read is inside x;
// every position written is below the row's non-zero count <= c.  A lane's
// non-zeros go to the positions after those of the lanes before it in the
// row (a group prefix sum of the per-lane counts by DPP row shifts), in index
// order.
template <typename T>
struct Vec16;
template <>
struct Vec16<float> {
  static constexpr int E = 4;
  using type = float4;
  static __device__ __forceinline__ float get(const float4& v, int e) {
    return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w));
  }
};
template <>
struct Vec16<int8_t> {
  static constexpr int E = 16;
  using type = int4;
  static __device__ __forceinline__ int8_t get(const int4& v, int e) {
    const int w = e < 4 ? v.x : (e < 8 ? v.y : (e < 12 ? v.z : v.w));
    return (int8_t)(w >> (8 * (e & 3)));
  }
};

// Inclusive prefix sum over aligned groups of 1 << lg lanes (lg <= 4, one DPP
// row) or the whole wavefront (lg == 6); p = the lane's place in its group.
__device__ __forceinline__ int compact_group_incl(int v, int lg, int p) {
  if (lg == 6) return (int)wave_incl_scan((uint32_t)v, 0u, OpAdd{});
  if (lg >= 1) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false); v += p >= 1 ? t : 0; }
  if (lg >= 2) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false); v += p >= 2 ? t : 0; }
  if (lg >= 3) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false); v += p >= 4 ? t : 0; }
  if (lg >= 4) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false); v += p >= 8 ? t : 0; }
  return v;
}

// lg: log2 of the lanes per row group (0..4, or 6: one row per wavefront).
template <typename T>
__global__ __launch_bounds__(256) void compact_vec(const T* __restrict__ x, int64_t rows, int c,
                                                   int lg, uint16_t* __restrict__ idx,
                                                   T* __restrict__ val,
                                                   int32_t* __restrict__ cnt) {
  using V = Vec16<T>;
  constexpr int E = V::E;
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int NL = c / E;                                   // vectors per row (c % E == 0)
  const int L = 1 << lg;
  const int rpw = 64 >> lg;                               // rows per wavefront (lg == 6: 1)
  const int sub = lane >> lg, p = lane & (L - 1);
  const int last = L - 1;
  for (int64_t r0 = wave * rpw; r0 < rows; r0 += nwaves * rpw) {
    const int64_t row = r0 + sub;
    const bool rv = row < rows;
    const T* xr = x + (rv ? row : 0) * c;
    uint16_t* ir = idx + (rv ? row : 0) * c;
    T* vr = val + (rv ? row : 0) * c;
    int run = 0;
    for (int v0 = 0; v0 < NL; v0 += L) {                  // uniform: one pass unless lg == 6
      const int vi = v0 + p;
      const bool ld = rv && vi < NL;
      typename V::type q{};
      if (ld) q = reinterpret_cast<const typename V::type*>(xr)[vi];
      uint32_t nzm = 0;
#pragma unroll
      for (int e = 0; e < E; ++e) nzm |= (ld && V::get(q, e) != T(0)) ? 1u << e : 0u;
      const int nl = __popc(nzm);
      const int incl = compact_group_incl(nl, lg, p);
      int pos = run + incl - nl;
      if (ld) {
        for (uint32_t m = nzm; m != 0u; m &= m - 1u) {
          const int e = __builtin_ctz(m);
          ir[pos] = (uint16_t)(vi * E + e);
          vr[pos] = V::get(q, e);
          ++pos;
        }
      }
      // the group's total: its last lane's inclusive sum
      run += lg == 6 ? __builtin_amdgcn_readlane(incl, 63) : __shfl(incl, (lane & ~last) + last, 64);
    }
    if (rv && p == 0) cnt[row] = run;
  }
}

}  // namespace cs
