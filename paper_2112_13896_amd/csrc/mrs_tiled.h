// Multiply, Route and Sum, staged version (Section 3.2 steps 3-5, Sections
// 3.3.1-3.3.2).  Same result as mrs_conv, organised for gfx950:
//
//  * the packed kernels of a slice of Gs sets are copied once per persistent
//    workgroup into LDS in an "augmented" layout (Section 3.3.1: each weight
//    carries its Kernel ID): int8 -> one 16-bit word (value | id << 8); fp32 ->
//    (value, byte offset of the id's accumulator).  With n == 1 no id is kept.
//    Multiply is then one LDS read per product, at row i = the activation's
//    slot (the fixed location of Section 3.2);
//  * lanes are ordered (output item, set, pool sub-pixel q, slice s) with q
//    and s fastest, so the Q*S lanes that make one (item, set) sit in one
//    wavefront: each computes a part of the sums (its sub-pixel of the 2x2
//    pool window, its share of the taps or list chunks) and the parts are
//    combined through LDS inside the wavefront - no workgroup barrier after
//    the table is staged, so wavefronts run independently;
//  * a lane walks its (tap, 4-entry chunk) units with loads in flight ahead
//    of use: the counts and first chunks of the next two taps, and the next
//    chunk of the current tap (vector loads: indices 8 bytes, values 4 or 16
//    bytes); lanes of one pixel read the same addresses;
//  * Route/Sum: accumulators acc[kid][lane] in LDS (bank = lane, conflict
//    free); integer products use the LDS integer atomic add (no return
//    value), fp32 products a lane-private read-add-write.  No HBM atomics;
//    every accumulator adds in a fixed order, so results are reproducible.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mrs_kernels.h"

namespace cs {

constexpr int MRS_BD = 512;     // threads per workgroup
constexpr int MRS_TAPS = 9;     // most taps one lane walks (host picks S accordingly)
constexpr int MRS_AHEAD = 2;    // taps prefetched ahead of the one being processed

template <typename T, bool ONE>
struct TabEntry;
template <>
struct TabEntry<int8_t, false> { using type = uint16_t; };
template <>
struct TabEntry<int8_t, true> { using type = int8_t; };
template <>
struct TabEntry<float, false> { using type = uint2; };        // x: value bits, y: acc byte offset
template <>
struct TabEntry<float, true> { using type = float; };

struct TiledArgs {
  int S, log2S;      // slices per (item, set, sub-pixel), power of two
  int log2Q;         // sub-pixels on separate lanes: 0 (none) or 2 (2x2 pool)
  int Gs;            // sets per table slice
  int gslices;       // number of table slices; gridDim.x is a multiple of it
  int chunk_mode;    // 1: a single tap, slices split its list chunks
  int64_t items;     // output items (pooled pixels when pooling)
};

template <typename T>
struct Chunk;
template <>
struct Chunk<int8_t> {
  uint2 idx;
  uint32_t val;
  __device__ __forceinline__ void load(const uint16_t* li, const int8_t* lv, int j) {
    idx = *reinterpret_cast<const uint2*>(li + j);
    val = *reinterpret_cast<const uint32_t*>(lv + j);
  }
  __device__ __forceinline__ int32_t v(int e) const { return (int32_t)(int8_t)(val >> (8 * e)); }
};
template <>
struct Chunk<float> {
  uint2 idx;
  float4 val;
  __device__ __forceinline__ void load(const uint16_t* li, const float* lv, int j) {
    idx = *reinterpret_cast<const uint2*>(li + j);
    val = *reinterpret_cast<const float4*>(lv + j);
  }
  __device__ __forceinline__ float v(int e) const {
    return e == 0 ? val.x : (e == 1 ? val.y : (e == 2 ? val.z : val.w));
  }
};
__device__ __forceinline__ int chunk_idx(const uint2& ii, int e) {
  const uint32_t wd = e < 2 ? ii.x : ii.y;
  return (int)((e & 1) ? (wd >> 16) : (wd & 0xFFFFu));
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename T, typename A, bool ONE>
__device__ __forceinline__ void mrs_chunk(const Chunk<T>& ch, int lim, int sbase,
                                          const typename TabEntry<T, ONE>::type* trow,
                                          int gcount, A* acc_lane, A& accr) {
  using E = typename TabEntry<T, ONE>::type;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (e < lim) {
      const E te = trow[(sbase + chunk_idx(ch.idx, e)) * gcount];     // Multiply: packed row
      if constexpr (ONE) {
        accr += (A)ch.v(e) * (A)te;                                      // Sum
      } else if constexpr (sizeof(T) == 1) {
        __hip_atomic_fetch_add(acc_lane + (int)(te >> 8) * MRS_BD,       // Route + Sum
                               ch.v(e) * (int32_t)(int8_t)(te & 0xFFu), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
      } else {
        A* p = reinterpret_cast<A*>(reinterpret_cast<unsigned char*>(acc_lane) + te.y);
        *p = *p + ch.v(e) * __uint_as_float(te.x);                       // Route + Sum
      }
    }
  }
}

template <typename T, typename A, bool ONE>
__global__ __launch_bounds__(MRS_BD) void mrs_tiled(const uint16_t* __restrict__ lidx,
                                                    const T* __restrict__ lval,
                                                    const int32_t* __restrict__ lcnt,
                                                    const T* __restrict__ pval,
                                                    const uint8_t* __restrict__ pkid,
                                                    const A* __restrict__ bias,
                                                    A* __restrict__ y, ConvGeom geo,
                                                    TiledArgs ta) {
  using E = typename TabEntry<T, ONE>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int n = ONE ? 1 : geo.n;
  const int T_ = geo.KH * geo.KW;
  const int R = T_ * geo.C;
  const int G = geo.G;
  const int gsl = blockIdx.x % ta.gslices;
  const int bis = blockIdx.x / ta.gslices;              // block index within the set slice
  const int nbs = gridDim.x / ta.gslices;               // blocks per set slice
  const int g0 = gsl * ta.Gs;
  const int gcount = min(ta.Gs, G - g0);

  A* acc = reinterpret_cast<A*>(smem);                  // [n][MRS_BD]
  E* tab = reinterpret_cast<E*>(smem + (size_t)n * MRS_BD * sizeof(A));

  // stage the augmented table of sets [g0, g0 + gcount): tab[i * gcount + gl]
  for (int e = tid; e < R * gcount; e += MRS_BD) {
    const int i = e / gcount, gl = e - i * gcount;
    const int64_t src = (int64_t)i * G + g0 + gl;
    if constexpr (ONE) {
      tab[e] = pval[src];
    } else if constexpr (sizeof(T) == 1) {
      tab[e] = (uint16_t)((uint8_t)pval[src] | ((uint16_t)pkid[src] << 8));
    } else {
      tab[e] = make_uint2(__float_as_uint((float)pval[src]),
                          (uint32_t)pkid[src] * MRS_BD * (uint32_t)sizeof(A));
    }
  }
  __syncthreads();                                      // the only workgroup barrier

  const int S = ta.S;
  const int log2QS = ta.log2S + ta.log2Q;
  const int QS = 1 << log2QS;                           // lanes per (item, set)
  const int nq = 1 << ta.log2Q;
  const int64_t work = ta.items * gcount * QS;
  const int64_t stride = (int64_t)nbs * MRS_BD;
  const int Hp = geo.Ho / geo.pool, Wp = geo.Wo / geo.pool;
  A* acc_lane = acc + tid;
  const int gbase_lane = tid & ~(QS - 1);               // first lane of this (item, set)
  const int r = tid & (QS - 1);                         // rank inside the group
  const int s = r & (S - 1);                            // slice
  const int q = r >> ta.log2S;                          // 2x2 pool sub-pixel
  const int t0 = ta.chunk_mode ? 0 : s;                 // first tap of the lane
  const int tstep = ta.chunk_mode ? T_ : S;             // tap step (chunk mode: one tap)
  const int c0 = ta.chunk_mode ? s : 0;                 // first chunk of a tap
  const int cstep = ta.chunk_mode ? S : 1;
  const int jfirst = c0 * 4 < geo.cap ? c0 * 4 : 0;    // speculative first chunk, in the row

  // every lane runs the same number of rounds (whole wavefronts reduce together)
  const int64_t rounds = (work + stride - 1) / stride;
  for (int64_t rd = 0; rd < rounds; ++rd) {
    const int64_t w = rd * stride + (int64_t)bis * MRS_BD + tid;
    const bool active = w < work;
    const int64_t grp = active ? (w >> log2QS) : 0;     // (item, set) index
    const int64_t item = grp / gcount;
    const int gl = (int)(grp - item * gcount);
    const int g = g0 + gl;
    const int wp = (int)(item % Wp);
    const int64_t tmp = item / Wp;
    const int hp = (int)(tmp % Hp);
    const int bb = (int)(tmp / Hp);
    const int ho = hp * geo.pool + q / geo.pool;
    const int wo = wp * geo.pool + q % geo.pool;
    const E* trow = tab + gl;

    A accr = A(0);
    if (!ONE)
      for (int k = 0; k < n; ++k) acc_lane[k * MRS_BD] = A(0);
    if (active) {
      // the lane's taps t0, t0 + tstep, ... walked with a rolling prefetch: the
      // count and first chunk of the next MRS_AHEAD taps are in flight while a
      // tap is processed (ring slots are compile-time after unrolling)
      int64_t prow[MRS_AHEAD + 1];
      int pcnt[MRS_AHEAD + 1];
      Chunk<T> first[MRS_AHEAD + 1];
      auto prefetch = [&](int u, int slot) {
        const int t = t0 + u * tstep;
        prow[slot] = -1;
        pcnt[slot] = 0;
        if (t < T_) {
          const int ky = t / geo.KW, kx = t - ky * geo.KW;
          const int hy = ho * geo.S + ky - geo.P, wx = wo * geo.S + kx - geo.P;
          if (hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W) {
            const int64_t pr = ((int64_t)bb * geo.H + hy) * geo.W + wx;
            prow[slot] = pr;
            pcnt[slot] = min(lcnt[pr], geo.C);
            // the row holds cap >= 4*ceil(C/4) entries: this chunk is in bounds
            first[slot].load(lidx + pr * geo.cap, lval + pr * geo.cap, jfirst);
          }
        }
      };
#pragma unroll
      for (int u = 0; u < MRS_AHEAD; ++u) prefetch(u, u);
#pragma unroll
      for (int u = 0; u < MRS_TAPS; ++u) {
        if (u + MRS_AHEAD < MRS_TAPS) prefetch(u + MRS_AHEAD, (u + MRS_AHEAD) % (MRS_AHEAD + 1));
        const int sl = u % (MRS_AHEAD + 1);
        if (prow[sl] >= 0 && c0 * 4 < pcnt[sl]) {
          const uint16_t* li = lidx + prow[sl] * geo.cap;
          const T* lv = lval + prow[sl] * geo.cap;
          const int sbase = (t0 + u * tstep) * geo.C;
          const int m = pcnt[sl];
          Chunk<T> cur = first[sl];
          int c = c0;
          while (true) {
            const int cn = c + cstep;
            const bool more = cn * 4 < m;
            Chunk<T> nxt;
            if (more) nxt.load(li, lv, cn * 4);          // next chunk in flight
            mrs_chunk<T, A, ONE>(cur, m - c * 4, sbase, trow, gcount, acc_lane, accr);
            if (!more) break;
            cur = nxt;
            c = cn;
          }
        }
      }
    }
    if (ONE) acc_lane[0] = accr;
    wave_sync();                                        // partial sums of the group visible
    // lane r of the group finishes kids k = r, r + QS, ...: sum the slices of
    // each sub-pixel, take the max over the sub-pixels, add the bias
    for (int k = r; k < n; k += QS) {
      A m = A(0);
      for (int qq = 0; qq < nq; ++qq) {
        A a = A(0);
        for (int t = 0; t < S; ++t) a += acc[k * MRS_BD + gbase_lane + qq * S + t];
        m = (qq == 0 || a > m) ? a : m;
      }
      if (active) {
        if (bias) m += bias[g * n + k];
        y[item * geo.c_out + g * n + k] = m;
      }
    }
    wave_sync();                                        // before the accumulators are reused
  }
}

// Sparse-dense layer with a dense input (Section 3.1; Section 4 runs the first
// layer this way because its input is dense): dense weights (n == 1), one
// wavefront per output item and 64 sets (= output channels) per wavefront,
// persistent over items.  Each lane keeps its channel's KH*KW*C weights in
// registers; the input patch of an item (at most 64 values) is loaded by the
// wavefront, then every input value is broadcast from its lane as a scalar
// operand of the multiply-adds.  Geometry is compile-time.
template <typename T, typename A, int KH, int KW, int C, int STR, int POOL>
__global__ __launch_bounds__(256) void conv_dense_n1(const T* __restrict__ x,
                                                     const T* __restrict__ pval,
                                                     const A* __restrict__ bias,
                                                     A* __restrict__ y, ConvGeom geo,
                                                     int64_t items) {
  constexpr int R = KH * KW * C;
  constexpr int PH = (POOL - 1) * STR + KH;
  constexpr int PW = (POOL - 1) * STR + KW;
  static_assert(PH * PW * C <= 64, "patch must fit one wavefront");
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  A w[R];
#pragma unroll
  for (int i = 0; i < R; ++i) w[i] = (A)pval[i * 64 + lane];
  const A b = bias ? bias[lane] : A(0);
  const int Hp = geo.Ho / POOL, Wp = geo.Wo / POOL;
  const int c = lane % C, pp = lane / C, py = pp / PW, px = pp % PW;
  for (int64_t it = wave; it < items; it += nwaves) {
    const int wp = (int)(it % Wp);
    const int64_t tmp = it / Wp;
    const int hp = (int)(tmp % Hp);
    const int bb = (int)(tmp / Hp);
    const int hy = hp * POOL * STR - geo.P + py, wx = wp * POOL * STR - geo.P + px;
    A xv = A(0);
    if (pp < PH * PW && hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W)
      xv = (A)x[(((int64_t)bb * geo.H + hy) * geo.W + wx) * C + c];
    A best = A(0);
#pragma unroll
    for (int q = 0; q < POOL * POOL; ++q) {
      const int oy = (q / POOL) * STR, ox = (q % POOL) * STR;
      A a = b;
#pragma unroll
      for (int i = 0; i < R; ++i) {
        const int ci = i % C, t = i / C;
        const int src = ((oy + t / KW) * PW + (ox + t % KW)) * C + ci;
        const A xs = __builtin_bit_cast(A, __builtin_amdgcn_readlane(__builtin_bit_cast(int, xv), src));
        a += xs * w[i];
      }
      best = (q == 0 || a > best) ? a : best;
    }
    y[it * 64 + lane] = best;
  }
}

// Same computation with runtime geometry (any shape within the limits the
// host checks: n == 1, 64 channels, r <= 32, patch <= 64 values).
template <typename T, typename A>
__global__ __launch_bounds__(256) void conv_dense_n1_rt(const T* __restrict__ x,
                                                        const T* __restrict__ pval,
                                                        const A* __restrict__ bias,
                                                        A* __restrict__ y, ConvGeom geo,
                                                        int64_t items) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int R = geo.KH * geo.KW * geo.C;
  const int ph = (geo.pool - 1) * geo.S + geo.KH;
  const int pw = (geo.pool - 1) * geo.S + geo.KW;
  const A b = bias ? bias[lane] : A(0);
  const int Hp = geo.Ho / geo.pool, Wp = geo.Wo / geo.pool;
  const int c = lane % geo.C, pp = lane / geo.C, py = pp / pw, px = pp % pw;
  for (int64_t it = wave; it < items; it += nwaves) {
    const int wp = (int)(it % Wp);
    const int64_t tmp = it / Wp;
    const int hp = (int)(tmp % Hp);
    const int bb = (int)(tmp / Hp);
    const int hy = hp * geo.pool * geo.S - geo.P + py, wx = wp * geo.pool * geo.S - geo.P + px;
    A xv = A(0);
    if (pp < ph * pw && hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W)
      xv = (A)x[(((int64_t)bb * geo.H + hy) * geo.W + wx) * geo.C + c];
    A best = A(0);
    for (int q = 0; q < geo.pool * geo.pool; ++q) {
      const int oy = (q / geo.pool) * geo.S, ox = (q % geo.pool) * geo.S;
      A a = b;
      for (int i = 0; i < R; ++i) {
        const int ci = i % geo.C, t = i / geo.C;
        const int src = ((oy + t / geo.KW) * pw + (ox + t % geo.KW)) * geo.C + ci;
        const A xs = __builtin_bit_cast(A, __builtin_amdgcn_readlane(__builtin_bit_cast(int, xv), src));
        a += xs * (A)pval[i * 64 + lane];
      }
      best = (q == 0 || a > best) ? a : best;
    }
    y[it * 64 + lane] = best;
  }
}

}  // namespace cs
