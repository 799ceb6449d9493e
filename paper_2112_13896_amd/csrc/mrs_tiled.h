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

#include "fastdiv.h"
#include "mrs_kernels.h"

namespace cs {

constexpr int MRS_BD = 256;     // threads per workgroup
constexpr int MRS_TAPS = 9;     // most taps one lane walks (host picks S accordingly)
constexpr int MRS_AHEAD = 2;    // taps prefetched ahead of the one being processed
constexpr int MRS_STAGE = 16;   // table entries a lane loads per batch while staging
constexpr int MRS_CHUNKS = 4;   // list chunks loaded together in single-tap layers

// The staged table keeps the global augmented entries unchanged (a copy).
template <typename T, bool ONE>
struct TabEntry {
  using type = typename Aug<T>::type;
};

struct TiledArgs {
  int S, log2S;      // slices per (item, set, sub-pixel), power of two
  int log2Q;         // sub-pixels on separate lanes: 0 (none) or 2 (2x2 pool)
  int Gs;            // sets per table slice (divides G, multiple of the sets per lane)
  int gslices;       // number of table slices; gridDim.x is a multiple of it
  int chunk_mode;    // 1: a single tap, slices split its list chunks
  int items;         // output items (pooled pixels when pooling)
  int vec_stage;     // 1: one slice, table bytes a multiple of 16, 16-byte aligned
  FastDiv fd_gs;     // / Gs
  FastDiv fd_units;  // / (Gs / sets per lane)
  FastDiv fd_wp;     // / pooled output width
  FastDiv fd_hp;     // / pooled output height
  FastDiv fd_kw;     // / kernel width
};

// Copy n16 16-byte words from global memory to LDS with MRS_COPY loads in
// flight per lane.  Every load is unconditional (a lane past the end reads the
// last word again), so the batch stays in registers and the loads overlap.
constexpr int MRS_COPY = 10;
__device__ __forceinline__ void copy16_to_lds(const uint4* __restrict__ src, uint4* dst, int n16) {
  if (n16 <= 0) return;
  const int tid = threadIdx.x;
  for (int base = 0; base < n16; base += MRS_BD * MRS_COPY) {
    uint4 v[MRS_COPY];
#pragma unroll
    for (int u = 0; u < MRS_COPY; ++u) {
      const int e = base + u * MRS_BD + tid;
      v[u] = src[e < n16 ? e : n16 - 1];
    }
#pragma unroll
    for (int u = 0; u < MRS_COPY; ++u) {
      const int e = base + u * MRS_BD + tid;
      if (e < n16) dst[e] = v[u];
    }
  }
}

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

// Entries of the staged table a lane reads at once: GB consecutive sets.
template <typename T, bool ONE, int GB>
struct __attribute__((aligned(GB * sizeof(typename TabEntry<T, ONE>::type)))) TabVec {
  typename TabEntry<T, ONE>::type e[GB];
};

// One 4-entry chunk of a list against the lane's GB sets.  All table reads of
// the chunk are issued before any is used; tail entries beyond the list
// (e >= lim) read row 0 and contribute a zero product, so there is no branch.
// The accumulator of (set j of the lane, kid) is acc[(j*n + kid)][lane].
template <typename T, typename A, bool ONE, int GB>
__device__ __forceinline__ void mrs_chunk(const Chunk<T>& ch, int lim,
                                          const unsigned char* tbase, uint32_t row_bytes,
                                          int n, A* acc_lane, A (&accr)[GB]) {
  using V = TabVec<T, ONE, GB>;
  V tv[4];
  A xv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ok = e < lim;
    const uint32_t c = ok ? (uint32_t)chunk_idx(ch.idx, e) : 0u;
    tv[e] = *reinterpret_cast<const V*>(tbase + __umul24(c, row_bytes));   // Multiply: row c
    xv[e] = ok ? (A)ch.v(e) : A(0);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if constexpr (ONE) {
#pragma unroll
      for (int j = 0; j < GB; ++j) accr[j] += xv[e] * (A)Aug<T>::value(tv[e].e[j]);   // Sum
    } else if constexpr (sizeof(T) == 1) {
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        // Route + Sum: LDS integer atomic into the entry's accumulator
        const auto te = tv[e].e[j];
        __hip_atomic_fetch_add(acc_lane + (Aug<T>::kid(te) + j * n) * MRS_BD,
                               xv[e] * Aug<T>::value(te), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    } else {
      // Route + Sum: the GB sets' accumulators are disjoint, so all GB reads
      // are issued before the writes
      A* p[GB];
      A a[GB];
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        p[j] = acc_lane + (Aug<T>::kid(tv[e].e[j]) + j * n) * MRS_BD;
        a[j] = *p[j];
      }
#pragma unroll
      for (int j = 0; j < GB; ++j) *p[j] = a[j] + xv[e] * Aug<T>::value(tv[e].e[j]);
    }
  }
}

template <typename T, typename A, bool ONE, int GB>
__global__ __launch_bounds__(MRS_BD) void mrs_tiled(const uint16_t* __restrict__ lidx,
                                                    const T* __restrict__ lval,
                                                    const int32_t* __restrict__ lcnt,
                                                    const typename Aug<T>::type* __restrict__ aug,
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
  const int gcount = ta.Gs;
  const int g0 = gsl * gcount;
  const int gunits = gcount / GB;

  A* acc = reinterpret_cast<A*>(smem);                  // [GB * n][MRS_BD]
  unsigned char* tab = smem + (size_t)GB * n * MRS_BD * sizeof(A);
  const uint32_t row_bytes = (uint32_t)(gcount * sizeof(E));

  // stage the augmented table of sets [g0, g0 + gcount): a copy of the rows'
  // slices, loads in batches of MRS_STAGE per lane so their latencies overlap
  const int total = R * gcount;
  if (ta.vec_stage) {
    // the whole table, contiguous: 16-byte copies
    copy16_to_lds(reinterpret_cast<const uint4*>(aug), reinterpret_cast<uint4*>(tab),
                  R * gcount * (int)sizeof(E) / 16);
  } else {
    for (int base = 0; base < total; base += MRS_BD * MRS_STAGE) {
      E v[MRS_STAGE];
#pragma unroll
      for (int u = 0; u < MRS_STAGE; ++u) {
        const int e0 = base + u * MRS_BD + tid;
        const int e = e0 < total ? e0 : total - 1;            // always a valid entry
        const int i = (int)fdiv((uint32_t)e, ta.fd_gs), gl = e - i * gcount;
        v[u] = aug[i * G + g0 + gl];
      }
#pragma unroll
      for (int u = 0; u < MRS_STAGE; ++u) {
        const int e = base + u * MRS_BD + tid;
        if (e < total) reinterpret_cast<E*>(tab)[e] = v[u];
      }
    }
  }
  // the slice's bias values next to the table (so the epilogue reads LDS)
  A* bias_s = reinterpret_cast<A*>(tab + ((size_t)R * gcount * sizeof(E) + 15) / 16 * 16);
  for (int k = tid; k < gcount * n; k += MRS_BD) bias_s[k] = bias ? bias[g0 * n + k] : A(0);
  __syncthreads();                                      // the only workgroup barrier

  const int S = ta.S;
  const int log2QS = ta.log2S + ta.log2Q;
  const int QS = 1 << log2QS;                           // lanes per (item, set unit)
  const int nq = 1 << ta.log2Q;
  const int nacc = GB * n;
  const int work = ta.items * gunits * QS;              // < 2^31 (host)
  const int stride = nbs * MRS_BD;
  A* acc_lane = acc + tid;
  const int gbase_lane = tid & ~(QS - 1);               // first lane of this (item, set unit)
  const int r = tid & (QS - 1);                         // rank inside the group
  const int s = r & (S - 1);                            // slice
  const int q = r >> ta.log2S;                          // 2x2 pool sub-pixel
  const int t0 = ta.chunk_mode ? 0 : s;                 // first tap of the lane
  const int tstep = ta.chunk_mode ? T_ : S;             // tap step (chunk mode: one tap)
  const int c0 = ta.chunk_mode ? s : 0;                 // first chunk of a tap
  const int cstep = ta.chunk_mode ? S : 1;
  const int jfirst = c0 * 4 < geo.cap ? c0 * 4 : 0;    // speculative first chunk, in the row
  const bool vec_out = QS == 1 && (nacc & 3) == 0 && (geo.c_out & 3) == 0;

  const int rounds = (work + stride - 1) / stride;      // same for every lane of the block
  for (int rd = 0; rd < rounds; ++rd) {
    const int w = rd * stride + bis * MRS_BD + tid;
    const bool active = w < work;
    const uint32_t grp = active ? (uint32_t)(w >> log2QS) : 0u;   // (item, set unit)
    const uint32_t item = fdiv(grp, ta.fd_units);
    const int gu = (int)(grp - item * (uint32_t)gunits);
    const int gfirst = g0 + gu * GB;                    // first set of the lane
    const uint32_t tmp = fdiv(item, ta.fd_wp);
    const int wp = (int)(item - tmp * ta.fd_wp.d);
    const uint32_t bbu = fdiv(tmp, ta.fd_hp);
    const int hp = (int)(tmp - bbu * ta.fd_hp.d);
    const int bb = (int)bbu;
    const int ho = hp * geo.pool + (q >> 1) * (geo.pool >> 1);
    const int wo = wp * geo.pool + (q & 1) * (geo.pool >> 1);
    const unsigned char* tcol = tab + (size_t)gu * GB * sizeof(E);

    A accr[GB];
#pragma unroll
    for (int j = 0; j < GB; ++j) accr[j] = A(0);
    if (!ONE)
      for (int k = 0; k < nacc; ++k) acc_lane[k * MRS_BD] = A(0);
    if (active) {
      // taps t0, t0 + tstep, ... with a rolling prefetch: the count and first
      // chunk of the next MRS_AHEAD taps are in flight while one is processed
      int prow[MRS_AHEAD + 1];
      int pcnt[MRS_AHEAD + 1];
      Chunk<T> first[MRS_AHEAD + 1];
      auto prefetch = [&](int u, int slot) {
        const int t = t0 + u * tstep;
        prow[slot] = -1;
        pcnt[slot] = 0;
        if (t < T_) {
          const int ky = (int)fdiv((uint32_t)t, ta.fd_kw), kx = t - ky * geo.KW;
          const int hy = ho * geo.S + ky - geo.P, wx = wo * geo.S + kx - geo.P;
          if (hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W) {
            const int pr = (bb * geo.H + hy) * geo.W + wx;       // < 2^31 (host)
            prow[slot] = pr;
            pcnt[slot] = min(lcnt[pr], geo.cap);
            // the row holds cap >= 4*ceil(C/4) entries: this chunk is in bounds
            const int off = pr * geo.cap;                      // < 2^31 (host)
            first[slot].load(lidx + off, lval + off, jfirst);
          }
        }
      };
      if (ta.chunk_mode) {
        // one tap: the count and the lane's first MRS_CHUNKS chunks (c0, c0 + S,
        // ...) are all issued before any of them is used (one round trip);
        // chunks past the row's capacity are not read
        int pr = -1;
        {
          const int hy = ho * geo.S - geo.P, wx = wo * geo.S - geo.P;
          if (hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W) pr = (bb * geo.H + hy) * geo.W + wx;
        }
        if (pr >= 0) {
          const int off = pr * geo.cap;
          const uint16_t* li = lidx + off;
          const T* lv = lval + off;
          const int mraw = lcnt[pr];
          Chunk<T> ch[MRS_CHUNKS];
#pragma unroll
          for (int z = 0; z < MRS_CHUNKS; ++z) {
            const int j = (c0 + z * cstep) * 4;
            if (j < geo.cap) ch[z].load(li, lv, j);
          }
          const int m = min(mraw, geo.cap);
#pragma unroll
          for (int z = 0; z < MRS_CHUNKS; ++z) {
            const int cz = c0 + z * cstep;
            if (cz * 4 < m)
              mrs_chunk<T, A, ONE, GB>(ch[z], m - cz * 4, tcol, row_bytes, n, acc_lane, accr);
          }
          // the rest of a long list, one chunk ahead
          int c = c0 + MRS_CHUNKS * cstep;
          if (c * 4 < m) {
            Chunk<T> cur;
            cur.load(li, lv, c * 4);
            while (true) {
              const int cn = c + cstep;
              const bool more = cn * 4 < m;
              Chunk<T> nxt;
              if (more) nxt.load(li, lv, cn * 4);
              mrs_chunk<T, A, ONE, GB>(cur, m - c * 4, tcol, row_bytes, n, acc_lane, accr);
              if (!more) break;
              cur = nxt;
              c = cn;
            }
          }
        }
      } else {
#pragma unroll
      for (int u = 0; u < MRS_AHEAD; ++u) prefetch(u, u);
#pragma unroll
      for (int u = 0; u < MRS_TAPS; ++u) {
        if (u + MRS_AHEAD < MRS_TAPS) prefetch(u + MRS_AHEAD, (u + MRS_AHEAD) % (MRS_AHEAD + 1));
        const int sl = u % (MRS_AHEAD + 1);
        if (prow[sl] >= 0 && c0 * 4 < pcnt[sl]) {
          const int off = prow[sl] * geo.cap;
          const uint16_t* li = lidx + off;
          const T* lv = lval + off;
          const unsigned char* tbase = tcol + (uint32_t)((t0 + u * tstep) * geo.C) * row_bytes;
          const int m = pcnt[sl];
          Chunk<T> cur = first[sl];
          int c = c0;
          while (true) {
            const int cn = c + cstep;
            const bool more = cn * 4 < m;
            Chunk<T> nxt;
            if (more) nxt.load(li, lv, cn * 4);          // next chunk in flight
            mrs_chunk<T, A, ONE, GB>(cur, m - c * 4, tbase, row_bytes, n, acc_lane, accr);
            if (!more) break;
            cur = nxt;
            c = cn;
          }
        }
      }
      }
    }
    if (ONE) {
#pragma unroll
      for (int j = 0; j < GB; ++j) acc_lane[j * MRS_BD] = accr[j];
    }
    wave_sync();                                        // partial sums of the group visible
    A* yrow = y + (item * (uint32_t)geo.c_out + (uint32_t)(gfirst * n));   // GB*n contiguous outputs
    if (vec_out) {
      // one lane per (item, set unit): 16-byte stores of 4 consecutive outputs
      for (int k = 0; k < nacc; k += 4) {
        A v4[4];
#pragma unroll
        for (int z = 0; z < 4; ++z) {
          v4[z] = acc_lane[(k + z) * MRS_BD];
          v4[z] += bias_s[(gfirst - g0) * n + k + z];
        }
        if (active) {
          if constexpr (sizeof(A) == 4 && sizeof(T) == 1)
            *reinterpret_cast<int4*>(yrow + k) = make_int4(v4[0], v4[1], v4[2], v4[3]);
          else
            *reinterpret_cast<float4*>(yrow + k) = make_float4(v4[0], v4[1], v4[2], v4[3]);
        }
      }
    } else {
      // lane r of the group finishes outputs kk = r, r + QS, ...: sum the slices
      // of each sub-pixel, max over the sub-pixels, add the bias
      for (int kk = r; kk < nacc; kk += QS) {
        A mv = A(0);
        for (int qq = 0; qq < nq; ++qq) {
          A a = A(0);
          for (int t = 0; t < S; ++t) a += acc[kk * MRS_BD + gbase_lane + qq * S + t];
          mv = (qq == 0 || a > mv) ? a : mv;
        }
        if (active) {
          mv += bias_s[(gfirst - g0) * n + kk];
          yrow[kk] = mv;
        }
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
                                                     const typename Aug<T>::type* __restrict__ aug,
                                                     const A* __restrict__ bias,
                                                     A* __restrict__ y, ConvGeom geo,
                                                     int items, FastDiv fd_wp, FastDiv fd_hp) {
  constexpr int R = KH * KW * C;
  constexpr int PH = (POOL - 1) * STR + KH;
  constexpr int PW = (POOL - 1) * STR + KW;
  static_assert(PH * PW * C <= 64, "patch must fit one wavefront");
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  A w[R];
#pragma unroll
  for (int i = 0; i < R; ++i) w[i] = (A)Aug<T>::value(aug[i * 64 + lane]);
  const A b = bias ? bias[lane] : A(0);
  const int c = lane % C, pp = lane / C, py = pp / PW, px = pp % PW;
  for (int it = (int)wave; it < items; it += (int)nwaves) {
    const uint32_t tmp = fdiv((uint32_t)it, fd_wp);
    const int wp = it - (int)(tmp * fd_wp.d);
    const uint32_t bbu = fdiv(tmp, fd_hp);
    const int hp = (int)(tmp - bbu * fd_hp.d);
    const int bb = (int)bbu;
    const int hy = hp * POOL * STR - geo.P + py, wx = wp * POOL * STR - geo.P + px;
    A xv = A(0);
    if (pp < PH * PW && hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W)
      xv = (A)x[((bb * geo.H + hy) * geo.W + wx) * C + c];
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
    y[it * 64 + lane] = best;                             // items * 64 < 2^31 (host)
  }
}

// Same computation with runtime geometry (any shape within the limits the
// host checks: n == 1, 64 channels, r <= 32, patch <= 64 values).
template <typename T, typename A>
__global__ __launch_bounds__(256) void conv_dense_n1_rt(const T* __restrict__ x,
                                                        const typename Aug<T>::type* __restrict__ aug,
                                                        const A* __restrict__ bias,
                                                        A* __restrict__ y, ConvGeom geo,
                                                        int items, FastDiv fd_wp, FastDiv fd_hp) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int R = geo.KH * geo.KW * geo.C;
  const int ph = (geo.pool - 1) * geo.S + geo.KH;
  const int pw = (geo.pool - 1) * geo.S + geo.KW;
  const A b = bias ? bias[lane] : A(0);
  const int c = lane % geo.C, pp = lane / geo.C, py = pp / pw, px = pp % pw;
  for (int it = (int)wave; it < items; it += (int)nwaves) {
    const uint32_t tmp = fdiv((uint32_t)it, fd_wp);
    const int wp = it - (int)(tmp * fd_wp.d);
    const uint32_t bbu = fdiv(tmp, fd_hp);
    const int hp = (int)(tmp - bbu * fd_hp.d);
    const int bb = (int)bbu;
    const int hy = hp * geo.pool * geo.S - geo.P + py, wx = wp * geo.pool * geo.S - geo.P + px;
    A xv = A(0);
    if (pp < ph * pw && hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W)
      xv = (A)x[((bb * geo.H + hy) * geo.W + wx) * geo.C + c];
    A best = A(0);
    for (int q = 0; q < geo.pool * geo.pool; ++q) {
      const int oy = (q / geo.pool) * geo.S, ox = (q % geo.pool) * geo.S;
      A a = b;
      for (int i = 0; i < R; ++i) {
        const int ci = i % geo.C, t = i / geo.C;
        const int src = ((oy + t / geo.KW) * pw + (ox + t % geo.KW)) * geo.C + ci;
        const A xs = __builtin_bit_cast(A, __builtin_amdgcn_readlane(__builtin_bit_cast(int, xv), src));
        a += xs * (A)Aug<T>::value(aug[i * 64 + lane]);
      }
      best = (q == 0 || a > best) ? a : best;
    }
    y[it * 64 + lane] = best;                             // items * 64 < 2^31 (host)
  }
}

}  // namespace cs
