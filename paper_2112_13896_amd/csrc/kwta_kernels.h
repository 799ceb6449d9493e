// k-WTA (Section 2.2.2: exactly the top k activations propagate; Section
// 3.3.3: global k-WTA over a whole vector, local k-WTA along the channels of
// one pixel).  Both variants are a per-row top-k here; a row is a sample or a
// pixel.
//
// Semantics: exactly k winners per row; equal values go to the lower index;
// fp32 compares numerically (-0.0 ties +0.0).  A value maps to an unsigned
// key whose integer order is the value order, so the search runs on integer
// keys: the threshold T is the k-th largest key, every key > T wins, and the
// first (k - #{key > T}) keys equal to T in index order win too.
//
// Two gfx950 kernels:
//  * kwta_lane  (row <= 64, k <= 32): one lane owns a row, staged through LDS
//    with a padded stride so the 64 lanes read 64 different banks.  The lane
//    keeps a descending top-K list by insertion (a max/min exchange per slot,
//    no branches), which yields T;
//  * kwta_wave  (row <= 2048): one wavefront owns a row, each lane holds up to
//    M keys in registers.  T is found by a radix select, most significant
//    digit first, in 9-bit digits over the bits below those every key of the
//    row shares: each pass builds a 512-bin histogram of the current digit in
//    the wavefront's own LDS bins (the histogram threshold search of Section
//    3.3.3 and Figure 10, repeated digit by digit so it is exact for 32-bit
//    keys), a DPP scan from the top bin finds the digit holding the k-th key,
//    and keys outside the prefix found so far go to a spare bin.  Ties are
//    ranked with a ballot + popcount in index order.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "wave_ops.h"

namespace cs {

__device__ __forceinline__ void wave_sync_kwta() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t order_key(int32_t v) { return (uint32_t)v ^ 0x80000000u; }
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;                    // -0.0 -> +0.0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Winner value to output: same type, or int32 -> int8 requantisation.
template <typename TI, typename TO>
__device__ __forceinline__ TO kwta_out(TI v, int shift);
template <>
__device__ __forceinline__ int32_t kwta_out<int32_t, int32_t>(int32_t v, int) { return v; }
template <>
__device__ __forceinline__ float kwta_out<float, float>(float v, int) { return v; }
template <>
__device__ __forceinline__ int8_t kwta_out<int32_t, int8_t>(int32_t v, int shift) {
  int32_t q = v >> shift;                           // arithmetic shift (floor)
  q = q < -127 ? -127 : (q > 127 ? 127 : q);
  return (int8_t)q;
}

// Optional list output: the winners of each row as (index, value) pairs in
// ascending index order, capacity `cap` per row, with winners whose output
// value is 0 left out (they contribute nothing downstream) - the form the
// next layer's multiply-route-sum reads (Figure 10: winners go on "along with
// their indices").  idx == nullptr selects the dense masked output instead.
struct ListOut {
  uint16_t* idx;
  void* val;
  int32_t* cnt;
  int cap;
};

// Radix select over a wavefront's keys: key[j] is element j*64 + lane of the
// row, elements >= c are not part of it, 0 < k < c.  Returns the k-th largest
// key T and sets *need to k minus the number of keys above T (the keys equal
// to T that win).  Keys are offset by the row minimum, then 9-bit digits are
// resolved from the top, as many passes as the offset range has bits / 9:
// each pass counts the keys that share the digits found so far into 512 LDS
// bins (the others into a spare bin per lane), and one inclusive scan over the
// lanes (lane l holds bins 8(63 - l) .. + 7, the highest first) finds the bin
// of the k-th.  hist: WAVE_HIST words of LDS owned by the wavefront.
constexpr int WAVE_BINS = 512;
constexpr int WAVE_HIST = WAVE_BINS + 64;

template <int M>
__device__ __forceinline__ uint32_t wave_kth_radix(const uint32_t (&key)[M], int c, int k,
                                                   int* need, uint32_t* hist) {
  typedef uint32_t u4_t __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & 63;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < M; ++j) {
    if (j * 64 + lane < c) {
      kmin = key[j] < kmin ? key[j] : kmin;
      kmax = key[j] > kmax ? key[j] : kmax;
    }
  }
  kmin = wave_min_u32(kmin);
  kmax = wave_max_u32(kmax);
  const uint32_t range = kmax - kmin;
  if (range == 0u) {
    *need = k;
    return kmin;
  }
  uint32_t ok[M];
#pragma unroll
  for (int j = 0; j < M; ++j) ok[j] = key[j] - kmin;
  int rem = 32 - __builtin_clz(range);
  int passes = (rem + 8) / 9;
  uint32_t prefix = 0u;
  int nd = k;
  const u4_t z = {0u, 0u, 0u, 0u};
  reinterpret_cast<u4_t*>(hist)[2 * lane] = z;
  reinterpret_cast<u4_t*>(hist)[2 * lane + 1] = z;
  const int spare = WAVE_BINS + lane;
  for (; passes > 0; --passes) {                                   // uniform
    const int width = (rem + passes - 1) / passes;
    const int sh = rem - width;
    const uint32_t hi = rem >= 32 ? 0u : (0xFFFFFFFFu << rem);
    const uint32_t lob = rem >= 32 ? 0u : (prefix << rem);
    wave_lds_order();
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const bool in = j * 64 + lane < c && (ok[j] & hi) == lob;
      const int bin = in ? (int)__builtin_amdgcn_ubfe(ok[j], (uint32_t)sh, (uint32_t)width) : spare;
      __hip_atomic_fetch_add(hist + bin, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    wave_lds_order();
    const int b0 = 8 * (63 - lane);
    const u4_t h0 = reinterpret_cast<const u4_t*>(hist + b0)[0];
    const u4_t h1 = reinterpret_cast<const u4_t*>(hist + b0)[1];
    reinterpret_cast<u4_t*>(hist + b0)[0] = z;                     // the next pass's bins
    reinterpret_cast<u4_t*>(hist + b0)[1] = z;
    const uint32_t hb[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
    int ls = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) ls += (int)hb[q];
    const int incl = (int)wave_incl_scan((uint32_t)ls, 0u, OpAdd{});
    const int above = incl - ls;
    int run = above, bin = b0, found = 0;
#pragma unroll
    for (int q = 7; q >= 0; --q) {
      const bool hit = !found && run + (int)hb[q] >= nd;
      bin = hit ? b0 + q : bin;
      run = (!found && !hit) ? run + (int)hb[q] : run;
      found |= hit;
    }
    const uint64_t fb = __ballot(above < nd && nd <= incl);        // exactly one lane
    const int f = __ffsll((unsigned long long)fb) - 1;
    prefix = (prefix << width) | (uint32_t)__builtin_amdgcn_readlane(bin, f);
    nd -= __builtin_amdgcn_readlane(run, f);
    rem = sh;
  }
  wave_lds_order();                                                // before the bins are reused
  *need = nd;
  return prefix + kmin;
}

constexpr int KWTA_LANE_ROWS = 128;   // rows (threads) per block of kwta_lane
constexpr int KWTA_BATCH = 16;        // tile elements a thread loads per batch

// LDS tile: KWTA_LANE_ROWS rows of c 32-bit words, stride c + 1.
template <typename TI, typename TO, int KMAX>
__global__ __launch_bounds__(KWTA_LANE_ROWS) void kwta_lane(const TI* __restrict__ in,
                                                            int64_t rows, int c, int k,
                                                            TO* __restrict__ out, int shift,
                                                            FastDiv fd_c, ListOut lo) {
  extern __shared__ __align__(16) unsigned char smem[];
  TI* tile = reinterpret_cast<TI*>(smem);
  const int stride = c + 1;
  const int tid = threadIdx.x;
  const int64_t row0 = (int64_t)blockIdx.x * KWTA_LANE_ROWS;
  const int64_t nrows64 = rows - row0 < KWTA_LANE_ROWS ? rows - row0 : KWTA_LANE_ROWS;
  const int nrows = (int)nrows64;
  const int nelem = nrows * c;
  const TI* src = in + row0 * c;
  for (int b0 = 0; b0 < nelem; b0 += KWTA_LANE_ROWS * KWTA_BATCH) {   // loads in flight together
    TI v[KWTA_BATCH];
#pragma unroll
    for (int u = 0; u < KWTA_BATCH; ++u) {
      const int e = b0 + u * KWTA_LANE_ROWS + tid;
      v[u] = e < nelem ? src[e] : TI(0);
    }
#pragma unroll
    for (int u = 0; u < KWTA_BATCH; ++u) {
      const int e = b0 + u * KWTA_LANE_ROWS + tid;
      if (e < nelem) {
        const int rr = (int)fdiv((uint32_t)e, fd_c);
        tile[rr * stride + (e - rr * c)] = v[u];
      }
    }
  }
  __syncthreads();

  uint32_t thr = 0;
  int need = 0;
  if (tid < nrows) {
    const TI* r = tile + tid * stride;
    uint32_t top[KMAX];
#pragma unroll
    for (int s = 0; s < KMAX; ++s) top[s] = 0u;
    for (int i = 0; i < c; ++i) {
      uint32_t x = order_key(r[i]);
#pragma unroll
      for (int s = 0; s < KMAX; ++s) {
        const uint32_t hi = top[s] > x ? top[s] : x;
        x = top[s] > x ? x : top[s];
        top[s] = hi;
      }
    }
    int gt = 0;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) thr = (s == k - 1) ? top[s] : thr;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) gt += (s < k && top[s] > thr) ? 1 : 0;
    need = k - gt;
  }
  if (lo.idx) {
    // list output: each lane writes its row's winners in index order
    if (tid < nrows) {
      const TI* r = tile + tid * stride;
      const int64_t row = row0 + tid;
      uint16_t* li = lo.idx + row * lo.cap;
      TO* lv = static_cast<TO*>(lo.val) + row * lo.cap;
      int pos = 0;
      for (int i = 0; i < c; ++i) {
        const TI v = r[i];
        const uint32_t x = order_key(v);
        bool win = false;
        if (k > 0) {
          if (x > thr) {
            win = true;
          } else if (x == thr && need > 0) {
            win = true;
            --need;
          }
        }
        const TO ov = kwta_out<TI, TO>(v, shift);
        if (win && ov != TO(0)) {
          li[pos] = (uint16_t)i;
          lv[pos] = ov;
          ++pos;
        }
      }
      lo.cnt[row] = pos;
    }
    return;                                             // no barrier follows
  }
  __syncthreads();
  // second pass, results written back in place (as TO in a TO-typed view)
  TO* otile = reinterpret_cast<TO*>(smem);
  const int ostride = (int)(stride * sizeof(TI) / sizeof(TO));
  if (tid < nrows) {
    TI* r = tile + tid * stride;
    TO* o = otile + tid * ostride;
    for (int i = 0; i < c; ++i) {
      const TI v = r[i];
      const uint32_t x = order_key(v);
      bool win = false;
      if (k > 0) {
        if (x > thr) {
          win = true;
        } else if (x == thr && need > 0) {
          win = true;
          --need;
        }
      }
      // o[i] never overlaps an r[j] read later: TO is not wider than TI
      o[i] = win ? kwta_out<TI, TO>(v, shift) : TO(0);
    }
  }
  __syncthreads();
  TO* dst = out + row0 * c;
  for (int e = tid; e < nelem; e += KWTA_LANE_ROWS) {
    const int rr = (int)fdiv((uint32_t)e, fd_c);
    dst[e] = otile[rr * ostride + (e - rr * c)];
  }
}

// k-WTA of one row held by one wavefront: lane l holds v[j] = element
// j*64 + l (elements >= c are not part of the row).  Winners: the k largest
// keys, ties to the lower index; written as the row's list (non-zero outputs
// in index order, ranked by ballot + popcount, and the count) or densely.
template <typename TI, typename TO, int M>
__device__ __forceinline__ void kwta_wave_row(const TI (&v)[M], int c, int k, int shift,
                                              const ListOut& lo, TO* __restrict__ out,
                                              int64_t row, uint32_t* hist) {
  const int lane = threadIdx.x & 63;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  const bool all_win = (k >= c);
  const bool none_win = (k == 0);
  uint32_t key[M];
#pragma unroll
  for (int j = 0; j < M; ++j) key[j] = j * 64 + lane < c ? order_key(v[j]) : 0u;
  int need = 0;
  uint32_t thr = 0u;
  if (!all_win && !none_win) thr = wave_kth_radix<M>(key, c, k, &need, hist);
  // ranks of the ties in index order (element index = j*64 + lane)
  int run = 0, lrun = 0;
#pragma unroll
  for (int j = 0; j < M; ++j) {
    const int e = j * 64 + lane;
    const bool valid = e < c;
    const bool eq = !all_win && !none_win && valid && key[j] == thr;
    const uint64_t b = __ballot(eq);
    const int rank = run + __popcll(b & below);
    run += __popcll(b);
    bool win;
    if (all_win) win = valid;
    else if (none_win) win = false;
    else win = valid && (key[j] > thr || (eq && rank < need));
    const TO ov = kwta_out<TI, TO>(v[j], shift);
    if (lo.idx) {
      // list output: non-zero winners, ranked in index order by ballot + popcount
      const bool put = win && ov != TO(0);
      const uint64_t pb = __ballot(put);
      if (put) {
        const int pos = lrun + __popcll(pb & below);
        lo.idx[row * lo.cap + pos] = (uint16_t)e;
        static_cast<TO*>(lo.val)[row * lo.cap + pos] = ov;
      }
      lrun += __popcll(pb);
    } else if (valid) {
      out[row * c + e] = win ? ov : TO(0);
    }
  }
  if (lo.idx && lane == 0) lo.cnt[row] = lrun;
}

// Exchanges within a quad of lanes (DPP quad permutations, no LDS).
__device__ __forceinline__ uint32_t quad_xor1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);   // [1,0,3,2]
}
__device__ __forceinline__ uint32_t quad_xor2(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);   // [2,3,0,1]
}
__device__ __forceinline__ int quad_excl_sum(int v, int qd) {
  // Hillis-Steele over the 4 lanes: from lane qd-1, then from lane qd-2
  int x = v;
  const int t1 = __builtin_amdgcn_update_dpp(0, x, 0x90, 0xF, 0xF, false);        // [0,0,1,2]
  x += qd >= 1 ? t1 : 0;
  const int t2 = __builtin_amdgcn_update_dpp(0, x, 0x40, 0xF, 0xF, false);        // [0,0,0,1]
  x += qd >= 2 ? t2 : 0;
  return x - v;
}

// Bitonic networks in registers (all indices compile-time): sort N keys
// descending; sort a bitonic sequence of N keys descending; and keep in a[]
// the N largest of two descending lists (a max against the reversed other
// list leaves a bitonic sequence holding them, which is then sorted).
template <int N>
__device__ __forceinline__ void bitonic_sort_desc(uint32_t (&a)[N]) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          const uint32_t x = a[i], y = a[l];
          const uint32_t hi = x > y ? x : y, lo = x > y ? y : x;
          const bool desc = (i & k) == 0;
          a[i] = desc ? hi : lo;
          a[l] = desc ? lo : hi;
        }
      }
}
// Eight keys: a 19-comparator network of depth 6 (Knuth, The Art of Computer
// Programming vol. 3, 5.3.4) in place of the 24 of the bitonic sort; by the
// 0-1 principle it sorts any input (all 256 0-1 inputs checked).
template <>
__device__ __forceinline__ void bitonic_sort_desc<8>(uint32_t (&a)[8]) {
  auto ce = [&](int i, int j) {
    const uint32_t x = a[i], y = a[j];
    a[i] = x > y ? x : y;
    a[j] = x > y ? y : x;
  };
  ce(0, 2); ce(1, 3); ce(4, 6); ce(5, 7);
  ce(0, 4); ce(1, 5); ce(2, 6); ce(3, 7);
  ce(0, 1); ce(2, 3); ce(4, 5); ce(6, 7);
  ce(2, 4); ce(3, 5);
  ce(1, 4); ce(3, 6);
  ce(1, 2); ce(3, 4); ce(5, 6);
}
template <int N>
__device__ __forceinline__ void bitonic_clean_desc(uint32_t (&a)[N]) {
#pragma unroll
  for (int j = N >> 1; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int l = i ^ j;
      if (l > i) {
        const uint32_t x = a[i], y = a[l];
        a[i] = x > y ? x : y;
        a[l] = x > y ? y : x;
      }
    }
}
template <int N>
__device__ __forceinline__ void top_merge_desc(uint32_t (&a)[N], const uint32_t (&b)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) a[i] = a[i] > b[N - 1 - i] ? a[i] : b[N - 1 - i];
  bitonic_clean_desc<N>(a);
}
// Keep the N largest of this lane's list and that of its DPP partner (CTRL: a
// permutation within each row of 16 lanes); both lists sorted descending.
template <int N, int CTRL>
__device__ __forceinline__ void row16_top_merge(uint32_t (&a)[N]) {
  uint32_t p[N];
#pragma unroll
  for (int s = 0; s < N; ++s) p[s] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)a[s], CTRL, 0xF, 0xF, false);
  top_merge_desc<N>(a, p);
}

// k-WTA of one row held by one row of 16 lanes (lanes 16q .. 16q + 15 of a
// wavefront hold one row each): lane r holds v[j] = element r*KPL + j
// (elements >= c are not part of the row).  The threshold T, the k-th largest
// key (keys offset by the row minimum), comes for k <= ROW16_TOPK from the
// lanes' sorted top lists merged over the row (partners at distance 1 and 2,
// then the mirrored lane of the half row and of the row: four DPP exchanges),
// else bit by bit below the row's range, counting with 16-lane DPP sums.
// Ties go to the lower index; the winners are written as the row's list
// (non-zero outputs in index order, and the count) or densely.  Every lane of
// the wavefront must be active; `live` rows write.
constexpr int ROW16_TOPK = 8;
template <typename TI, typename TO, int KPL>
__device__ __forceinline__ void kwta_row16(const TI (&v)[KPL], int c, int k, int shift, bool live,
                                           const ListOut& lo, TO* __restrict__ out, int64_t row) {
  const int r = threadIdx.x & 15;
  const int i0 = r * KPL;
  uint32_t key[KPL];
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    key[j] = order_key(v[j]);
    if (i0 + j < c) {
      kmin = key[j] < kmin ? key[j] : kmin;
      kmax = key[j] > kmax ? key[j] : kmax;
    }
  }
  kmin = row16_reduce(kmin, OpMin{});
  kmax = row16_reduce(kmax, OpMax{});
#pragma unroll
  for (int j = 0; j < KPL; ++j) key[j] = i0 + j < c ? key[j] - kmin : 0u;
  const uint32_t range = kmax - kmin;
  // winners: key > thr, and the first `need` keys (lowest indices) == thr
  uint32_t thr = 0u;
  int need = 0;
  if (k == 0) {
    thr = 0xFFFFFFFFu;
  } else if (k >= c) {
    need = c;
  } else if (range == 0u) {
    need = k;
  } else if (k <= ROW16_TOPK) {
    // keys outside the row are 0, the smallest key: with k < c they never
    // change the k-th largest
    uint32_t top[ROW16_TOPK];
#pragma unroll
    for (int s = 0; s < ROW16_TOPK; ++s) top[s] = 0u;
#pragma unroll
    for (int b0 = 0; b0 < KPL; b0 += ROW16_TOPK) {
      uint32_t blk[ROW16_TOPK];
#pragma unroll
      for (int s = 0; s < ROW16_TOPK; ++s) blk[s] = b0 + s < KPL ? key[b0 + s] : 0u;
      bitonic_sort_desc<ROW16_TOPK>(blk);
      top_merge_desc<ROW16_TOPK>(top, blk);
    }
    row16_top_merge<ROW16_TOPK, 0xB1>(top);                         // quad [1,0,3,2]
    row16_top_merge<ROW16_TOPK, 0x4E>(top);                         // quad [2,3,0,1]
    row16_top_merge<ROW16_TOPK, 0x141>(top);                        // half-row mirror
    row16_top_merge<ROW16_TOPK, 0x140>(top);                        // row mirror
#pragma unroll
    for (int s = 0; s < ROW16_TOPK; ++s) thr = (s == k - 1) ? top[s] : thr;
    int gt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) gt += (i0 + j < c && key[j] > thr) ? 1 : 0;
    need = k - (int)row16_reduce((uint32_t)gt, OpAdd{});
  } else {
    uint32_t T = 0u;
    for (int b = 31 - __builtin_clz(range); b >= 0; --b) {         // uniform within a row
      const uint32_t cand = T | (1u << b);
      int cnt = 0;
#pragma unroll
      for (int j = 0; j < KPL; ++j) cnt += (i0 + j < c && key[j] >= cand) ? 1 : 0;
      cnt = (int)row16_reduce((uint32_t)cnt, OpAdd{});
      if (cnt >= k) T = cand;
    }
    int gt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) gt += (i0 + j < c && key[j] > T) ? 1 : 0;
    thr = T;
    need = k - (int)row16_reduce((uint32_t)gt, OpAdd{});
  }
  // ranks of the ties and list positions, in index order
  int eq_l = 0;
#pragma unroll
  for (int j = 0; j < KPL; ++j) eq_l += (i0 + j < c && key[j] == thr) ? 1 : 0;
  int rank = row16_incl_sum(eq_l) - eq_l;
  bool win[KPL];
  TO ov[KPL];
  int put_l = 0;
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const bool in = i0 + j < c;
    const bool eq = in && key[j] == thr;
    win[j] = in && (key[j] > thr || (eq && rank < need));
    rank += eq ? 1 : 0;
    ov[j] = kwta_out<TI, TO>(v[j], shift);
    put_l += (win[j] && ov[j] != TO(0)) ? 1 : 0;
  }
  if (lo.idx) {
    const int incl = row16_incl_sum(put_l);
    const int total = (int)row16_reduce((uint32_t)put_l, OpAdd{});
    if (live) {
      int pos = incl - put_l;
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        if (win[j] && ov[j] != TO(0)) {
          lo.idx[row * lo.cap + pos] = (uint16_t)(i0 + j);
          static_cast<TO*>(lo.val)[row * lo.cap + pos] = ov[j];
          ++pos;
        }
      }
      if (r == 0) lo.cnt[row] = total;
    }
  } else if (live) {
#pragma unroll
    for (int j = 0; j < KPL; ++j)
      if (i0 + j < c) out[row * c + i0 + j] = win[j] ? ov[j] : TO(0);
  }
}

constexpr int KWTA_WAVE_WAVES = 4;   // wavefronts (rows) per block of kwta_wave

template <typename TI, typename TO, int M>
__global__ __launch_bounds__(64 * KWTA_WAVE_WAVES) void kwta_wave(const TI* __restrict__ in,
                                                                  int64_t rows, int c, int k,
                                                                  TO* __restrict__ out,
                                                                  int shift, ListOut lo) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem) + wv * WAVE_HIST;   // this wavefront's bins
  for (int64_t row = (int64_t)blockIdx.x * KWTA_WAVE_WAVES + wv; row < rows;
       row += (int64_t)gridDim.x * KWTA_WAVE_WAVES) {            // uniform across the wave
    TI v[M];
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const int e = j * 64 + lane;
      v[j] = e < c ? in[row * c + e] : TI(0);
    }
    kwta_wave_row<TI, TO, M>(v, c, k, shift, lo, out, row, hist);
  }
}

}  // namespace cs
