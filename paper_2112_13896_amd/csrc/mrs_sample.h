// One sample per workgroup: Multiply, Route and Sum (Section 3.2 steps 3-5)
// and k-WTA (Section 3.3.3, applied to the whole output vector) for a layer
// whose output is one vector per sample - a linear layer, or a convolution
// whose window is the whole input map (a linear layer after a conv layer) -
// with a packed table too large for LDS.
//
//  * the sample's (index, value) lists are staged in LDS as one flat entry
//    list (pixel order, then list order); entry (pixel p, index c) uses table
//    row p*C + c, the window's taps being the map's pixels;
//  * a job (slice s, set g) runs over the entries s, s + S, s + 2S, ...: it
//    reads aug[row][g] straight from global memory (the lanes of a wavefront
//    read one contiguous row segment; the table stays in L2), SAMPLE_BATCH
//    entries in flight, and routes each product to its own accumulator
//    acc[s][kid][g] in LDS; the S slices' accumulators are summed at the end;
//  * k-WTA over the sums row: each thread holds KEYS consecutive keys; the
//    k-th largest key is fixed 8 bits at a time below the bits all keys share,
//    with a 256-bin LDS histogram and a workgroup scan over the bins, and
//    workgroup prefix sums give the ties' ranks (lower index wins) and the
//    winners' positions in the emitted list.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kwta_kernels.h"
#include "mrs_kernels.h"

namespace cs {

constexpr int SAMPLE_BD = 1024;                    // threads per workgroup
constexpr int SAMPLE_MAX_ROW = 2048;               // k-WTA row limit (KEYS per thread)
constexpr int SAMPLE_KEYS = SAMPLE_MAX_ROW / SAMPLE_BD;
constexpr int SAMPLE_BATCH = 8;                    // table entries a job has in flight
constexpr int SAMPLE_MISC = 64;                    // ints of LDS scratch (scans, results)
constexpr int SAMPLE_MAX_SLICES = 16;              // slices per set (bounds the final sum)

struct SampleArgs {
  int npix;          // pixels (taps) per sample, <= SAMPLE_BD
  int S;             // entry slices per set
  int jobs;          // S * G
  int k;             // k-WTA winners; < 0: none (sums only)
  int shift;
  int write_sums;
  uint32_t off_row, off_ent, off_val, off_pix, off_hist, off_misc;   // LDS byte offsets (acc at 0)
};

// Exclusive prefix sum of one int per thread over the workgroup; *total gets
// the sum.  ws: SAMPLE_BD / 64 ints.  Barriers inside (call uniformly).
__device__ __forceinline__ int sample_scan(int v, int* ws, int* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) ws[wv] = incl;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SAMPLE_BD / 64; ++w) {
    const int s = ws[w];
    base += (w < wv) ? s : 0;
    tot += s;
  }
  *total = tot;
  __syncthreads();
  return base + incl - v;
}

template <typename T, typename A, typename TO>
__global__ __launch_bounds__(SAMPLE_BD) void mrs_sample(const uint16_t* __restrict__ lidx,
                                                        const T* __restrict__ lval,
                                                        const int32_t* __restrict__ lcnt,
                                                        const typename Aug<T>::type* __restrict__ aug,
                                                        const A* __restrict__ bias,
                                                        A* __restrict__ y, TO* __restrict__ out,
                                                        ListOut lo, ConvGeom geo, SampleArgs sa) {
  using E = typename Aug<T>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int n = geo.n, G = geo.G, C = geo.C, c_out = geo.c_out, cap = geo.cap;
  const int npix = sa.npix, S = sa.S;
  const int64_t item = blockIdx.x;
  A* acc = reinterpret_cast<A*>(smem);                              // [S][n][G]
  A* row = reinterpret_cast<A*>(smem + sa.off_row);                 // [c_out]
  int* erow = reinterpret_cast<int*>(smem + sa.off_ent);            // [npix * cap]
  A* eval = reinterpret_cast<A*>(smem + sa.off_val);                // [npix * cap]
  int2* pix = reinterpret_cast<int2*>(smem + sa.off_pix);           // [npix] (entry offset, count)
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem + sa.off_hist); // [256]
  int* misc = reinterpret_cast<int*>(smem + sa.off_misc);

  // ---- stage the lists: counts and offsets, then the entries (coalesced)
  int c = 0;
  if (tid < npix) {
    c = lcnt[item * npix + tid];
    c = c < 0 ? 0 : (c > cap ? cap : c);
  }
  int tot = 0;
  const int e0 = sample_scan(c, misc, &tot);
  if (tid < npix) pix[tid] = make_int2(e0, c);
  for (int e = tid; e < S * c_out; e += SAMPLE_BD) acc[e] = A(0);
  __syncthreads();
  {
    const int64_t base = item * npix * cap;
    for (int e = tid; e < npix * cap; e += SAMPLE_BD) {
      const int p = e / cap, j = e - (e / cap) * cap;
      const int2 pc = pix[p];
      if (j < pc.y) {
        erow[pc.x + j] = p * C + lidx[base + e];
        eval[pc.x + j] = (A)lval[base + e];
      }
    }
  }
  __syncthreads();

  // ---- multiply, route, sum
  for (int jb = tid; jb < sa.jobs; jb += SAMPLE_BD) {
    const int s = jb / G, g = jb - (jb / G) * G;
    A* accj = acc + s * c_out + g;                                  // + kid * G
    for (int e = s; e < tot; e += S * SAMPLE_BATCH) {
      E te[SAMPLE_BATCH];
      A xv[SAMPLE_BATCH];
#pragma unroll
      for (int j = 0; j < SAMPLE_BATCH; ++j) {
        const int ej = e + j * S;
        const int ec = ej < tot ? ej : tot - 1;                     // a staged entry
        te[j] = aug[(int64_t)erow[ec] * G + g];
        xv[j] = ej < tot ? eval[ec] : A(0);
      }
#pragma unroll
      for (int j = 0; j < SAMPLE_BATCH; ++j)
        route_add<A>(accj + Aug<T>::kid(te[j]) * G, xv[j] * (A)Aug<T>::value(te[j]));
    }
  }
  __syncthreads();
  // the slices' sums + bias; channel g*n + kid sits at acc[s][kid][g]
  for (int o = tid; o < c_out; o += SAMPLE_BD) {
    const int g = o / n, kd = o - (o / n) * n;
    A v = bias ? bias[o] : A(0);
    for (int s = 0; s < S; ++s) v += acc[s * c_out + kd * G + g];
    row[o] = v;
    if (sa.write_sums) y[item * c_out + o] = v;
  }
  if (sa.k < 0) return;                                             // uniform
  __syncthreads();

  // ---- k-WTA over the row: thread t holds keys [KEYS*t, KEYS*t + KEYS)
  const int i0 = tid * SAMPLE_KEYS;
  uint32_t key[SAMPLE_KEYS];
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) {
    const bool in = i0 + j < c_out;
    key[j] = order_key(row[in ? i0 + j : 0]);
    if (in) {
      kmin = key[j] < kmin ? key[j] : kmin;
      kmax = key[j] > kmax ? key[j] : kmax;
    }
  }
  {
    const int lane = tid & 63, wv = tid >> 6;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const uint32_t a = __shfl_xor(kmin, off, 64), b = __shfl_xor(kmax, off, 64);
      kmin = a < kmin ? a : kmin;
      kmax = b > kmax ? b : kmax;
    }
    uint32_t* wmm = reinterpret_cast<uint32_t*>(misc) + SAMPLE_BD / 64;   // [2][waves]
    if (lane == 0) {
      wmm[wv] = kmin;
      wmm[SAMPLE_BD / 64 + wv] = kmax;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < SAMPLE_BD / 64; ++w) {
      kmin = wmm[w] < kmin ? wmm[w] : kmin;
      kmax = wmm[SAMPLE_BD / 64 + w] > kmax ? wmm[SAMPLE_BD / 64 + w] : kmax;
    }
  }
  const int k = sa.k;
  uint32_t thr = 0u;   // keys > thr win, and the first `need` keys == thr
  int need = 0;
  if (k >= c_out) {
    need = c_out;
  } else if (k > 0) {
    const uint32_t diff = kmin ^ kmax;
    thr = kmax;
    need = k;
    if (diff != 0u) {
      int rem = 32 - __builtin_clz(diff);                          // bits below the shared prefix
      uint32_t pmask = rem == 32 ? 0u : ~((1u << rem) - 1u);
      uint32_t prefix = kmax & pmask;
      int nd = k;   // invariant: at least nd keys match (prefix, pmask); nd - 1 of them rank above
      int* res = misc + SAMPLE_MISC - 2;
      while (rem > 0) {                                             // uniform
        const int width = rem < 8 ? rem : 8;
        const int sh = rem - width;
        const uint32_t dmask = (1u << width) - 1u;
        if (tid < 256) hist[tid] = 0u;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < SAMPLE_KEYS; ++j)
          if (i0 + j < c_out && (key[j] & pmask) == prefix)
            __hip_atomic_fetch_add(&hist[(key[j] >> sh) & dmask], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_WORKGROUP);
        __syncthreads();
        // thread t < 256 takes bin 255 - t: the scan counts the keys in higher bins
        const int bin = 255 - tid;
        const int hc = tid < 256 ? (int)hist[bin] : 0;
        int all = 0;
        const int above = sample_scan(hc, misc, &all);
        if (hc > 0 && above < nd && nd <= above + hc) {
          res[0] = bin;
          res[1] = above;
        }
        __syncthreads();
        nd -= res[1];
        prefix |= (uint32_t)res[0] << sh;
        pmask |= dmask << sh;
        rem = sh;
        __syncthreads();
      }
      thr = prefix;
      need = nd;
    }
  }
  // ---- winners: key > thr, or key == thr among the first `need` such keys
  int ties_t = 0;
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) ties_t += (i0 + j < c_out && key[j] == thr) ? 1 : 0;
  int ntie = 0;
  const int tie0 = sample_scan(ties_t, misc, &ntie);
  int win_t = 0;
  bool win[SAMPLE_KEYS];
  A wv[SAMPLE_KEYS];
  {
    int tr = tie0;
#pragma unroll
    for (int j = 0; j < SAMPLE_KEYS; ++j) {
      const bool in = i0 + j < c_out;
      const bool eq = in && key[j] == thr;
      win[j] = k > 0 && in && (key[j] > thr || (eq && tr < need));
      tr += eq ? 1 : 0;
      wv[j] = row[in ? i0 + j : 0];
      // a list leaves out winners whose output value is 0
      if (lo.idx) win[j] = win[j] && kwta_out<A, TO>(wv[j], sa.shift) != TO(0);
      win_t += win[j] ? 1 : 0;
    }
  }
  if (lo.idx) {
    int total = 0;
    int pos = sample_scan(win_t, misc, &total);
    const int64_t ob = item * lo.cap;
#pragma unroll
    for (int j = 0; j < SAMPLE_KEYS; ++j) {
      if (win[j]) {
        lo.idx[ob + pos] = (uint16_t)(i0 + j);
        static_cast<TO*>(lo.val)[ob + pos] = kwta_out<A, TO>(wv[j], sa.shift);
        ++pos;
      }
    }
    if (tid == 0) lo.cnt[item] = total;
  } else {
#pragma unroll
    for (int j = 0; j < SAMPLE_KEYS; ++j) {
      const int i = i0 + j;
      if (i < c_out) out[item * c_out + i] = win[j] ? kwta_out<A, TO>(wv[j], sa.shift) : TO(0);
    }
  }
}

}  // namespace cs
