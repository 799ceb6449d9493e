// One sample per workgroup: Multiply, Route and Sum (Section 3.2 steps 3-5)
// and k-WTA (Section 3.3.3, applied to the whole output vector) for a layer
// whose output is one vector per sample - a linear layer, or a convolution
// whose window is the whole input map (a linear layer after a conv layer).
// The packed table is read from global memory (it may be far larger than
// LDS); each workgroup reads only the rows its sample's non-zeros select.
//
//  * the sample's (index, value) lists are staged in LDS as one flat entry
//    list (pixel order, then list order); entry (pixel p, index c) uses table
//    row p*C + c, the window's taps being the map's pixels;
//  * a job (slice s, set g) runs over one contiguous range of entries: it
//    reads aug[row][g] straight from global memory (the lanes of a wavefront
//    read one contiguous row segment; the table stays in L2), SAMPLE_BATCH
//    entries in flight, and routes each product to its own accumulator
//    acc[s][kid][g] in LDS; the slices' accumulators are summed at the end;
//  * k-WTA over the sums row: each thread holds KEYS consecutive keys, offset
//    by the row's smallest key; the k-th largest is fixed SAMPLE_DIGIT bits
//    per pass from the top of the row's range, with a double-buffered LDS
//    histogram (one pass = atomics, barrier, one wavefront finds the digit
//    with a DPP scan, barrier), and one workgroup prefix sum of packed counts
//    gives the ties' ranks (lower index wins) and the winners' positions in
//    the emitted list.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "wave_ops.h"

namespace cs {

constexpr int SAMPLE_BD = 1024;                    // threads per workgroup
constexpr int SAMPLE_MAX_ROW = 2048;               // k-WTA row limit (KEYS per thread)
constexpr int SAMPLE_KEYS = SAMPLE_MAX_ROW / SAMPLE_BD;
constexpr int SAMPLE_BATCH = 16;                   // table entries a job has in flight
constexpr int SAMPLE_PRE = 2;                      // list entries per thread loaded up front
constexpr int SAMPLE_DIGIT = 8;                    // k-WTA radix digit (bits per pass)
constexpr int SAMPLE_BINS = 1 << SAMPLE_DIGIT;     // 4 per lane of one wavefront
constexpr int SAMPLE_MISC = 64;                    // ints of LDS scratch (scans, results)
constexpr int SAMPLE_MAX_SLICES = 16;              // slices per set (bounds the final sum)
constexpr int SAMPLE_ENT_PAD = SAMPLE_BATCH;       // entry-array slack read past the end

struct SampleArgs {
  int npix;          // pixels (taps) per sample, <= SAMPLE_BD
  int S;             // entry slices per set, at most (fewer when the lists are short)
  int k;             // k-WTA winners; < 0: none (sums only)
  int shift;
  int write_sums;
  uint32_t off_row, off_ent, off_val, off_pix, off_hist, off_misc;   // LDS byte offsets (acc at 0)
  FastDiv fd_cap;    // / list capacity
  FastDiv fd_g;      // / G
  FastDiv fd_n;      // / n
};

// An optional linear layer without k-WTA fed by this layer's winners (the
// last layer of a chain): its packed table aug [c_out of this layer][G]
// (int8 entries), bias [c_out] and sums y [rows][c_out].  aug == nullptr:
// none.  int8 chains only.
constexpr int NX_MAXG = 16;   // next-layer sets whose rows a thread loads ahead

struct NextLayer {
  const uint16_t* aug;
  const int32_t* bias;
  int32_t* y;
  int G, n, c_out;
  uint32_t off_acc;  // LDS byte offset of its c_out accumulators
};

// Exclusive prefix sum of one int per thread over the workgroup; *total gets
// the sum.  ws: SAMPLE_BD / 64 ints.  Barriers inside (call uniformly, with
// every thread active).
__device__ __forceinline__ int sample_scan(int v, int* ws, int* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int incl = (int)wave_incl_scan((uint32_t)v, 0u, OpAdd{});
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

template <typename A>
__device__ __forceinline__ A acc_from_bits(uint32_t b);
template <>
__device__ __forceinline__ int32_t acc_from_bits<int32_t>(uint32_t b) { return (int32_t)b; }
template <>
__device__ __forceinline__ float acc_from_bits<float>(uint32_t b) { return __uint_as_float(b); }

typedef uint32_t su32x4 __attribute__((ext_vector_type(4)));

// The workgroup body for sample `item` (SAMPLE_BD threads).
template <typename T, typename A, typename TO>
__device__ __forceinline__ void sample_body(const uint16_t* __restrict__ lidx,
                                            const T* __restrict__ lval,
                                            const int32_t* __restrict__ lcnt,
                                            const typename Aug<T>::type* __restrict__ aug,
                                            const A* __restrict__ bias, A* __restrict__ y,
                                            TO* __restrict__ out, const ListOut& lo,
                                            const ConvGeom& geo, const SampleArgs& sa,
                                            const NextLayer& nx, int64_t item) {
  using E = typename Aug<T>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = geo.n, G = geo.G, C = geo.C, c_out = geo.c_out, cap = geo.cap;
  const int npix = sa.npix, ne = npix * cap;
  A* acc = reinterpret_cast<A*>(smem);                              // [S][n][G]
  A* row = reinterpret_cast<A*>(smem + sa.off_row);                 // [c_out]
  int* erow = reinterpret_cast<int*>(smem + sa.off_ent);            // [ne + pad]
  A* eval = reinterpret_cast<A*>(smem + sa.off_val);                // [ne + pad]
  int2* pix = reinterpret_cast<int2*>(smem + sa.off_pix);           // [npix] (entry offset, count)
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem + sa.off_hist); // [2][SAMPLE_BINS]
  int* misc = reinterpret_cast<int*>(smem + sa.off_misc);

  // ---- global loads issued together: pixel tid's count, this thread's
  // first SAMPLE_PRE list entries, the bias of its outputs
  const int64_t base = item * ne;
  int c = 0;
  if (tid < npix) c = lcnt[item * npix + tid];
  uint16_t pidx[SAMPLE_PRE];
  T pval[SAMPLE_PRE];
#pragma unroll
  for (int u = 0; u < SAMPLE_PRE; ++u) {
    const int e = u * SAMPLE_BD + tid;
    const int ec = e < ne ? e : ne - 1;                             // ne >= 1
    pidx[u] = lidx[base + ec];
    pval[u] = lval[base + ec];
  }
  A bv[SAMPLE_KEYS];
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) {
    const int o = tid + j * SAMPLE_BD;
    bv[j] = (bias && o < c_out) ? bias[o] : A(0);
  }
  c = c < 0 ? 0 : (c > cap ? cap : c);
  int tot = 0;
  const int e0 = sample_scan(c, misc, &tot);
  // slices in use: enough for SAMPLE_BATCH entries per job, at most S
  int Sr = (tot + SAMPLE_BATCH - 1) / SAMPLE_BATCH;
  Sr = Sr < 1 ? 1 : (Sr > sa.S ? sa.S : Sr);
  // accumulator rows: integer sums are exact in any order, so every slice
  // adds into one row with LDS atomics; fp32 slices keep rows of their own
  // (a lane-private read-add-write, summed in slice order at the end)
  constexpr bool kShared = std::is_same<A, int32_t>::value;
  const int nrows = kShared ? 1 : Sr;
  if (tid < npix) pix[tid] = make_int2(e0, c);
  {
    su32x4* a4 = reinterpret_cast<su32x4*>(acc);
    const su32x4 z = {0u, 0u, 0u, 0u};
    for (int e = tid; e < (nrows * c_out + 3) / 4; e += SAMPLE_BD) a4[e] = z;
  }
  if (sa.k >= 0 && tid < SAMPLE_BINS) hist[tid] = 0u;               // first pass's bins
  __syncthreads();
  // ---- the entries into LDS in (pixel, list) order
#pragma unroll
  for (int u = 0; u < SAMPLE_PRE; ++u) {
    const int e = u * SAMPLE_BD + tid;
    if (e < ne) {
      const int p = (int)fdiv((uint32_t)e, sa.fd_cap), j = e - p * cap;
      const int2 pc = pix[p];
      if (j < pc.y) {
        erow[pc.x + j] = p * C + pidx[u];
        eval[pc.x + j] = (A)pval[u];
      }
    }
  }
  for (int e = SAMPLE_PRE * SAMPLE_BD + tid; e < ne; e += SAMPLE_BD) {
    const int p = (int)fdiv((uint32_t)e, sa.fd_cap), j = e - p * cap;
    const int2 pc = pix[p];
    if (j < pc.y) {
      erow[pc.x + j] = p * C + lidx[base + e];
      eval[pc.x + j] = (A)lval[base + e];
    }
  }
  __syncthreads();
  CS_STAMP(8);

  // ---- multiply, route, sum: job (s, g) takes the entries [s*per, s*per +
  // per) (per a multiple of 4: 16-byte LDS reads), all its table loads of a
  // batch in flight before the first product
  int per = (tot + Sr - 1) / Sr;
  per = (per + 3) & ~3;
  for (int jb = tid; jb < Sr * G; jb += SAMPLE_BD) {
    const int s = (int)fdiv((uint32_t)jb, sa.fd_g), g = jb - s * G;
    A* accj = acc + (kShared ? 0 : s * c_out) + g;                  // + kid * G
    const int eb = s * per;
    const int ee = eb + per < tot ? eb + per : tot;
    for (int e = eb; e < ee; e += SAMPLE_BATCH) {
      int er[SAMPLE_BATCH];
      uint32_t xb[SAMPLE_BATCH];
#pragma unroll
      for (int q = 0; q < SAMPLE_BATCH / 4; ++q) {
        const su32x4 r4 = *reinterpret_cast<const su32x4*>(erow + e + 4 * q);
        const su32x4 v4 = *reinterpret_cast<const su32x4*>(eval + e + 4 * q);
        er[4 * q] = (int)r4.x;
        er[4 * q + 1] = (int)r4.y;
        er[4 * q + 2] = (int)r4.z;
        er[4 * q + 3] = (int)r4.w;
        xb[4 * q] = v4.x;
        xb[4 * q + 1] = v4.y;
        xb[4 * q + 2] = v4.z;
        xb[4 * q + 3] = v4.w;
      }
      E te[SAMPLE_BATCH];
      CS_COUNT_PRODUCTS_ADD(min(SAMPLE_BATCH, ee - e));
#pragma unroll
      for (int j = 0; j < SAMPLE_BATCH; ++j)
        te[j] = aug[(int64_t)(e + j < ee ? er[j] : 0) * G + g];    // row 0 past the end
#pragma unroll
      for (int j = 0; j < SAMPLE_BATCH; ++j) {
        const A xv = e + j < ee ? acc_from_bits<A>(xb[j]) : A(0);
        route_add<A>(accj + Aug<T>::kid(te[j]) * G, xv * (A)Aug<T>::value(te[j]));
      }
    }
  }
  __syncthreads();
  CS_STAMP(9);
  // ---- the slices' sums + bias (channel g*n + kid sits at acc[s][kid][g]),
  // and the row's smallest and largest keys
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) {
    const int o = tid + j * SAMPLE_BD;
    if (o < c_out) {
      const int g = (int)fdiv((uint32_t)o, sa.fd_n), kd = o - g * n;
      A v = bv[j];
      for (int s = 0; s < nrows; ++s) v += acc[s * c_out + kd * G + g];
      row[o] = v;
      if (sa.write_sums) y[item * c_out + o] = v;
      const uint32_t kv = order_key(v);
      kmin = kv < kmin ? kv : kmin;
      kmax = kv > kmax ? kv : kmax;
    }
  }
  if (sa.k < 0) return;                                             // uniform
  kmin = wave_min_u32(kmin);
  kmax = wave_max_u32(kmax);
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

  CS_STAMP(10);
  // ---- k-WTA over the row: thread t holds keys [KEYS*t, KEYS*t + KEYS),
  // offset by the row's smallest key (order kept, fewer significant bits)
  const int i0 = tid * SAMPLE_KEYS;
  uint32_t key[SAMPLE_KEYS];
  A rv[SAMPLE_KEYS];
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) {
    const bool in = i0 + j < c_out;
    rv[j] = row[in ? i0 + j : 0];
    key[j] = in ? order_key(rv[j]) - kmin : 0u;
  }
  const int k = sa.k;
  const uint32_t range = kmax - kmin;
  // winners: key > thr, and the first `need` keys (lowest indices) == thr
  uint32_t thr = 0u;
  int need = 0;
  if (k == 0) {
    thr = 0xFFFFFFFFu;                                              // nothing exceeds it
  } else if (k >= c_out) {
    need = c_out;                                                   // every key >= 0 wins
  } else if (range == 0u) {
    need = k;                                                       // all equal
  } else {
    // the k-th largest offset key, SAMPLE_DIGIT bits per pass from the top;
    // the keys still in the running share the bits above `rem` with `prefix`
    int rem = 32 - __builtin_clz(range);
    uint32_t prefix = 0u;
    int nd = k;       // keys of the running prefix that must be >= the threshold
    int* res = misc + SAMPLE_MISC - 2;
    for (int pass = 0; rem > 0; ++pass) {                           // uniform
      const int width = rem < SAMPLE_DIGIT ? rem : SAMPLE_DIGIT;
      const int sh = rem - width;
      const uint32_t dmask = (1u << width) - 1u;
      uint32_t* h = hist + (pass & 1) * SAMPLE_BINS;
#pragma unroll
      for (int j = 0; j < SAMPLE_KEYS; ++j)
        if (i0 + j < c_out && (uint32_t)((uint64_t)key[j] >> rem) == prefix)
          __hip_atomic_fetch_add(&h[(key[j] >> sh) & dmask], 1u, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_WORKGROUP);
      if (tid < SAMPLE_BINS) hist[((pass + 1) & 1) * SAMPLE_BINS + tid] = 0u;   // next pass
      __syncthreads();
      if (wv == 0) {
        // lane l holds the 4 bins at 4*(63 - l) (lane 0 the highest), so an
        // inclusive scan over the lanes counts the keys in a lane's bins and
        // above; the one lane holding the nd-th largest key walks its bins
        const int b0 = 4 * (63 - lane);
        const su32x4 hb = *reinterpret_cast<const su32x4*>(h + b0);
        const int ls = (int)(hb.x + hb.y + hb.z + hb.w);
        const int incl = (int)wave_incl_scan((uint32_t)ls, 0u, OpAdd{});
        const int above = incl - ls;
        if (above < nd && nd <= incl) {
          int run = above, bin = b0, ab = above;
          if (run + (int)hb.w >= nd) {
            bin = b0 + 3;
          } else {
            run += (int)hb.w;
            if (run + (int)hb.z >= nd) {
              bin = b0 + 2;
            } else {
              run += (int)hb.z;
              if (run + (int)hb.y >= nd) {
                bin = b0 + 1;
              } else {
                run += (int)hb.y;
              }
            }
          }
          ab = run;
          res[0] = bin;
          res[1] = ab;
        }
      }
      __syncthreads();
      prefix = (prefix << width) | (uint32_t)res[0];
      nd -= res[1];
      rem = sh;
    }
    thr = prefix;
    need = nd;
  }

  // the next layer's accumulators start at zero (the scan's barriers order
  // this before its adds); the packed rows of the keys that can win (key >=
  // T) are loaded now, their latency hidden behind the scan and the lists
  int32_t* acc2 = reinterpret_cast<int32_t*>(smem + nx.off_acc);
  uint32_t pw[SAMPLE_KEYS][NX_MAXG / 2];                // two 16-bit entries per register
  if (nx.aug != nullptr) {
    for (int o = tid; o < nx.c_out; o += SAMPLE_BD) acc2[o] = 0;
    if (nx.G <= NX_MAXG) {
#pragma unroll
      for (int j = 0; j < SAMPLE_KEYS; ++j) {
        if (i0 + j < c_out && key[j] >= thr) {
          const uint16_t* r = nx.aug + (int64_t)(i0 + j) * nx.G;
#pragma unroll
          for (int g = 0; g < NX_MAXG; g += 2)
            pw[j][g / 2] = (g < nx.G ? (uint32_t)r[g] : 0u) |
                           ((g + 1 < nx.G ? (uint32_t)r[g + 1] : 0u) << 16);
        }
      }
    }
  }

  CS_STAMP(11);
  // ---- one scan: keys above the threshold (with a non-zero output, for
  // lists) and keys equal to it, packed as two 16-bit counts
  int gt_t = 0, eq_t = 0;
#pragma unroll
  for (int j = 0; j < SAMPLE_KEYS; ++j) {
    const bool in = i0 + j < c_out;
    const bool nz = !lo.idx || kwta_out<A, TO>(rv[j], sa.shift) != TO(0);
    gt_t += (in && key[j] > thr && nz) ? 1 : 0;
    eq_t += (in && key[j] == thr) ? 1 : 0;
  }
  int tot2 = 0;
  const int pre = sample_scan(gt_t | (eq_t << 16), misc, &tot2);
  int gt_before = pre & 0xFFFF, eq_before = pre >> 16;
  bool wins[SAMPLE_KEYS];
  if (lo.idx) {
    // keys equal to thr hold one value, so their outputs are all zero or all
    // non-zero: the thread holding the first tie tells the others through LDS
    const int64_t ob = item * lo.cap;
    int ntie_nz = 0;
    {
      int* tie_nz = misc + SAMPLE_MISC - 3;
      if (eq_before == 0 && eq_t > 0) {
#pragma unroll
        for (int j = SAMPLE_KEYS - 1; j >= 0; --j)
          if (i0 + j < c_out && key[j] == thr)
            *tie_nz = kwta_out<A, TO>(rv[j], sa.shift) != TO(0) ? 1 : 0;
      }
      __syncthreads();
      ntie_nz = (tot2 >> 16) > 0 ? *tie_nz : 0;
    }
#pragma unroll
    for (int j = 0; j < SAMPLE_KEYS; ++j) {
      const bool in = i0 + j < c_out;
      const bool eq = in && key[j] == thr;
      const bool win = in && (key[j] > thr || (eq && eq_before < need));
      const TO ov = kwta_out<A, TO>(rv[j], sa.shift);
      wins[j] = win;
      if (win && ov != TO(0)) {
        const int pos = gt_before + (ntie_nz ? (eq_before < need ? eq_before : need) : 0);
        lo.idx[ob + pos] = (uint16_t)(i0 + j);
        static_cast<TO*>(lo.val)[ob + pos] = ov;
      }
      gt_before += (in && key[j] > thr && ov != TO(0)) ? 1 : 0;
      eq_before += eq ? 1 : 0;
    }
    if (tid == 0) {
      const int ties = tot2 >> 16;
      lo.cnt[item] = (tot2 & 0xFFFF) + (ntie_nz ? (need < ties ? need : ties) : 0);
    }
  } else {
#pragma unroll
    for (int j = 0; j < SAMPLE_KEYS; ++j) {
      const int i = i0 + j;
      const bool eq = i < c_out && key[j] == thr;
      const bool win = i < c_out && (key[j] > thr || (eq && eq_before < need));
      wins[j] = win;
      if (i < c_out) out[item * c_out + i] = win ? kwta_out<A, TO>(rv[j], sa.shift) : TO(0);
      eq_before += eq ? 1 : 0;
    }
  }
  CS_STAMP(12);
  // ---- the next layer on the winners: a winner (channel i, output v) adds
  // v * value to the next layer's output g*n + kid for every set g of its
  // packed row i (integer sums: exact in any order)
  if constexpr (std::is_same<T, int8_t>::value) {
    if (nx.aug != nullptr) {
#pragma unroll
      for (int j = 0; j < SAMPLE_KEYS; ++j) {
        const int32_t ov = (int32_t)kwta_out<A, TO>(rv[j], sa.shift);
        if (wins[j] && ov != 0) {
          CS_COUNT_PRODUCTS_ADD(nx.G);
          if (nx.G <= NX_MAXG) {
#pragma unroll
            for (int g = 0; g < NX_MAXG; ++g) {
              const uint32_t w = (pw[j][g / 2] >> (16 * (g & 1))) & 0xFFFFu;
              if (g < nx.G)
                __hip_atomic_fetch_add(acc2 + g * nx.n + (int)(w >> 8),
                                       ov * (int)(int8_t)(w & 0xFFu), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
            }
          } else {
            const uint16_t* r = nx.aug + (int64_t)(i0 + j) * nx.G;
            for (int g = 0; g < nx.G; ++g) {
              const uint32_t w = r[g];
              __hip_atomic_fetch_add(acc2 + g * nx.n + (int)(w >> 8),
                                     ov * (int)(int8_t)(w & 0xFFu), __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_WORKGROUP);
            }
          }
        }
      }
      __syncthreads();
      for (int o = tid; o < nx.c_out; o += SAMPLE_BD)
        nx.y[item * nx.c_out + o] = acc2[o] + (nx.bias != nullptr ? nx.bias[o] : 0);
    }
  }
}

template <typename T, typename A, typename TO>
__global__ __launch_bounds__(SAMPLE_BD) void mrs_sample(const uint16_t* __restrict__ lidx,
                                                        const T* __restrict__ lval,
                                                        const int32_t* __restrict__ lcnt,
                                                        const typename Aug<T>::type* __restrict__ aug,
                                                        const A* __restrict__ bias,
                                                        A* __restrict__ y, TO* __restrict__ out,
                                                        ListOut lo, ConvGeom geo, SampleArgs sa,
                                                        NextLayer nx) {
  sample_body<T, A, TO>(lidx, lval, lcnt, aug, bias, y, out, lo, geo, sa, nx, blockIdx.x);
}

}  // namespace cs
