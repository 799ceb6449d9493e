// One wavefront per item: Multiply, Route and Sum (Section 3.2 steps 3-5)
// and k-WTA (Section 3.3.3) for a layer whose window is one tap (a 1x1
// convolution with stride 1, or a linear layer) with many items, each with a
// short list and a row of at most 2048 outputs.
//
//  * the workgroup stages the packed table (value + Kernel ID per slot) in LDS
//    once; after that its wavefronts work without workgroup barriers, each on
//    its own items;
//  * an item: its list is loaded into a wavefront-private LDS buffer; lane
//    (slice s, set g) takes the entries s, s + S, ... (S = 64 / G slices when
//    G <= 64, else one slice and the lane's sets g, g + 64, ...), reads the
//    table entry of each (entry, set) and routes the product into its own
//    accumulator acc[s][kid][g] (a column no other lane touches);
//  * lane l then gathers the outputs l, l + 64, ... (summing the slices, plus
//    bias) into a wavefront-private LDS row, and the wavefront runs k-WTA on
//    it (radix select with a wavefront-private LDS histogram), or writes the
//    sums.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "wave_ops.h"

namespace cs {

constexpr int ROWS_BD = 256;          // threads per workgroup
constexpr int ROWS_WAVES = ROWS_BD / 64;
constexpr int ROWS_ENT = 64;          // list entries staged per wavefront at a time
constexpr int ROWS_BATCH = 8;         // entries (or channels) a lane reads before it adds

struct RowsArgs {
  int S;              // entry slices per set (S * G <= 64), or 1 when G > 64
  int gpl;            // sets per lane (1, or ceil(G / 64) when G > 64)
  int ipw;            // items per workgroup
  int k;              // k-WTA winners; < 0: none (sums only)
  int shift;
  int write_sums;
  uint32_t off_acc;   // LDS byte offset of the wavefronts' accumulators (table at 0)
  uint32_t acc_words; // accumulator words per wavefront (S * c_out, rounded up to 4)
  uint32_t off_ent;   // LDS byte offset of the wavefronts' entry buffers
  uint32_t off_hist;  // LDS byte offset of the wavefronts' k-WTA histograms (512 words each)
  uint32_t off_row;   // LDS byte offset of the wavefronts' sums rows
  uint32_t off_bias;  // LDS byte offset of the bias (c_out values)
  uint32_t row_words; // words per sums row (c_out, rounded up to 4)
  FastDiv fd_g;       // / G
  FastDiv fd_n;       // / n
};

// Route a product into a lane-private accumulator (int32: LDS add without
// return; fp32: read-add-write, the lane being the only writer).
template <typename A>
__device__ __forceinline__ void rows_add(A* p, A v);
template <>
__device__ __forceinline__ void rows_add<int32_t>(int32_t* p, int32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <>
__device__ __forceinline__ void rows_add<float>(float* p, float v) {
  *p = *p + v;
}

template <typename T, typename A, typename TO>
__global__ __launch_bounds__(ROWS_BD) void mrs_rows(const uint16_t* __restrict__ lidx,
                                                    const T* __restrict__ lval,
                                                    const int32_t* __restrict__ lcnt,
                                                    const typename Aug<T>::type* __restrict__ aug,
                                                    const A* __restrict__ bias,
                                                    A* __restrict__ y, TO* __restrict__ out,
                                                    ListOut lo, ConvGeom geo, RowsArgs ra,
                                                    int64_t items) {
  using E = typename Aug<T>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int G = geo.G, n = geo.n, c_out = geo.c_out, cap = geo.cap;
  E* tab = reinterpret_cast<E*>(smem);                               // [R][G]
  A* acc = reinterpret_cast<A*>(smem + ra.off_acc) + wv * ra.acc_words;   // [S][n][G]
  int2* ent = reinterpret_cast<int2*>(smem + ra.off_ent) + wv * ROWS_ENT;  // (index, value bits)
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem + ra.off_hist) + wv * 512;   // k-WTA bins

  // ---- the table into LDS (16-byte pieces), once per workgroup
  {
    const int nb = geo.C * G * (int)sizeof(E);                      // R = C (one tap)
    const int n16 = nb / 16;
    const uint4* src = reinterpret_cast<const uint4*>(aug);
    uint4* dst = reinterpret_cast<uint4*>(tab);
    for (int b0 = 0; b0 < n16; b0 += ROWS_BD * 4) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = b0 + u * ROWS_BD + tid;
        v[u] = src[e < n16 ? e : n16 - 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = b0 + u * ROWS_BD + tid;
        if (e < n16) dst[e] = v[u];
      }
    }
    for (int e = n16 * 16 + tid; e < nb; e += ROWS_BD)              // the tail bytes
      reinterpret_cast<unsigned char*>(tab)[e] = reinterpret_cast<const unsigned char*>(aug)[e];
  }
  A* bias_s = reinterpret_cast<A*>(smem + ra.off_bias);             // [c_out]
  for (int o = tid; o < c_out; o += ROWS_BD) bias_s[o] = bias ? bias[o] : A(0);
  __syncthreads();

  // this lane's job: slice s, first set g0 (sets g0, g0 + 64, ... when gpl > 1)
  const int S = ra.S;
  const int s = (int)fdiv((uint32_t)lane, ra.fd_g);
  const int g0 = lane - s * G;
  const bool job = s < S;                                           // lanes past S*G idle
  A* rowb = reinterpret_cast<A*>(smem + ra.off_row) + wv * ra.row_words;   // [c_out]

  const int64_t it0 = (int64_t)blockIdx.x * ra.ipw;
  const int64_t it1 = it0 + ra.ipw < items ? it0 + ra.ipw : items;
  // the next item's count and first ROWS_ENT list entries are loaded while
  // the current item is processed (their global latency hidden)
  int cnt_n = 0;
  uint16_t pi_n = 0;
  T pv_n = T(0);
  auto prefetch = [&](int64_t itn) {
    if (itn < it1) {
      cnt_n = lcnt[itn];
      const int j = lane < cap ? lane : cap - 1;
      pi_n = lidx[itn * cap + j];
      pv_n = lval[itn * cap + j];
    }
  };
  prefetch(it0 + wv);
  for (int64_t it = it0 + wv; it < it1; it += ROWS_WAVES) {         // uniform per wavefront
    int cnt = __builtin_amdgcn_readfirstlane(cnt_n);
    cnt = cnt < 0 ? 0 : (cnt > cap ? cap : cnt);
    const uint16_t pi = pi_n;
    const T pv = pv_n;
    prefetch(it + ROWS_WAVES);
    {
      const int na = (int)ra.acc_words;
      typedef uint32_t a4_t __attribute__((ext_vector_type(4)));
      const a4_t z = {0u, 0u, 0u, 0u};
      for (int e = lane; e < na / 4; e += 64) reinterpret_cast<a4_t*>(acc)[e] = z;
    }
    const int64_t lb = it * cap;
    for (int j0 = 0; j0 < cnt; j0 += ROWS_ENT) {                    // uniform
      const int nb = cnt - j0 < ROWS_ENT ? cnt - j0 : ROWS_ENT;
      if (lane < nb) {
        const uint16_t ix = j0 == 0 ? pi : lidx[lb + j0 + lane];
        const T v = j0 == 0 ? pv : lval[lb + j0 + lane];
        A av = (A)v;
        ent[lane] = make_int2((int)ix, __builtin_bit_cast(int, av));
      }
      wave_lds_sync();                                              // entries and zeros visible
      if (job) {
        A* accs = acc + s * c_out;
        for (int q = 0; q < ra.gpl; ++q) {
          const int g = g0 + 64 * q;
          if (g < G) {
            // batches of ROWS_BATCH entries: every read of a batch is issued
            // before its adds (LDS operations complete in order)
            for (int e = s; e < nb; e += S * ROWS_BATCH) {
              int2 en[ROWS_BATCH];
#pragma unroll
              for (int u = 0; u < ROWS_BATCH; ++u) {
                const int ee = e + u * S;
                en[u] = ent[ee < nb ? ee : nb - 1];
              }
              E w[ROWS_BATCH];
#pragma unroll
              for (int u = 0; u < ROWS_BATCH; ++u) w[u] = tab[en[u].x * G + g];
#pragma unroll
              for (int u = 0; u < ROWS_BATCH; ++u) {
                const A x = e + u * S < nb ? __builtin_bit_cast(A, en[u].y) : A(0);
                rows_add<A>(accs + Aug<T>::kid(w[u]) * G + g, x * (A)Aug<T>::value(w[u]));
              }
            }
          }
        }
      }
      wave_lds_sync();                                              // before the buffer is reused
    }
    // the row: output ch = g*n + kid sums the slices' acc[s][kid][g], plus
    // bias (from LDS), ROWS_BATCH channels per lane at a time
    for (int c0 = 0; c0 < c_out; c0 += 64 * ROWS_BATCH) {
      A a[ROWS_BATCH];
#pragma unroll
      for (int u = 0; u < ROWS_BATCH; ++u) {
        const int ch = c0 + u * 64 + lane;
        const int chc = ch < c_out ? ch : c_out - 1;
        const int g = (int)fdiv((uint32_t)chc, ra.fd_n), kd = chc - g * n;
        const A* p = acc + kd * G + g;
        A t = bias_s[chc];
        for (int ss = 0; ss < S; ++ss) t += p[ss * c_out];
        a[u] = t;
      }
#pragma unroll
      for (int u = 0; u < ROWS_BATCH; ++u) {
        const int ch = c0 + u * 64 + lane;
        if (ch < c_out) {
          rowb[ch] = a[u];
          if (ra.write_sums) y[it * c_out + ch] = a[u];
        }
      }
    }
    if (ra.k >= 0) {
      wave_lds_sync();                                              // the row
      kwta_wave_radix<A, TO>(rowb, c_out, ra.k, ra.shift, lo, out, it, hist);
    }
    wave_lds_sync();                                                // before acc and the row are reused
  }
}

}  // namespace cs
