// Input-stationary Multiply, Route and Sum (Section 3.2 steps 3-5) for int8
// convolutions with stride 1 on maps small enough that a band of output rows
// - every column and every channel - fits in LDS, followed by the 2x2
// max-pool, bias, k-WTA (Section 3.3.3) and the next layer's lists, all in
// one kernel.
//
// Each non-zero input (pixel, channel c, value x) and each packed set g
// visits the taps (ky, kx) whose output lies in the band: the product of x
// and the packed weight of slot (ky*KW + kx)*C + c goes to the accumulator of
// output (iy + P - ky, ix + P - kx), channel g*n + kid (the slot's Kernel ID).
// Every (non-zero, tap, output) triple belongs to exactly one band, so the
// products are those of the gather form, each formed once.  Accumulators are
// shared by all lanes and updated with LDS atomics: integer sums are exact in
// any order, so the result does not depend on timing.
//
//  * staging: the band's input rows (with the window halo) are staged as one
//    flat entry list (pixel order), the table with the Kernel ID stored as a
//    byte offset (kid * 4) in each entry's high byte;
//  * compute: job = (entry, group of GPL sets); the tap row ky runs over the
//    rows any lane of the wavefront has in the band, the KW taps of a row are
//    unrolled, the next row's table words are read before the current row's
//    atomics (LDS operations complete in order, so a read issued after the
//    atomics would wait for them); lanes whose output is outside the band or
//    the map are masked off;
//  * epilogue: 16 lanes per pooled item (four items per wavefront), each
//    lane KPL consecutive channels: the 2x2 max + bias, the k-WTA threshold
//    by a bit search with 16-lane DPP counts, the winners as a list (ties to
//    the lower index) or densely.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "mrs_sample.h"
#include "wave_ops.h"

#include <type_traits>

namespace cs {

constexpr int SCAT_BD = 1024;        // threads per workgroup
constexpr int SCAT_PRE = 4;          // list entries per thread loaded up front
constexpr int SCAT_TAB = 4;          // 16-byte table pieces per thread in flight
constexpr int SCAT_MAX_KH = 16;
static_assert(SCAT_BD == SAMPLE_BD, "the workgroup scan is sized for SAMPLE_BD threads");

struct ScatterArgs {
  int BR;            // conv output rows per band (a multiple of the pool size)
  int bands;         // bands per image
  int guard;         // accumulator entries before and after the band tile
  int ostride;       // accumulator words per output pixel: c_out + 16, so that
                     // neighbouring outputs' channels fall in different banks
  int k, shift, write_sums;
  uint32_t off_tab, off_ent, off_pix, off_bias, off_misc;   // LDS byte offsets (accumulators at 0)
  FastDiv fd_gpc;    // / (G / GPL)
  FastDiv fd_bands;  // / bands
  FastDiv fd_wp;     // / pooled width
  FastDiv fd_cap;    // / list capacity
  FastDiv fd_w;      // / input width
};

// The workgroup body for workgroup index blk (SCAT_BD threads).
template <typename TO, int KW, int GPL, int M>
__device__ __forceinline__ void scatter_body(const uint16_t* __restrict__ lidx,
                                             const int8_t* __restrict__ lval,
                                             const int32_t* __restrict__ lcnt,
                                             const uint16_t* __restrict__ aug,
                                             const int32_t* __restrict__ bias,
                                             int32_t* __restrict__ y, TO* __restrict__ out,
                                             const ListOut& lo, const ConvGeom& geo,
                                             const ScatterArgs& sc, uint32_t blk) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int H = geo.H, W = geo.W, C = geo.C, G = geo.G, n = geo.n, P = geo.P;
  const int Wo = geo.Wo, c_out = geo.c_out, cap = geo.cap, pool = geo.pool;
  const uint32_t img = fdiv(blk, sc.fd_bands);
  const int band = (int)(blk - img * (uint32_t)sc.bands);
  const int oy0 = band * sc.BR;
  const int nrows = min(sc.BR, geo.Ho - oy0);
  const int iy0 = max(oy0 - P, 0);
  const int iy1 = min(oy0 + nrows - 1 - P + geo.KH, H);            // exclusive
  const int npix = (iy1 - iy0) * W;                                // <= SCAT_BD (host)
  const int ne = npix * cap;

  int* accg = reinterpret_cast<int*>(smem);                        // [guard + tile + guard]
  int* acc = accg + sc.guard;                                      // [nrows][Wo][ostride]
  uint32_t* tab = reinterpret_cast<uint32_t*>(smem + sc.off_tab);  // [KH*KW][C][G] 16-bit entries
  int2* ent = reinterpret_cast<int2*>(smem + sc.off_ent);          // (ly<<24 | lx<<16 | c, x)
  int2* pix = reinterpret_cast<int2*>(smem + sc.off_pix);          // (entry offset, count)
  int* bias_s = reinterpret_cast<int*>(smem + sc.off_bias);        // [c_out]
  int* misc = reinterpret_cast<int*>(smem + sc.off_misc);

  // ---- global loads issued together: counts, the first list entries, table, bias
  const int64_t prow0 = ((int64_t)img * H + iy0) * W;
  int c = 0;
  if (tid < npix) c = lcnt[prow0 + tid];
  uint16_t pidx[SCAT_PRE];
  int8_t pval[SCAT_PRE];
  const int64_t lbase = prow0 * cap;
#pragma unroll
  for (int u = 0; u < SCAT_PRE; ++u) {
    const int e = u * SCAT_BD + tid;
    const int ec = e < ne ? e : ne - 1;                            // ne >= 1 (host)
    pidx[u] = lidx[lbase + ec];
    pval[u] = lval[lbase + ec];
  }
  // the table copied as it is ([tap][c][set] 16-bit entries), Kernel IDs
  // turned into byte offsets kid * 4 (kid < 32, so the byte holds it); with
  // two sets per lane the second set's byte is (n + kid) * 4, its channel's
  // offset from the first set's channel 0 (n + kid < 64)
  const int gpc = G / GPL;
  {
    const uint32_t hi_add = GPL == 2 ? (uint32_t)n << 26 : 0u;
    auto kid4 = [hi_add](uint32_t w) {
      return ((w & 0x00FF00FFu) | ((w & 0x1F001F00u) << 2)) + hi_add;
    };
    const int nw = geo.KH * KW * C * G / 2;                         // words; R*G even (host)
    const int n16 = nw / 4;                                         // 16-byte pieces
    const su32x4* src = reinterpret_cast<const su32x4*>(aug);
    su32x4* dst = reinterpret_cast<su32x4*>(tab);
    for (int b0 = 0; b0 < n16; b0 += SCAT_BD * SCAT_TAB) {          // loads issued together
      su32x4 v[SCAT_TAB];
#pragma unroll
      for (int u = 0; u < SCAT_TAB; ++u) {
        const int e = b0 + u * SCAT_BD + tid;
        v[u] = src[e < n16 ? e : n16 - 1];
      }
#pragma unroll
      for (int u = 0; u < SCAT_TAB; ++u) {
        const int e = b0 + u * SCAT_BD + tid;
        if (e < n16) {
          su32x4 t;
          t.x = kid4(v[u].x);
          t.y = kid4(v[u].y);
          t.z = kid4(v[u].z);
          t.w = kid4(v[u].w);
          dst[e] = t;
        }
      }
    }
    for (int e = n16 * 4 + tid; e < nw; e += SCAT_BD)                // the tail words
      tab[e] = kid4(reinterpret_cast<const uint32_t*>(aug)[e]);
  }
  for (int o = tid; o < c_out; o += SCAT_BD) bias_s[o] = bias ? bias[o] : 0;
  c = c < 0 ? 0 : (c > cap ? cap : c);
  int tot = 0;
  const int e0 = sample_scan(c, misc, &tot);
  if (tid < npix) pix[tid] = make_int2(e0, c);
  {
    const int nacc = 2 * sc.guard + nrows * Wo * sc.ostride;       // allocated rounded up to 4
    su32x4* a4 = reinterpret_cast<su32x4*>(accg);
    const su32x4 z = {0u, 0u, 0u, 0u};
    for (int e = tid; e < (nacc + 3) / 4; e += SCAT_BD) a4[e] = z;
  }
  __syncthreads();
  // ---- the entries into LDS in (pixel, list) order
  auto put = [&](int e, int ix16, int x) {
    const int p = (int)fdiv((uint32_t)e, sc.fd_cap), j = e - p * cap;
    const int2 pc = pix[p];
    if (j < pc.y) {
      const int ly = (int)fdiv((uint32_t)p, sc.fd_w), lx = p - ly * W;
      ent[pc.x + j] = make_int2((ly << 24) | (lx << 16) | ix16, x);
    }
  };
#pragma unroll
  for (int u = 0; u < SCAT_PRE; ++u) {
    const int e = u * SCAT_BD + tid;
    if (e < ne) put(e, pidx[u], pval[u]);
  }
  for (int e = SCAT_PRE * SCAT_BD + tid; e < ne; e += SCAT_BD) put(e, lidx[lbase + e], lval[lbase + e]);
  __syncthreads();
  CS_STAMP(5);

  // ---- multiply, route, sum
  const int njobs = tot * gpc;
  const int ost = sc.ostride;                                      // words per output pixel
  const int row_b = Wo * ost * 4;                                  // one output row of the tile
  const int col_b = ost * 4;
  const uint32_t acc_b = (uint32_t)(sc.guard * 4);                 // byte offset of acc in accg
  const uint32_t tap_b = (uint32_t)(C * G * 2);                    // one tap of the table
  unsigned char* accb = reinterpret_cast<unsigned char*>(accg);
  const unsigned char* tabb = reinterpret_cast<const unsigned char*>(tab);
  for (int jb0 = 0; jb0 < njobs; jb0 += SCAT_BD) {                 // uniform
    const int jb = jb0 + tid;
    const bool live = jb < njobs;
    const int jc = live ? jb : 0;
    const int e = (int)fdiv((uint32_t)jc, sc.fd_gpc);
    const int gq = jc - e * gpc;
    const int2 en = ent[e];
    const int x = en.y;
    const int ly = (int)((uint32_t)en.x >> 24), lx = (en.x >> 16) & 0xFF, ch = en.x & 0xFFFF;
    const int g = gq * GPL;
    // tap rows with an output row in the band: oy - oy0 = ly + iy0 + P - ky - oy0
    const int dy = ly + iy0 + P - oy0;
    int klo = dy - nrows + 1, khi = dy;
    klo = klo < 0 ? 0 : klo;
    khi = khi > geo.KH - 1 ? geo.KH - 1 : khi;
    if (!live) {
      klo = geo.KH;
      khi = -1;
    }
    // the wavefront's rows (uniform), each lane adding only on its own
    const int wlo = (int)wave_min_u32((uint32_t)klo);
    const int whi = (int)wave_max_u32((uint32_t)(khi + 1)) - 1;
    if (wlo > whi) continue;                                        // uniform
    // the value per tap column: x, or 0 where the output column is outside the map
    int xk[KW];
#pragma unroll
    for (int kx = 0; kx < KW; ++kx) xk[kx] = (unsigned)(lx + P - kx) < (unsigned)Wo ? x : 0;
    // byte offsets of the outputs (row dy - wlo, column lx + P - kx) plus the
    // set's channels, one per tap column; one tap row lower is row_b less
    uint32_t bk[KW];
#pragma unroll
    for (int kx = 0; kx < KW; ++kx)
      bk[kx] = acc_b + (uint32_t)((dy - wlo) * row_b + (lx + P - kx) * col_b + g * n * 4);
    const unsigned char* tp0 = tabb + (uint32_t)((ch * G + g) * 2);
    // the table words of a tap row are read one row ahead, before the atomics
    // of the current row (LDS operations complete in order, so a read issued
    // after them would wait for them); two register sets alternate
    using TW = typename std::conditional<GPL == 2, uint32_t, uint16_t>::type;
    auto load_row = [&](uint32_t (&w)[KW], int ky) {
      const unsigned char* rp = tp0 + (uint32_t)(ky * KW) * tap_b;
#pragma unroll
      for (int kx = 0; kx < KW; ++kx) w[kx] = *reinterpret_cast<const TW*>(rp + kx * tap_b);
    };
    // lanes whose output is outside the band or the map are masked off (the
    // LDS cycles an atomic costs grow with its active lanes); the entry's
    // Kernel-ID bytes are the offsets within the output pixel
    auto add_row = [&](const uint32_t (&w)[KW], int ky) {
      const bool vy = ky >= klo && ky <= khi;
#pragma unroll
      for (int kx = 0; kx < KW; ++kx) {
        if (vy && xk[kx] != 0) {
          CS_COUNT_PRODUCTS_ADD(GPL);
          const uint32_t wk = w[kx];
          __hip_atomic_fetch_add(reinterpret_cast<int*>(accb + bk[kx] + ((wk >> 8) & 0xFFu)),
                                 __mul24(xk[kx], (int)(int8_t)(wk & 0xFFu)), __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_WORKGROUP);
          if constexpr (GPL == 2)
            __hip_atomic_fetch_add(reinterpret_cast<int*>(accb + bk[kx] + (wk >> 24)),
                                   __mul24(xk[kx], (int)(int8_t)((wk >> 16) & 0xFFu)),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
#pragma unroll
      for (int kx = 0; kx < KW; ++kx) {
        bk[kx] -= (uint32_t)row_b;
        asm volatile("" : "+v"(bk[kx]));   // kept per lane: one add per atomic address
      }
    };
    uint32_t wa[KW], wb[KW];
    load_row(wa, wlo);
    // wait for this first row here: with nothing pending on entry, the waits
    // inside the loop only cover the reads of the previous half-iteration
    __builtin_amdgcn_s_waitcnt(0xC07F);                             // lgkmcnt(0)
    for (int ky = wlo; ky <= whi; ky += 2) {                        // uniform
      load_row(wb, ky + 1 <= whi ? ky + 1 : ky);
      add_row(wa, ky);
      if (ky + 1 > whi) break;
      load_row(wa, ky + 2 <= whi ? ky + 2 : ky + 1);
      add_row(wb, ky + 1);
    }
  }
  __syncthreads();
  CS_STAMP(6);

  // ---- epilogue: 16 lanes per pooled item, KPL consecutive channels per lane
  constexpr int KPL = 4 * M;                                        // c_out <= 64 * M (host)
  const int Wp = Wo / pool, Hp = geo.Ho / pool;
  const int nitems = (nrows / pool) * Wp;
  const int r16 = lane & 15;
  for (int ib = wv * 4; ib < nitems; ib += SCAT_BD / 16) {          // uniform per wavefront
    const int it = ib + (lane >> 4);
    const bool live = it < nitems;
    const int itc = live ? it : ib;
    const int pr = (int)fdiv((uint32_t)itc, sc.fd_wp), pc = itc - pr * Wp;
    const int* base = acc + ((pr * pool) * Wo + pc * pool) * ost + r16 * KPL;
    int v[KPL];
#pragma unroll
    for (int q = 0; q < KPL / 4; ++q) {
      su32x4 a = *reinterpret_cast<const su32x4*>(base + 4 * q);
      if (pool == 2) {
        const su32x4 b = *reinterpret_cast<const su32x4*>(base + 4 * q + ost);
        const su32x4 d = *reinterpret_cast<const su32x4*>(base + 4 * q + Wo * ost);
        const su32x4 e = *reinterpret_cast<const su32x4*>(base + 4 * q + Wo * ost + ost);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = (uint32_t)max(max((int)a[i], (int)b[i]), max((int)d[i], (int)e[i]));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int chn = r16 * KPL + 4 * q + i;
        v[4 * q + i] = chn < c_out ? (int)a[i] + bias_s[chn] : 0;
      }
    }
    const int64_t row = ((int64_t)img * Hp + oy0 / pool + pr) * Wp + pc;
    if (sc.write_sums && live) {
#pragma unroll
      for (int j = 0; j < KPL; ++j)
        if (r16 * KPL + j < c_out) y[row * c_out + r16 * KPL + j] = v[j];
    }
    if (sc.k >= 0) kwta_row16<int32_t, TO, KPL>(v, c_out, sc.k, sc.shift, live, lo, out, row);
  }
}

template <typename TO, int KW, int GPL, int M>
__global__ __launch_bounds__(SCAT_BD) void mrs_scatter(const uint16_t* __restrict__ lidx,
                                                       const int8_t* __restrict__ lval,
                                                       const int32_t* __restrict__ lcnt,
                                                       const uint16_t* __restrict__ aug,
                                                       const int32_t* __restrict__ bias,
                                                       int32_t* __restrict__ y,
                                                       TO* __restrict__ out, ListOut lo,
                                                       ConvGeom geo, ScatterArgs sc) {
  scatter_body<TO, KW, GPL, M>(lidx, lval, lcnt, aug, bias, y, out, lo, geo, sc, blockIdx.x);
}

// Two layers and a third in one launch, one workgroup per image: a convolution
// whose band is the whole image writes its k-WTA lists (int8) to lo; after a
// workgroup barrier (which orders the workgroup's global stores before its
// loads) the same workgroup runs the next layer, a window over the whole
// pooled map (one output vector per image), on those lists, with its own
// k-WTA lists lo2 and the last linear layer nx on its winners.
template <int KW, int GPL, int M>
__global__ __launch_bounds__(SCAT_BD) void mrs_scatter_sample(
    const uint16_t* __restrict__ lidx, const int8_t* __restrict__ lval,
    const int32_t* __restrict__ lcnt, const uint16_t* __restrict__ aug,
    const int32_t* __restrict__ bias, int32_t* __restrict__ y, ListOut lo, ConvGeom geo,
    ScatterArgs sc, const uint16_t* __restrict__ aug2, const int32_t* __restrict__ bias2,
    int32_t* __restrict__ y2, ListOut lo2, ConvGeom geo2, SampleArgs sa2, NextLayer nx) {
  scatter_body<int8_t, KW, GPL, M>(lidx, lval, lcnt, aug, bias, y, nullptr, lo, geo, sc,
                                   blockIdx.x);
  __syncthreads();
  sample_body<int8_t, int32_t, int8_t>(lo.idx, static_cast<const int8_t*>(lo.val), lo.cnt, aug2,
                                       bias2, y2, nullptr, lo2, geo2, sa2, nx, blockIdx.x);
}

}  // namespace cs
