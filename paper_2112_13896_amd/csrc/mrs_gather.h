// Output-stationary Multiply, Route and Sum (Section 3.2 steps 3-5) for the
// second layer of the keyword-spotting chain: an int8 convolution, stride 1,
// on the 64-channel lists of the dense first layer, whose whole output map
// (every pixel and channel, int32) fits in LDS; followed by the 2x2 max-pool
// (or none), bias, k-WTA (Section 3.3.3) and the next layer's lists.
//
// Each lane owns one output pixel and one tap row ky and walks the KW input
// pixels of that row under its window; for every list entry (channel c, value
// x) of such a pixel and every packed set g the product of x and the weight
// of slot (ky*KW + kx)*C + c goes to the accumulator of its output pixel,
// channel g*n + kid.  The accumulators are laid out channel-major in blocks of
// 64 output pixels, [block][channel][64 pixels], so the 64 lanes of one add
// (64 consecutive pixels) fall in 64 different banks whatever their Kernel
// IDs; lanes of different tap rows meet on the same words and add with LDS
// integer atomics, exact in any order.  The table is split by pairs of sets,
// [pair][tap][channel] 32-bit words, so the lanes' reads of one tap hit the
// bank of their channel: equal channels share a word, different ones differ
// in bank.
//
//  * staging: the list entries as 16-bit (channel | value << 8) in cap = 8
//    slots per input pixel and the counts; the table with each set's Kernel
//    ID replaced by its output channel g*n + kid (so one shift gives the
//    accumulator row);
//  * compute: wavefront w < KW * NH: tap row w / NH, pixel block w % NH; the
//    table words of a pixel's eight entries are read before its adds;
//  * epilogue: the pooled sums + bias transposed into an [item][c_out + 1]
//    tile, then 16 lanes per item run the k-WTA as in the input-stationary
//    layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "mrs_sample.h"

namespace cs {

constexpr int GATH_BD = 1024;              // threads per workgroup
constexpr int GATH_C = 64;                 // input channels
constexpr int GATH_CAP = 8;                // list slots per input pixel
constexpr int GATH_BLK_B = 64 * 64 * 4;    // bytes of one block of 64 output pixels (64 channels)
static_assert(GATH_BD == SAMPLE_BD, "the chain's phases share the workgroup size");

struct GatherArgs {
  int NH;            // blocks of 64 output pixels: ceil(Ho * Wo / 64), KW * NH <= 16
  int nitems;        // pooled items: (Ho / pool) * (Wo / pool)
  int k, shift, write_sums;
  uint32_t off_tab, off_ent, off_cnt, off_bias, off_pt;   // LDS byte offsets (accumulators at 0)
  FastDiv fd_wo;     // / Wo
  FastDiv fd_wp;     // / pooled width
  FastDiv fd_items;  // / nitems
};

// The workgroup body for image blk (GATH_BD threads).  G: sets (4: two pairs).
template <typename TO, int KW, int G>
__device__ __forceinline__ void gather_body(const uint16_t* __restrict__ lidx,
                                            const int8_t* __restrict__ lval,
                                            const int32_t* __restrict__ lcnt,
                                            const uint16_t* __restrict__ aug,
                                            const int32_t* __restrict__ bias,
                                            int32_t* __restrict__ y, TO* __restrict__ out,
                                            const ListOut& lo, const ConvGeom& geo,
                                            const GatherArgs& ga, uint32_t blk) {
  static_assert(G % 2 == 0 && G <= 4, "sets are taken in pairs");
  constexpr int T = KW * KW;                // taps (square window)
  constexpr int NPR = G / 2;                // set pairs
  constexpr int TAB_PAIR_B = T * GATH_C * 4;   // bytes of one pair's table
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int H = geo.H, W = geo.W, P = geo.P, Wo = geo.Wo, n = geo.n, c_out = geo.c_out;
  const int npix = H * W;                                          // <= GATH_BD (host)
  const int64_t prow0 = (int64_t)blk * npix;

  unsigned char* accb = smem;                                      // [NH][64 ch][64 px] int32
  uint32_t* tab = reinterpret_cast<uint32_t*>(smem + ga.off_tab);  // [NPR][T][64] words
  uint32_t* ent = reinterpret_cast<uint32_t*>(smem + ga.off_ent);  // [npix][8] 16-bit
  int* cnt_s = reinterpret_cast<int*>(smem + ga.off_cnt);          // [npix]
  int* bias_s = reinterpret_cast<int*>(smem + ga.off_bias);        // [c_out]
  int* pt = reinterpret_cast<int*>(smem + ga.off_pt);              // [nitems][c_out + 1]

  // ---- global loads issued together: counts, entries (two per thread and
  // round), table pieces (16 bytes per thread and round)
  int c = 0;
  if (tid < npix) c = lcnt[prow0 + tid];
  const int npairs = npix * (GATH_CAP / 2);                        // entry pairs
  const uint32_t* li2 = reinterpret_cast<const uint32_t*>(lidx + prow0 * GATH_CAP);
  const uint16_t* lv2 = reinterpret_cast<const uint16_t*>(lval + prow0 * GATH_CAP);
  constexpr int PRE = 4;                                           // npairs <= PRE * GATH_BD
  uint32_t ei[PRE];
  uint32_t ev[PRE];
#pragma unroll
  for (int u = 0; u < PRE; ++u) {
    const int m = u * GATH_BD + tid;
    const int mc = m < npairs ? m : npairs - 1;                    // npairs >= 4 (host)
    ei[u] = li2[mc];
    ev[u] = lv2[mc];
  }
  // the table: word (tap*C + channel)*NPR + pr of the packed tensor holds
  // sets 2pr, 2pr + 1; each 16-bit half's Kernel ID becomes the output
  // channel (2pr + half)*n + min(kid, n - 1) (< 64).  Piece m (16 bytes) is
  // words 4m .. 4m + 3: rows 4m/NPR .. of pair (word mod NPR).
  constexpr int N16 = T * GATH_C * NPR / 4;                        // pieces
  constexpr int TPRE = (N16 + GATH_BD - 1) / GATH_BD;
  const su32x4* src = reinterpret_cast<const su32x4*>(aug);
  su32x4 tv[TPRE];
#pragma unroll
  for (int u = 0; u < TPRE; ++u) {
    const int m = u * GATH_BD + tid;
    tv[u] = src[m < N16 ? m : N16 - 1];
  }
  auto chan = [n](uint32_t w, int pr) -> uint32_t {
    const uint32_t k0 = (w >> 8) & 0xFFu, k1 = w >> 24;
    const uint32_t c0 = (uint32_t)(2 * pr * n) + (k0 < (uint32_t)n ? k0 : (uint32_t)(n - 1));
    const uint32_t c1 = (uint32_t)((2 * pr + 1) * n) + (k1 < (uint32_t)n ? k1 : (uint32_t)(n - 1));
    return (w & 0x00FF00FFu) | c0 << 8 | c1 << 24;
  };
  for (int o = tid; o < c_out; o += GATH_BD) bias_s[o] = bias ? bias[o] : 0;
#pragma unroll
  for (int u = 0; u < TPRE; ++u) {
    const int m = u * GATH_BD + tid;
    if (m < N16) {
      const su32x4 v = tv[u];
      if constexpr (NPR == 2) {
        // rows 2m, 2m + 1: (pair 0, pair 1) words (x, y) and (z, w)
        *reinterpret_cast<uint2*>(tab + 2 * m) = make_uint2(chan(v.x, 0), chan(v.z, 0));
        *reinterpret_cast<uint2*>(tab + T * GATH_C + 2 * m) = make_uint2(chan(v.y, 1), chan(v.w, 1));
      } else {
        su32x4 o;
        o.x = chan(v.x, 0);
        o.y = chan(v.y, 0);
        o.z = chan(v.z, 0);
        o.w = chan(v.w, 0);
        reinterpret_cast<su32x4*>(tab)[m] = o;
      }
    }
  }
  {
    su32x4* a4 = reinterpret_cast<su32x4*>(accb);
    const su32x4 z = {0u, 0u, 0u, 0u};
    for (int e = tid; e < ga.NH * (GATH_BLK_B / 16); e += GATH_BD) a4[e] = z;
  }
  if (tid < npix) cnt_s[tid] = c < 0 ? 0 : (c > GATH_CAP ? GATH_CAP : c);
  // entries: (channel & 63) | value << 8, two per word (channels of the
  // first layer's lists are < 64)
#pragma unroll
  for (int u = 0; u < PRE; ++u) {
    const int m = u * GATH_BD + tid;
    if (m < npairs)
      ent[m] = (ei[u] & 0x3Fu) | (ev[u] & 0xFFu) << 8 | (ei[u] & 0x3F0000u) |
               (ev[u] & 0xFF00u) << 16;
  }
  __syncthreads();
  CS_STAMP(5);

  // ---- multiply, route, sum
  if (wv < KW * ga.NH) {                                           // uniform
    const int ky = __builtin_amdgcn_readfirstlane(wv / ga.NH);
    const int hb = wv - ky * ga.NH;
    const int p = hb * 64 + lane;
    const bool live = p < geo.Ho * Wo;
    const int oy = (int)fdiv((uint32_t)p, ga.fd_wo), ox = p - oy * Wo;
    const int iy = oy + ky - P;
    const bool rok = live && (unsigned)iy < (unsigned)H;
    const uint32_t abase = (uint32_t)(hb * GATH_BLK_B + lane * 4);
    const unsigned char* tabb = reinterpret_cast<const unsigned char*>(tab) + ky * KW * GATH_C * 4;
    const su32x4* ent4 = reinterpret_cast<const su32x4*>(ent);
#pragma unroll
    for (int kx = 0; kx < KW; ++kx) {
      const int ix = ox + kx - P;
      const bool ok = rok && (unsigned)ix < (unsigned)W;
      const int q = ok ? iy * W + ix : 0;
      const int cq = ok ? cnt_s[q] : 0;
      const su32x4 e4 = ent4[q];
      // the eight entries' table words first (channel bits only: in range
      // for every slot, live or not)
      uint32_t tw[GATH_CAP][NPR];
#pragma unroll
      for (int j = 0; j < GATH_CAP; ++j) {
        const uint32_t ch = (e4[j >> 1] >> (16 * (j & 1))) & 0x3Fu;
        const unsigned char* tp = tabb + kx * GATH_C * 4 + ch * 4;
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr)
          tw[j][pr] = *reinterpret_cast<const uint32_t*>(tp + pr * TAB_PAIR_B);
      }
#pragma unroll
      for (int j = 0; j < GATH_CAP; ++j) {
        if (j < cq) {
          CS_COUNT_PRODUCTS_ADD(G);
          const int x = (int)(int8_t)(e4[j >> 1] >> (16 * (j & 1) + 8));
#pragma unroll
          for (int pr = 0; pr < NPR; ++pr) {
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
              const uint32_t wk = tw[j][pr] >> (16 * hf);
              const uint32_t och = (wk >> 8) & 0xFFu;             // output channel (< 64)
              __hip_atomic_fetch_add(reinterpret_cast<int*>(accb + abase + och * 256u),
                                     __mul24(x, (int)(int8_t)(wk & 0xFFu)), __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_WORKGROUP);
            }
          }
        }
      }
    }
  }
  __syncthreads();
  CS_STAMP(6);

  // ---- epilogue: pooled sums + bias into [item][c_out + 1], lanes along
  // items (consecutive pixels, different banks)
  const int pool = geo.pool;
  const int Wp = Wo / pool, Hp = geo.Ho / pool;
  const int nitems = ga.nitems;
  const int pts = c_out + 1;
  auto accw = [&](int px, int ch) -> int {
    return *reinterpret_cast<const int*>(accb + (px >> 6) * GATH_BLK_B + ch * 256 + (px & 63) * 4);
  };
  for (int t = tid; t < nitems * c_out; t += GATH_BD) {
    const int ch = (int)fdiv((uint32_t)t, ga.fd_items), it = t - ch * nitems;
    const int pr = (int)fdiv((uint32_t)it, ga.fd_wp), pc = it - pr * Wp;
    const int px = pr * pool * Wo + pc * pool;
    int a = accw(px, ch);
    if (pool == 2) a = max(max(a, accw(px + 1, ch)), max(accw(px + Wo, ch), accw(px + Wo + 1, ch)));
    pt[it * pts + ch] = a + bias_s[ch];
  }
  __syncthreads();
  constexpr int KPL = 4;                                           // c_out <= 64
  const int r16 = lane & 15;
  for (int ib = wv * 4; ib < nitems; ib += GATH_BD / 16) {         // uniform per wavefront
    const int it = ib + (lane >> 4);
    const bool live = it < nitems;
    const int itc = live ? it : ib;
    const int pr = (int)fdiv((uint32_t)itc, ga.fd_wp), pc = itc - pr * Wp;
    int v[KPL];
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int chn = r16 * KPL + i;
      v[i] = chn < c_out ? pt[itc * pts + chn] : 0;
    }
    const int64_t row = ((int64_t)blk * Hp + pr) * Wp + pc;
    if (ga.write_sums && live) {
#pragma unroll
      for (int j = 0; j < KPL; ++j)
        if (r16 * KPL + j < c_out) y[row * c_out + r16 * KPL + j] = v[j];
    }
    if (ga.k >= 0) kwta_row16<int32_t, TO, KPL>(v, c_out, ga.k, ga.shift, live, lo, out, row);
  }
}

}  // namespace cs
