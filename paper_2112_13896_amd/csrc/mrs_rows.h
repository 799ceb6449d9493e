// One wavefront per item: Multiply, Route and Sum (Section 3.2 steps 3-5)
// and k-WTA (Section 3.3.3) for an int8 layer whose window is one tap (a 1x1
// convolution with stride 1, or a linear layer) with many items, each with a
// short list and a row of 129-2048 outputs or a k over 32.
//
//  * the workgroup stages the packed table (value + Kernel ID per slot) in LDS
//    once; after that its wavefronts work without workgroup barriers, each
//    on its own items;
//  * a wavefront's accumulator row is in output-channel order and starts at
//    the bias; lane j holds entry j of the item's list (its table row offset
//    and value); when G > 32 each lane takes the sets g = lane + 64 q and the
//    entries one after another (broadcast from their lanes), else the lanes
//    form 64 / G slices of G sets, a slice taking every (64 / G)-th entry;
//    a lane reads the table entry of (entry, set g), multiplies and adds the
//    product to channel g*n + kid with an LDS integer add (exact in any
//    order, so lanes may meet on one channel);
//  * lane l then holds the CPL consecutive channels l*CPL, ... of the row in
//    registers (CPL odd: the strided reads are free of bank conflicts), and the
//    row's memory serves as a 512-bin histogram for an exact radix select of
//    the k-th largest sum (9-bit digits of the sum minus the row minimum; keys
//    outside the current prefix go to per-lane spare bins, so no lane is
//    masked); ties go to the lower channel, winners are written in channel
//    order; the lane then puts its bias back into the row for the next item.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "wave_ops.h"

namespace cs {

constexpr int ROWS_BD = 1024;             // most threads per workgroup (16 wavefronts)
constexpr int ROWS_BATCH = 4;             // table entries a lane reads before it adds
constexpr int ROWS_ENT_STRIDE = 66;       // int2 slots per wavefront entry copy (64 + zero + pad)
constexpr int ROWS_DIGIT = 9;             // bits per radix pass
constexpr int ROWS_BINS = 1 << ROWS_DIGIT;
constexpr int ROWS_HIST = ROWS_BINS + 64; // bins + one spare bin per lane

struct RowsArgs {
  int k;
  int shift;
  int write_sums;
  int qf;             // groups of 64 sets with wavefront-uniform entries (the last may be partial)
  int S;              // slices of the remaining Gs sets (0: none)
  int gbase;          // first of the remaining sets (64 qf)
  uint32_t off_acc;    // LDS byte offset of the wavefronts' rows (table at 0)
  uint32_t acc_words;  // words per wavefront row (>= c_out and >= ROWS_HIST)
  uint32_t off_bias;   // LDS byte offset of the bias (c_out words)
  uint32_t off_ent;    // LDS byte offset of the wavefronts' entry copies (S > 1 only)
  int64_t per_wg;      // items per workgroup
  FastDiv fd_g;        // / Gs
};

template <typename TO, int CPL, bool FULL>
__global__ __launch_bounds__(ROWS_BD) void mrs_rows(const uint16_t* __restrict__ lidx,
                                                    const int8_t* __restrict__ lval,
                                                    const int32_t* __restrict__ lcnt,
                                                    const uint16_t* __restrict__ aug,
                                                    const int32_t* __restrict__ bias,
                                                    int32_t* __restrict__ y, TO* __restrict__ out,
                                                    ListOut lo, ConvGeom geo, RowsArgs ra,
                                                    int64_t items) {
  static_assert(CPL % 2 == 1, "odd channels per lane keep the row reads conflict-free");
  static_assert(CPL <= 64, "the winner mask holds 64 slots");
  using Mask = typename std::conditional<(CPL > 32), uint64_t, uint32_t>::type;
  typedef uint32_t u4_t __attribute__((ext_vector_type(4)));
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nthr = (int)blockDim.x, nwv = nthr >> 6;
  const int G = geo.G, n = geo.n, c = geo.c_out, cap = geo.cap;
  // the packed table [C][G] is at LDS offset 0
  int32_t* acc = reinterpret_cast<int32_t*>(smem + ra.off_acc) + wv * ra.acc_words;
  uint32_t* hist = reinterpret_cast<uint32_t*>(acc);                      // the same words
  int32_t* bias_s = reinterpret_cast<int32_t*>(smem + ra.off_bias);     // [c_out]
  // (row offset, value) of up to 64 entries, then a (0, 0) entry for slots past the list
  int2* ent = reinterpret_cast<int2*>(smem + ra.off_ent) + wv * ROWS_ENT_STRIDE;

  // ---- the table into LDS (16-byte pieces), once per workgroup
  {
    const int nb = geo.C * G * 2;                                   // R = C (one tap)
    const int n16 = nb / 16;
    const uint4* src = reinterpret_cast<const uint4*>(aug);
    uint4* dst = reinterpret_cast<uint4*>(smem);
    for (int b0 = 0; b0 < n16; b0 += nthr * 4) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = b0 + u * nthr + tid;
        v[u] = src[e < n16 ? e : n16 - 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = b0 + u * nthr + tid;
        if (e < n16) dst[e] = v[u];
      }
    }
    for (int e = n16 * 16 + tid; e < nb; e += nthr)              // the tail bytes
      smem[e] = reinterpret_cast<const unsigned char*>(aug)[e];
  }
  // the lane's channels ch0 .. ch0 + nv - 1 and their bias; rows start at the bias
  const int ch0 = lane * CPL;
  // FULL: c_out = 64 CPL, every lane's slots are channels
  const int nv = FULL ? CPL : (c - ch0 < 0 ? 0 : (c - ch0 < CPL ? c - ch0 : CPL));
  for (int o = tid; o < c; o += nthr) bias_s[o] = bias != nullptr ? bias[o] : 0;
  if (lane == 0) ent[64] = make_int2(0, 0);
  __syncthreads();
  // a lane's slots past c_out (pads) take part as the row's smallest keys and
  // never win; their row words are scratch
#pragma unroll
  for (int i = 0; i < CPL; ++i) acc[ch0 + i] = bias_s[ch0 + i < c ? ch0 + i : c - 1];

  const int64_t ib = (int64_t)blockIdx.x * ra.per_wg;
  const int nit = (int)(items - ib < ra.per_wg ? items - ib : ra.per_wg);
  // the remaining sets as slices: this lane's slice s and set gbase + g0
  // (lanes past S * Gs idle)
  const int s = (int)fdiv((uint32_t)lane, ra.fd_g);
  const int g0 = lane - s * (int)ra.fd_g.d;
  const bool job = s < ra.S;

  // the next item's count and first 64 list entries (one per lane) are loaded while
  // the current item is processed
  int cnt_n = 0;
  uint16_t pi_n = 0;
  int8_t pv_n = 0;
  auto prefetch = [&](int li) {
    if (li < nit) {
      const int64_t it = ib + li;
      cnt_n = lcnt[it];
      const int j = lane < cap ? lane : cap - 1;
      pi_n = lidx[it * cap + j];
      pv_n = lval[it * cap + j];
    }
  };
  int li = wv;                                                      // uniform
  prefetch(li);
  while (li < nit) {
    // the lane's first channel, recomputed per item (not held in registers per slot)
    const int cl = opaque_int(ch0);
    const int lnext = li + nwv;
    const int64_t it = ib + li;
    int cnt = __builtin_amdgcn_readfirstlane(cnt_n);
    cnt = cnt < 0 ? 0 : (cnt > cap ? cap : cnt);
    const uint16_t pi = pi_n;
    const int8_t pv = pv_n;
    prefetch(lnext);

    // ---- Multiply, Route, Sum
    const int64_t lb = it * cap;
    for (int j0 = 0; j0 < cnt; j0 += 64) {                          // uniform
      const int nb = cnt - j0 < 64 ? cnt - j0 : 64;
      // lane j holds entry j0 + j: its table row's byte offset and its value
      int pre, xv;
      {
        const int j = lane < nb ? lane : nb - 1;
        const uint16_t ix = j0 == 0 ? pi : lidx[lb + j0 + j];
        const int8_t v = j0 == 0 ? pv : lval[lb + j0 + j];
        pre = (int)ix * G * 2;
        xv = lane < nb ? (int)v : 0;
      }
      // groups of 64 sets: lane l takes set 64 q + l, the entries one after
      // another (wavefront-uniform, read from their lanes)
      for (int e = 0; ra.qf > 0 && e < nb; e += ROWS_BATCH) {       // uniform
        int sp[ROWS_BATCH], sx[ROWS_BATCH];
#pragma unroll
        for (int u = 0; u < ROWS_BATCH; ++u) {
          const int eu = e + u < nb ? e + u : nb - 1;
          sp[u] = __builtin_amdgcn_readlane(pre, eu);
          sx[u] = e + u < nb ? __builtin_amdgcn_readlane(xv, eu) : 0;
        }
        for (int q = 0; q < ra.qf; ++q) {                           // uniform
          const int g = lane + 64 * q;
          if (g < G) {                                              // all lanes but in a last partial group
            CS_COUNT_PRODUCTS_ADD(min(ROWS_BATCH, nb - e));
            uint32_t w[ROWS_BATCH];
#pragma unroll
            for (int u = 0; u < ROWS_BATCH; ++u)
              w[u] = *reinterpret_cast<const uint16_t*>(smem + sp[u] + 2 * g);
            int32_t* ag = acc + g * n;
#pragma unroll
            for (int u = 0; u < ROWS_BATCH; ++u)
              __hip_atomic_fetch_add(ag + (int)(w[u] >> 8),
                                     __mul24(sx[u], (int)(int8_t)(w[u] & 0xFFu)),
                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
        }
      }
      // the remaining Gs sets (from gbase on) as S slices: lane (s, g0) takes
      // set gbase + g0 and the entries s, s + S, ..., read from a
      // wavefront-private copy of the entries in LDS
      if (ra.S > 0) {
        ent[lane] = make_int2(pre, xv);
        wave_lds_order();
        if (job) {
          const int S = ra.S;
          const int g = ra.gbase + g0;
          int32_t* ag = acc + g * n;
          for (int e = 0; e < nb; e += S * ROWS_BATCH) {            // uniform
            int2 en[ROWS_BATCH];
#pragma unroll
            for (int u = 0; u < ROWS_BATCH; ++u) {
              const int el = e + s + S * u;
              en[u] = ent[el < nb ? el : 64];
            }
            CS_COUNT_PRODUCTS_ADD(min(ROWS_BATCH, (nb - e - s + S - 1) / S));
            uint32_t w[ROWS_BATCH];
#pragma unroll
            for (int u = 0; u < ROWS_BATCH; ++u)
              w[u] = *reinterpret_cast<const uint16_t*>(smem + en[u].x + 2 * g);
#pragma unroll
            for (int u = 0; u < ROWS_BATCH; ++u)
              __hip_atomic_fetch_add(ag + (int)(w[u] >> 8),
                                     __mul24(en[u].y, (int)(int8_t)(w[u] & 0xFFu)),
                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
        }
        wave_lds_order();                                           // before the buffer is rewritten
      }
    }

    if (ra.k < 0) {
      // ---- sums only: the row to HBM (16-byte stores when c_out allows),
      // then back to the bias
      wave_lds_order();
      if ((c & 3) == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0) {
        typedef int32_t i4_t __attribute__((ext_vector_type(4)));
        i4_t* y4 = reinterpret_cast<i4_t*>(y + it * c);
        for (int o = lane; o < (c >> 2); o += 64) y4[o] = reinterpret_cast<const i4_t*>(acc)[o];
      } else {
        for (int o = lane; o < c; o += 64) y[it * c + o] = acc[o];
      }
      wave_lds_order();
#pragma unroll
      for (int i = 0; i < CPL; ++i) acc[cl + i] = bias_s[cl + i < c ? cl + i : c - 1];
      li = lnext;
      continue;
    }

    // ---- the row into registers; its memory becomes the histogram
    uint32_t key[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) key[i] = order_key(acc[cl + i]);
    if (ra.write_sums) {
#pragma unroll
      for (int i = 0; i < CPL; ++i)
        if (i < nv) y[it * c + cl + i] = (int32_t)(key[i] ^ 0x80000000u);
    }
    uint32_t kmn = 0xFFFFFFFFu, kmx = 0u;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if (i < nv) {
        kmn = key[i] < kmn ? key[i] : kmn;
        kmx = key[i] > kmx ? key[i] : kmx;
      }
    }
    kmn = wave_min_u32(kmn);
    kmx = wave_max_u32(kmx);
#pragma unroll
    for (int i = 0; i < CPL; ++i) key[i] = i < nv ? key[i] - kmn : 0u;   // pads: 0
    const uint32_t range = kmx - kmn;
    const int k = ra.k;
    uint32_t thr = 0u;                                              // an offset key
    int need = 0;
    if (k <= 0) {
      thr = 0xFFFFFFFFu;
    } else if (k >= c) {
      need = c;
    } else if (range == 0u) {
      need = k;
    } else {
      int rem = 32 - __builtin_clz(range);
      int passes = (rem + ROWS_DIGIT - 1) / ROWS_DIGIT;
      uint32_t prefix = 0u;
      int nd = k;
      const u4_t z = {0u, 0u, 0u, 0u};
      wave_lds_order();                                             // the row reads first
      reinterpret_cast<u4_t*>(hist)[2 * lane] = z;
      reinterpret_cast<u4_t*>(hist)[2 * lane + 1] = z;
      const int spare = ROWS_BINS + lane;
      for (; passes > 0; --passes) {                                // uniform
        const int width = (rem + passes - 1) / passes;
        const int sh = rem - width;
        const uint32_t hi = rem >= 32 ? 0u : (0xFFFFFFFFu << rem);
        const uint32_t lob = rem >= 32 ? 0u : (prefix << rem);
        wave_lds_order();
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
          const bool in = (key[i] & hi) == lob;
          const int bin = in ? (int)__builtin_amdgcn_ubfe(key[i], (uint32_t)sh, (uint32_t)width)
                             : spare;
          __hip_atomic_fetch_add(hist + bin, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        wave_lds_order();
        // lane l holds bins 8(63 - l) .. 8(63 - l) + 7: an inclusive scan over
        // lanes counts the keys in a lane's bins and above
        const int b0 = 8 * (63 - lane);
        const u4_t h0 = reinterpret_cast<const u4_t*>(hist + b0)[0];
        const u4_t h1 = reinterpret_cast<const u4_t*>(hist + b0)[1];
        reinterpret_cast<u4_t*>(hist + b0)[0] = z;                  // the next pass's bins
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
        const uint64_t fb = __ballot(above < nd && nd <= incl);     // exactly one lane
        const int f = __ffsll((unsigned long long)fb) - 1;
        prefix = (prefix << width) | (uint32_t)__builtin_amdgcn_readlane(bin, f);
        nd -= __builtin_amdgcn_readlane(run, f);
        rem = sh;
      }
      thr = prefix;
      need = nd;
    }
    // ---- winners in channel order: key > thr, or key == thr among the first `need`
    int gt_l = 0, eq_l = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      gt_l += key[i] > thr ? 1 : 0;
      eq_l += key[i] == thr ? 1 : 0;
    }
    const uint32_t pk = (uint32_t)eq_l | ((uint32_t)gt_l << 16);
    const uint32_t pincl = wave_incl_scan(pk, 0u, OpAdd{});
    int eqb = (int)((pincl - pk) & 0xFFFFu);                        // ties in lower lanes
    // the list of the non-zero winners staged in the row's memory (positions
    // in channel order, the other slots to spare entries k + lane) and copied
    // out with consecutive lanes on consecutive entries, when it fits there
    const int sidx_b = ((k + 64) * 2 + 3) & ~3;
    const bool stage = lo.idx != nullptr && k >= 0 &&
                       sidx_b + (k + 64) * (int)sizeof(TO) <= 4 * (int)ra.acc_words;
    if (lo.idx) {
      // the non-zero winners: counted first (bit i of pb), then written at
      // their list positions
      Mask pb = 0;
      int np = 0, er = eqb;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const bool eq = key[i] == thr;
        const bool win = i < nv && (key[i] > thr || (eq && er < need));
        er += eq ? 1 : 0;
        const TO ov = kwta_out<int32_t, TO>((int32_t)((key[i] + kmn) ^ 0x80000000u), ra.shift);
        const bool put = win && ov != TO(0);
        pb |= put ? (Mask(1) << i) : Mask(0);
        np += put ? 1 : 0;
      }
      const int pin = (int)wave_incl_scan((uint32_t)np, 0u, OpAdd{});
      uint32_t pos = (uint32_t)(pin - np);
      // row base pointers (uniform) and 32-bit byte offsets per lane
      unsigned char* lv = reinterpret_cast<unsigned char*>(static_cast<TO*>(lo.val) + it * lo.cap);
      unsigned char* lx = reinterpret_cast<unsigned char*>(lo.idx + it * lo.cap);
      if (stage) {
        uint16_t* sx = reinterpret_cast<uint16_t*>(acc);
        TO* sv = reinterpret_cast<TO*>(reinterpret_cast<unsigned char*>(acc) + sidx_b);
        wave_lds_order();                                           // after the histogram reads
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
          const bool put = (pb >> i) & Mask(1);
          const int p = put ? (int)pos : k + lane;
          sx[p] = (uint16_t)(cl + i);
          sv[p] = kwta_out<int32_t, TO>((int32_t)((key[i] + kmn) ^ 0x80000000u), ra.shift);
          pos += put ? 1u : 0u;
        }
        wave_lds_order();
        const int total = __builtin_amdgcn_readlane(pin, 63);
        for (int j = lane; j < total; j += 64) {
          *reinterpret_cast<uint16_t*>(lx + 2u * (uint32_t)j) = sx[j];
          *reinterpret_cast<TO*>(lv + (uint32_t)sizeof(TO) * (uint32_t)j) = sv[j];
        }
        wave_lds_order();                                           // before the row is reset
      } else {
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
          if ((pb >> i) & Mask(1)) {
            *reinterpret_cast<uint16_t*>(lx + 2u * pos) = (uint16_t)(cl + i);
            *reinterpret_cast<TO*>(lv + (uint32_t)sizeof(TO) * pos) =
                kwta_out<int32_t, TO>((int32_t)((key[i] + kmn) ^ 0x80000000u), ra.shift);
            ++pos;
          }
        }
      }
      if (lane == 63) lo.cnt[it] = pin;
    } else {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const bool eq = key[i] == thr;
        const bool win = key[i] > thr || (eq && eqb < need);
        eqb += eq ? 1 : 0;
        const TO ov = kwta_out<int32_t, TO>((int32_t)((key[i] + kmn) ^ 0x80000000u), ra.shift);
        if (i < nv) out[it * c + cl + i] = win ? ov : TO(0);
      }
    }
    // ---- the row back to the bias for the next item
    wave_lds_order();
#pragma unroll
    for (int i = 0; i < CPL; ++i) acc[cl + i] = bias_s[cl + i < c ? cl + i : c - 1];
    li = lnext;
  }
}

}  // namespace cs
