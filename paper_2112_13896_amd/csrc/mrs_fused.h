// One layer in one kernel: Multiply, Route and Sum (Section 3.2 steps 3-5)
// followed by the optional 2x2 max-pool, bias, k-WTA and requantisation, with
// the winners written as the next layer's (index, value) lists (Figure 10:
// winners go on together with their indices) or as a dense masked tensor.
//
// A workgroup owns a tile of output items that is complete in the channel
// dimension: every set of the layer, so every output channel of its items,
// is computed inside the workgroup, which is what lets k-WTA run in the
// epilogue without a round trip through HBM.
//
//  * tiles: for a 1x1 layer with stride 1, no padding and no pooling (and a
//    linear layer) TI consecutive items, which read TI consecutive input rows;
//    otherwise TPR rows of pooled outputs times TW pooled columns of one image,
//    which read a rectangle of input pixels (the window halo included);
//  * staging: the whole augmented table (value + Kernel ID per slot, Section
//    3.3.1) is copied into LDS; the input pixels' counts are read, a
//    workgroup prefix sum gives each pixel's place, and the pixels' list
//    chunks are copied into LDS.  Pixels that do not fit the LDS list budget
//    are read from global memory later instead - staging never changes what
//    is computed;
//  * compute: lanes are (item, set unit of GB sets, pool sub-pixel q); a lane
//    walks the taps of its sub-pixel and the 4-entry chunks of each tap's
//    list, reading lists and packed rows from LDS (Multiply), and routes each
//    product to acc[kid] (Route, Sum) as in the staged kernel; the 2x2 max
//    of the sub-pixel lanes plus the bias go to an LDS tile of the items'
//    c_out sums;
//  * epilogue: the sums are written out if asked for; k-WTA finds each item's
//    threshold key (the k-th largest of the order-preserving keys; Section
//    3.3.3) with one lane per item (top-k insertion; rows of at most 128
//    channels, k <= 32 - longer rows go to the separate k-WTA kernel); then
//    one wavefront per item writes the winners, ties to the lower index,
//    requantised, as lists (staged in LDS, written out 4 entries at a time)
//    or densely.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "mrs_tiled.h"

namespace cs {

constexpr int FUSED_PPT = 4;     // most input pixels whose counts one thread reads
constexpr int FUSED_NACC = 32;   // most accumulators of one lane (sets per lane x n)
                                 // (the LDS holds them rounded up to a multiple of 8)
constexpr int FUSED_CB = 8;      // list chunks a thread copies per batch (int8; fp32: 4)

struct FusedArgs {
  int tile_mode;      // 0: items = consecutive input rows; 1: image rectangles
  int TI;             // mode 0: items per tile
  int TPR, TW;        // mode 1: pooled rows and pooled columns per tile
  int tiles_x;        // mode 1: tiles across the pooled width
  int tiles_img;      // mode 1: tiles per image
  int IW;             // mode 1: most input columns a tile reads
  int units;          // set units (G / GB)
  int log2Q;          // 0, or 2 with a 2x2 pool (one lane per sub-pixel)
  int log2S;          // slices: lanes sharing one (item, set unit, sub-pixel)'s taps,
                      // or its list chunks when the window is one tap
  int LPI;            // lanes per item = units << (log2Q + log2S)
  int IPR;            // items per round = MRS_BD / LPI
  int npix_cap;       // most staged input pixels of a tile (<= MRS_BD * FUSED_PPT)
  int list_cap;       // LDS capacity for list chunks (one more slot is allocated as a spare)
  int k;              // k-WTA winners per item; < 0: no k-WTA
  int shift;          // requantisation shift (int32 -> int8)
  int write_sums;     // 1: the sums after pool and bias are written to y
  int ostride;        // row stride of the LDS sum tile (c_out, or c_out + 1 for lane selection)
  int kmode;          // selection, one lane per item: 1/2/3 top-8/16/32 insertion
  uint32_t off_tab, off_bias, off_pix, off_cidx, off_cval, off_out, off_sel, off_misc;
  uint32_t off_lidx, off_lval;   // output lists of the tile, written out at the end
  FastDiv fd_lpi;     // / LPI
  FastDiv fd_tw;      // / TW
  FastDiv fd_iw;      // / IW
  FastDiv fd_kw;      // / KW
  FastDiv fd_tx;      // / tiles_x
  FastDiv fd_timg;    // / tiles_img
  FastDiv fd_cout;    // / c_out
  FastDiv fd_ochunks; // / (output list capacity / 4)
};

__device__ __forceinline__ int32_t shfl_xor_a(int32_t v, int m) { return __shfl_xor(v, m, 64); }
__device__ __forceinline__ float shfl_xor_a(float v, int m) { return __shfl_xor(v, m, 64); }

// Which slots of a tile hold an item (mode 1: column inside the image).
struct SlotMap {
  int mode, TW, npc, nslots;
  FastDiv fd_tw;
  __device__ __forceinline__ bool live(int it) const {
    if (it >= nslots) return false;
    if (mode == 0) return true;
    const int ir = (int)fdiv((uint32_t)it, fd_tw);
    return it - ir * TW < npc;
  }
};

// Output row (pixel) of tile slot it.
struct RowMap {
  int mode, TW, bb, Hp, Wp, pr0, pc0;
  int64_t item0;
  FastDiv fd_tw;
  __device__ __forceinline__ int64_t row(int it) const {
    if (mode == 0) return item0 + it;
    const int ir = (int)fdiv((uint32_t)it, fd_tw);
    const int ic = it - ir * TW;
    return ((int64_t)bb * Hp + pr0 + ir) * Wp + pc0 + ic;
  }
};

// k-WTA with four lanes per item (a quad): each lane keeps the KMAX largest
// keys of its quarter of the row, sorted (blocks of KMAX keys sorted and
// merged with bitonic networks), the quad merges the four lists (two exchange
// steps) and reads the threshold key T = the k-th largest.
// The winners are key > T and the first `need` keys equal to T in index
// order (ties go to the lower index); a quad prefix sum gives each lane its
// ties' ranks and its winners' positions in the row's list.  List output: the
// winners with a non-zero output value go to the tile's LDS lists in index
// order and their count to cnt.  sel[it] = (T, index of the last winning tie
// or -1).  Rows are read with an odd stride (bank-conflict free).
// One item (tile slot `it`) per quad; every lane of the wavefront takes part
// (the DPP exchanges), `live` quads write.
// ES: element stride of the row (1: a row-major tile; other: the quad's lanes
// read their quarters from LDS columns of that stride, `otile` then being the
// lane's own column and ostride unused).  CC: the row length when the caller
// knows it at compile time (c is then ignored; the quarters' bounds checks
// fold away and the block loops unroll), 0: c.
template <typename A, typename TO, int KMAX, int ES = 1, int CC = 0>
__device__ __forceinline__ void kwta_quad_item(const A* otile, int ostride, int it, bool live,
                                               const RowMap& rm, int c, int k, int shift,
                                               uint2* sel, uint16_t* tl_idx, TO* tl_val, int cap,
                                               int32_t* gcnt) {
  if constexpr (CC > 0) c = CC;
  constexpr int BK = 16;                               // keys read per batch (loads issued together)
  const int qd = threadIdx.x & 3;
  const int L = (c + 3) >> 2;                          // row quarter of a lane
  const int i_lo = qd * L, i_hi = min(c, i_lo + L);
  {
    // element i of the row (i_lo <= i < i_hi) is vq[(i - i_lo) * ES]
    const A* vq = ES == 1 ? otile + (live ? it : 0) * ostride + i_lo : otile;
    auto v = [&](int i) -> A { return vq[(i - i_lo) * ES]; };
    // --- the threshold: per-lane top-KMAX of the quarter, merged over the quad
    // (keys past the quarter are 0: a 0 never changes the k-th largest)
    uint32_t top[KMAX];
#pragma unroll
    for (int s = 0; s < KMAX; ++s) top[s] = 0u;
    const bool search = live && k > 0 && k < c;
    if (search) {
      // the first block, sorted, is the list; later blocks are merged into it
      for (int i0 = i_lo; i0 < i_hi; i0 += KMAX) {
        uint32_t blk[KMAX];
#pragma unroll
        for (int j = 0; j < KMAX; ++j) {
          const int i = i0 + j;
          const uint32_t kx = order_key(v(i < i_hi ? i : i_hi - 1));
          blk[j] = i < i_hi ? kx : 0u;
        }
        // the block's reads leave together (left to itself the scheduler
        // waits for each read before issuing the next)
        __builtin_amdgcn_sched_barrier(0);
        bitonic_sort_desc<KMAX>(blk);
        if (i0 == i_lo) {
#pragma unroll
          for (int j = 0; j < KMAX; ++j) top[j] = blk[j];
        } else {
          top_merge_desc<KMAX>(top, blk);
        }
      }
    }
    // merge with the neighbour at distance 1, then 2 (all four lanes end equal);
    // executed by every lane of the wavefront (DPP reads the partner's registers)
    {
      uint32_t px[KMAX];
#pragma unroll
      for (int s = 0; s < KMAX; ++s) px[s] = quad_xor1(top[s]);
      top_merge_desc<KMAX>(top, px);
#pragma unroll
      for (int s = 0; s < KMAX; ++s) px[s] = quad_xor2(top[s]);
      top_merge_desc<KMAX>(top, px);
    }
    uint32_t thr = 0u;
    int need = 0;
    if (k >= c) {
      need = c;                                        // every element wins (key >= 0)
    } else if (k > 0) {
#pragma unroll
      for (int s = 0; s < KMAX; ++s) thr = (s == k - 1) ? top[s] : thr;
      int gt = 0;
#pragma unroll
      for (int s = 0; s < KMAX; ++s) gt += (s < k && top[s] > thr) ? 1 : 0;
      need = k - gt;
    }
    // --- the lane's quarter as bit masks (bit j: element i_lo + j; c <= 128,
    // so a quarter has at most 32 elements): keys above T, keys equal to T,
    // and (list output) elements whose output value is non-zero
    uint32_t gtm = 0u, eqm = 0u, nzm = 0u;
    const bool lists = tl_idx != nullptr;
    if (live && k > 0) {
      for (int i0 = i_lo; i0 < i_hi; i0 += BK) {
        A vb[BK];
#pragma unroll
        for (int j = 0; j < BK; ++j) {
          const int i = i0 + j;
          vb[j] = v(i < i_hi ? i : i_hi - 1);
        }
        __builtin_amdgcn_sched_barrier(0);               // the batch's reads leave together
#pragma unroll
        for (int j = 0; j < BK; ++j) {
          const int i = i0 + j;
          const uint32_t bit = i < i_hi ? 1u << (i - i_lo) : 0u;
          const uint32_t key = order_key(vb[j]);
          gtm |= key > thr ? bit : 0u;
          eqm |= key == thr ? bit : 0u;
          if (lists) nzm |= kwta_out<A, TO>(vb[j], shift) != TO(0) ? bit : 0u;
        }
      }
    }
    // the winning ties are the first `need` equal keys of the row: this lane's
    // first need - (ties in the quarters before) of its own
    const int ties_l = __popc(eqm);
    const int tie0 = quad_excl_sum(ties_l, qd);
    int m = need - tie0;
    m = m < 0 ? 0 : (m > ties_l ? ties_l : m);
    uint32_t tm = 0u;
    for (uint32_t e2 = eqm; m > 0; --m) {
      const uint32_t lb = e2 & (0u - e2);
      tm |= lb;
      e2 ^= lb;
    }
    int last_tie = tm ? i_lo + 31 - __builtin_clz(tm) : -1;
    // winners with a non-zero output value: their list positions
    const uint32_t putm = (gtm | tm) & nzm;
    const int win_l = __popc(putm);
    const int pos0 = quad_excl_sum(win_l, qd);           // list position of the first winner
    // the last winning tie of the row: the largest over the quad
    {
      uint32_t lt = (uint32_t)(last_tie + 1);
      uint32_t o1 = quad_xor1(lt);
      lt = o1 > lt ? o1 : lt;
      uint32_t o2 = quad_xor2(lt);
      lt = o2 > lt ? o2 : lt;
      last_tie = (int)lt - 1;
    }
    if (live) {
      if (tl_idx) {
        int pos = pos0;
        for (uint32_t w = putm; w != 0u; w &= w - 1u) {
          const int i = i_lo + __builtin_ctz(w);
          tl_idx[it * cap + pos] = (uint16_t)i;
          tl_val[it * cap + pos] = kwta_out<A, TO>(v(i), shift);
          ++pos;
        }
      }
      if (qd == 0) sel[it] = make_uint2(thr, (uint32_t)last_tie);
      if (tl_idx && qd == 3) gcnt[rm.row(it)] = pos0 + win_l;
    }
  }
}

// All the tile's slots, one per quad of the workgroup's BD threads.
template <typename A, typename TO, int KMAX, int BD = MRS_BD, int CC = 0>
__device__ void kwta_quad_items(const A* otile, int ostride, const SlotMap& sm, const RowMap& rm,
                                int c, int k, int shift, uint2* sel, uint16_t* tl_idx,
                                TO* tl_val, int cap, int32_t* gcnt) {
  const int nsl = (sm.nslots + 3) & ~3;
  for (int base = 0; base < ((nsl + BD / 4 - 1) / (BD / 4)) * (BD / 4); base += BD / 4) {
    const int it = base + (threadIdx.x >> 2);
    kwta_quad_item<A, TO, KMAX, 1, CC>(otile, ostride, it, sm.live(it), rm, c, k, shift, sel, tl_idx,
                                tl_val, cap, gcnt);
  }
}

// Exclusive prefix sum over the workgroup's threads in thread order; *total
// receives the sum over all threads.  ws: MRS_BD / 64 ints of LDS.  Ends with
// a barrier, so ws can be reused afterwards.
__device__ __forceinline__ int block_exclusive_scan(int v, int* ws, int* total) {
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
  for (int w = 0; w < MRS_BD / 64; ++w) {
    const int s = ws[w];
    base += (w < wv) ? s : 0;
    tot += s;
  }
  *total = tot;
  __syncthreads();
  return base + incl - v;
}

// The 4 values of a list chunk as one vector (for copies, as bits; a native
// vector type keeps arrays of them in registers).
template <typename T>
struct ChunkVal;
template <>
struct ChunkVal<int8_t> {
  using type = uint32_t;
};
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
template <>
struct ChunkVal<float> {
  using type = u32x4;
};
template <>
struct ChunkVal<int32_t> {
  using type = u32x4;
};

// A list chunk read from LDS (the staged copy).
template <typename T>
__device__ __forceinline__ void load_chunk_lds(Chunk<T>& ch, const uint16_t* ci, const T* cv,
                                               int e);
template <>
__device__ __forceinline__ void load_chunk_lds<int8_t>(Chunk<int8_t>& ch, const uint16_t* ci,
                                                       const int8_t* cv, int e) {
  ch.idx = reinterpret_cast<const uint2*>(ci)[e];
  ch.val = reinterpret_cast<const uint32_t*>(cv)[e];
}
template <>
__device__ __forceinline__ void load_chunk_lds<float>(Chunk<float>& ch, const uint16_t* ci,
                                                      const float* cv, int e) {
  ch.idx = reinterpret_cast<const uint2*>(ci)[e];
  ch.val = reinterpret_cast<const float4*>(cv)[e];
}

template <typename T, typename A, typename TO, bool ONE, int GB>
__global__ __launch_bounds__(MRS_BD) void mrs_fused(const uint16_t* __restrict__ lidx,
                                                    const T* __restrict__ lval,
                                                    const int32_t* __restrict__ lcnt,
                                                    const typename Aug<T>::type* __restrict__ aug,
                                                    const A* __restrict__ bias,
                                                    A* __restrict__ y, TO* __restrict__ out,
                                                    ListOut lo, ConvGeom geo, FusedArgs fa) {
  using E = typename Aug<T>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int n = ONE ? 1 : geo.n;
  const int T_ = geo.KH * geo.KW;
  const int R = T_ * geo.C;
  const int G = geo.G;
  const int c_out = geo.c_out;
  const int Wp = geo.Wo / geo.pool, Hp = geo.Ho / geo.pool;

  A* acc = reinterpret_cast<A*>(smem);                               // [GB * n][MRS_BD]
  unsigned char* tab = smem + fa.off_tab;                            // [R][G] entries
  A* bias_s = reinterpret_cast<A*>(smem + fa.off_bias);              // [c_out]
  int2* pix = reinterpret_cast<int2*>(smem + fa.off_pix);            // (count, chunk offset)
  uint16_t* cidx = reinterpret_cast<uint16_t*>(smem + fa.off_cidx);  // [list_cap][4]
  T* cval = reinterpret_cast<T*>(smem + fa.off_cval);                // [list_cap][4]
  A* otile = reinterpret_cast<A*>(smem + fa.off_out);                // [slots][ostride]
  int* misc = reinterpret_cast<int*>(smem + fa.off_misc);            // scan space + 2 counters

  // ---- tile geometry.  Item slots: mode 0, slot it = item item0 + it;
  // mode 1, slot it = (it / TW, it % TW) of the tile's pooled rectangle, live
  // when the column is inside the image.  Staged pixels: mode 0, pixel p =
  // input row item0 + p; mode 1, pixel p = (p / IW, p % IW) of the input
  // rectangle at (ry0, rx0), present when inside the image.
  int nslots, npix;
  int64_t item0;
  int bb = 0, pr0 = 0, pc0 = 0, npr = 0, npc = 0, ry0 = 0, rx0 = 0;
  if (fa.tile_mode == 0) {
    item0 = (int64_t)blockIdx.x * fa.TI;
    const int64_t items = (int64_t)geo.B * geo.Ho * geo.Wo;
    nslots = (int)(items - item0 < fa.TI ? items - item0 : fa.TI);
    npix = nslots;
  } else {
    const uint32_t img = fdiv(blockIdx.x, fa.fd_timg);
    const int tin = (int)(blockIdx.x - img * (uint32_t)fa.tiles_img);
    const int ty = (int)fdiv((uint32_t)tin, fa.fd_tx);
    const int tx = tin - ty * fa.tiles_x;
    bb = (int)img;
    pr0 = ty * fa.TPR;
    pc0 = tx * fa.TW;
    npr = min(fa.TPR, Hp - pr0);
    npc = min(fa.TW, Wp - pc0);
    nslots = npr * fa.TW;
    item0 = 0;
    // input rows read by the tile's windows, clipped to the image; IW columns
    // from rx0 hold every column the windows read (host: IW = window span)
    const int iy0 = pr0 * geo.pool * geo.S - geo.P;
    const int iy1 = ((pr0 + npr) * geo.pool - 1) * geo.S - geo.P + geo.KH;   // exclusive
    ry0 = max(iy0, 0);
    rx0 = max(pc0 * geo.pool * geo.S - geo.P, 0);
    npix = max(min(iy1, geo.H) - ry0, 0) * fa.IW;          // <= npix_cap (host)
  }
  // global input row of staged pixel p, or -1 outside the image
  auto gpix = [&](int p) -> int64_t {
    if (fa.tile_mode == 0) return item0 + p;
    const int r = (int)fdiv((uint32_t)p, fa.fd_iw);
    const int cx = rx0 + p - r * fa.IW;
    if (cx >= geo.W) return -1;
    return ((int64_t)bb * geo.H + ry0 + r) * geo.W + cx;
  };

  // ---- staging, phase 1: each thread owns pixels p = u*MRS_BD + tid and
  // loads their counts together with their first SPEC list chunks (most lists
  // are that short), all before the table copy, so one round trip covers all
  using V = typename ChunkVal<T>::type;
  constexpr int SPEC = sizeof(T) == 1 ? 3 : 2;
  const int nu = (npix + MRS_BD - 1) / MRS_BD;             // <= FUSED_PPT (host)
  int pc[FUSED_PPT];
  uint2 si[FUSED_PPT * SPEC];
  V sv[FUSED_PPT * SPEC];
#pragma unroll
  for (int u = 0; u < FUSED_PPT; ++u) {
    const int p = u * MRS_BD + tid;
    const int64_t gp = (u < nu && p < npix) ? gpix(p) : -1;
    pc[u] = gp >= 0 ? lcnt[gp] : 0;
#pragma unroll
    for (int s2 = 0; s2 < SPEC; ++s2) {
      // a lane without that chunk reads chunk 0 of row 0, which exists
      const int64_t a2 = (gp >= 0 && s2 * 4 < geo.cap) ? gp * geo.cap + s2 * 4 : 0;
      si[u * SPEC + s2] = *reinterpret_cast<const uint2*>(lidx + a2);
      sv[u * SPEC + s2] = *reinterpret_cast<const V*>(lval + a2);
    }
  }
  const int ntab = R * G;                                   // < 2^31 (host)
  const int ntab16 = (int)(((int64_t)ntab * (int64_t)sizeof(E)) >> 4);
  copy16_to_lds(reinterpret_cast<const uint4*>(aug), reinterpret_cast<uint4*>(tab), ntab16);
  for (int e = ntab16 * 16 / (int)sizeof(E) + tid; e < ntab; e += MRS_BD)   // the tail
    reinterpret_cast<E*>(tab)[e] = aug[e];
  for (int k2 = tid; k2 < c_out; k2 += MRS_BD) bias_s[k2] = bias ? bias[k2] : A(0);
  if (tid == 0) {
    misc[8] = 0;                                           // staged pixels
    misc[9] = 0;                                           // staged chunks
    misc[10] = 0;                                          // 1: a staged list has more than SPEC chunks
  }
  // chunk offsets in pixel order: one workgroup prefix sum per MRS_BD pixels
  int offs[FUSED_PPT];
  int base = 0;
#pragma unroll
  for (int u = 0; u < FUSED_PPT; ++u) {
    if (u < nu) {                                          // uniform
      const int c = pc[u] < 0 ? 0 : (pc[u] > geo.cap ? geo.cap : pc[u]);
      pc[u] = c;
      const int nch = (c + 3) >> 2;
      int tot = 0;
      const int off = base + block_exclusive_scan(nch, misc, &tot);   // barriers inside
      base += tot;
      offs[u] = off;
      const int p = u * MRS_BD + tid;
      if (p < npix) pix[p] = make_int2(c, off);
    } else {
      offs[u] = 0;
    }
  }
  // the speculative chunks of staged pixels into their slots (a lane without
  // one writes the spare slot list_cap, allocated and never read)
#pragma unroll
  for (int u = 0; u < FUSED_PPT; ++u) {
    const int p = u * MRS_BD + tid;
    const int nch = (pc[u] + 3) >> 2;
    const bool st = u < nu && p < npix && offs[u] + nch <= fa.list_cap;
#pragma unroll
    for (int s2 = 0; s2 < SPEC; ++s2) {
      const int e = (st && s2 < nch) ? offs[u] + s2 : fa.list_cap;
      reinterpret_cast<uint2*>(cidx)[e] = si[u * SPEC + s2];
      reinterpret_cast<V*>(cval)[e] = sv[u * SPEC + s2];
    }
  }
  __syncthreads();
  // staged pixels are a prefix (offsets grow with p): the last one records
  // how many there are and where their chunks end; a staged pixel with more
  // than SPEC chunks flags the second copy phase
#pragma unroll
  for (int u = 0; u < FUSED_PPT; ++u) {
    const int p = u * MRS_BD + tid;
    if (u < nu && p < npix) {
      const int nch = (pc[u] + 3) >> 2;
      if (offs[u] + nch <= fa.list_cap) {
        if (nch > SPEC) __hip_atomic_store(&misc[10], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        bool next_staged = false;
        if (p + 1 < npix) {
          const int2 nx = pix[p + 1];
          next_staged = nx.y + ((nx.x + 3) >> 2) <= fa.list_cap;
        }
        if (!next_staged) {
          misc[8] = p + 1;
          misc[9] = offs[u] + nch;
        }
      }
    }
  }
  __syncthreads();
  const int nst = misc[8];              // pixels [0, nst) are staged
  const int nchunks = misc[9];

  // ---- staging, phase 2: chunks past the first SPEC of longer lists
  if (misc[10] != 0) {
    constexpr int CB = sizeof(T) == 1 ? FUSED_CB : FUSED_CB / 2;
    for (int b0 = 0; b0 < nchunks; b0 += MRS_BD * CB) {
      int64_t src[CB];
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        const int e = b0 + u * MRS_BD + tid;
        src[u] = -1;
        if (e < nchunks) {
          // the staged pixel holding chunk e: the last p with offset <= e
          int lo_ = 0, hi_ = nst - 1;
          while (lo_ < hi_) {
            const int mid = (lo_ + hi_ + 1) >> 1;
            if (pix[mid].y <= e) lo_ = mid;
            else hi_ = mid - 1;
          }
          const int jc = e - pix[lo_].y;
          if (jc >= SPEC) src[u] = gpix(lo_) * geo.cap + (int64_t)jc * 4;
        }
      }
      uint2 ci[CB];
      V cv[CB];
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        const int64_t sa = src[u] >= 0 ? src[u] : 0;
        ci[u] = *reinterpret_cast<const uint2*>(lidx + sa);
        cv[u] = *reinterpret_cast<const V*>(lval + sa);
      }
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        const int e = src[u] >= 0 ? b0 + u * MRS_BD + tid : fa.list_cap;
        reinterpret_cast<uint2*>(cidx)[e] = ci[u];
        reinterpret_cast<V*>(cval)[e] = cv[u];
      }
    }
    __syncthreads();
  }

  // ---- compute: lanes (item of the round, set unit, sub-pixel q, slice s);
  // the Q*S lanes of one (item, set unit) are consecutive in one wavefront
  const int S = 1 << fa.log2S;
  const int log2QS = fa.log2Q + fa.log2S;
  const int QS = 1 << log2QS;
  const int nacc = GB * n;
  const int nacc8 = (nacc + 7) & ~7;                      // accumulator rows (host)
  const bool chunk_mode = T_ == 1;                         // slices split list chunks
  const uint32_t row_bytes = (uint32_t)(G * sizeof(E));
  const int io = (int)fdiv((uint32_t)tid, fa.fd_lpi);     // item within the round
  const int rem = tid - io * fa.LPI;
  const int unit = rem >> log2QS;
  const int r = rem & (QS - 1);                           // rank in the group
  const int sl = r & (S - 1);                             // slice
  const int q = r >> fa.log2S;                            // 2x2 pool sub-pixel
  const int gfirst = unit * GB;                           // first set of the lane
  A* acc_lane = acc + tid;
  const unsigned char* tcol = tab + (size_t)gfirst * sizeof(E);
  const int c0 = chunk_mode ? sl : 0, cstep = chunk_mode ? S : 1;

  // chunks c0, c0 + cstep, ... of staged pixel p's list (record pi) against
  // the table rows at tbase; the next chunk is read while one is processed
  auto run_list = [&](int p, int2 pi, const unsigned char* tbase, A (&accr)[GB]) {
    const int m = pi.x;
    if (c0 * 4 >= m) return;
    if (p < nst) {
      Chunk<T> cur;
      load_chunk_lds<T>(cur, cidx, cval, pi.y + c0);
      for (int c = c0;; c += cstep) {
        const bool more = (c + cstep) * 4 < m;
        Chunk<T> nxt;
        if (more) load_chunk_lds<T>(nxt, cidx, cval, pi.y + c + cstep);
        mrs_chunk<T, A, ONE, GB>(cur, m - c * 4, tbase, row_bytes, n, acc_lane, accr);
        if (!more) break;
        cur = nxt;
      }
    } else {
      const int64_t g = gpix(p) * geo.cap;
      const uint16_t* li = lidx + g;
      const T* lv = lval + g;
      Chunk<T> cur;
      cur.load(li, lv, c0 * 4);
      for (int c = c0;; c += cstep) {
        const bool more = (c + cstep) * 4 < m;
        Chunk<T> nxt;
        if (more) nxt.load(li, lv, (c + cstep) * 4);
        mrs_chunk<T, A, ONE, GB>(cur, m - c * 4, tbase, row_bytes, n, acc_lane, accr);
        if (!more) break;
        cur = nxt;
      }
    }
  };

  const SlotMap sm{fa.tile_mode, fa.TW, npc, nslots, fa.fd_tw};
  for (int it0 = 0; it0 < nslots; it0 += fa.IPR) {
    const int it = it0 + io;
    const bool active = io < fa.IPR && sm.live(it);
    A accr[GB];
#pragma unroll
    for (int j = 0; j < GB; ++j) accr[j] = A(0);
    for (int k2 = ONE ? GB : 0; k2 < nacc8; ++k2) acc_lane[k2 * MRS_BD] = A(0);
    if (active) {
      if (fa.tile_mode == 0) {
        run_list(it, pix[it], tcol, accr);
      } else {
        const int ir = (int)fdiv((uint32_t)it, fa.fd_tw);
        const int ic = it - ir * fa.TW;
        const int ho = (pr0 + ir) * geo.pool + (q >> 1) * (geo.pool >> 1);
        const int wo = (pc0 + ic) * geo.pool + (q & 1) * (geo.pool >> 1);
        // staged pixel under tap t, or -1 (padding)
        auto tap_pix = [&](int t) -> int {
          const int ky = (int)fdiv((uint32_t)t, fa.fd_kw), kx = t - ky * geo.KW;
          const int hy = ho * geo.S + ky - geo.P, wx = wo * geo.S + kx - geo.P;
          return (hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W)
                     ? (hy - ry0) * fa.IW + (wx - rx0) : -1;
        };
        const int tstep = chunk_mode ? 1 : S;
        int t = chunk_mode ? 0 : sl;
        int p = t < T_ ? tap_pix(t) : -1;
        int2 pi = p >= 0 ? pix[p] : make_int2(0, 0);
        while (t < T_) {
          // the next tap's pixel record is read while this tap is processed
          const int tn = t + tstep;
          const int pn = tn < T_ ? tap_pix(tn) : -1;
          const int2 pin = pn >= 0 ? pix[pn] : make_int2(0, 0);
          if (p >= 0) run_list(p, pi, tcol + (uint32_t)(t * geo.C) * row_bytes, accr);
          t = tn;
          p = pn;
          pi = pin;
        }
      }
    }
    // the group's partial sums are combined 8 channels at a time: each lane
    // reads its own LDS column (or registers), the slices are summed and the
    // sub-pixels maxed across the group's Q*S lanes with xor butterflies, and
    // lane r writes the channels kk = r (mod Q*S).  The 8 reads and the 8
    // shuffles of a step are independent and issue back to back; accumulator
    // rows past nacc (up to nacc8) hold zeros.
    if constexpr (ONE) {
#pragma unroll
      for (int j = 0; j < GB; ++j) acc_lane[j * MRS_BD] = accr[j];
    }
    wave_sync();                                          // the lane's sums are in its column
    for (int kb = 0; kb < nacc8; kb += 8) {
      A v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = acc_lane[(kb + u) * MRS_BD];
      for (int m = 1; m < S; m <<= 1) {
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] += shfl_xor_a(v[u], m);
      }
      for (int m = S; m < QS; m <<= 1) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const A o2 = shfl_xor_a(v[u], m);
          v[u] = o2 > v[u] ? o2 : v[u];
        }
      }
      if (active) {
        A* orow = otile + it * fa.ostride + gfirst * n;
        const A* brow = bias_s + gfirst * n;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int kk = kb + u;
          if (kk < nacc && (kk & (QS - 1)) == r) orow[kk] = v[u] + brow[kk];
        }
      }
    }
    wave_sync();                                          // before the accumulators are reused
  }
  __syncthreads();

  // ---- epilogue
  const RowMap rm{fa.tile_mode, fa.TW, bb, Hp, Wp, pr0, pc0, item0, fa.fd_tw};
  const int ostride = fa.ostride;
  if (fa.write_sums) {
    if (fa.tile_mode == 0 || fa.TW == Wp) {
      // the tile's slots are consecutive output rows: one contiguous block
      const int64_t o0 = rm.row(0) * c_out;
      const int tot = nslots * c_out;                     // c_out % 4 == 0 (host)
      if (ostride == c_out) {
        for (int e = tid * 4; e < tot; e += MRS_BD * 4) {
          if constexpr (sizeof(A) == 4 && sizeof(T) == 1)
            *reinterpret_cast<int4*>(y + o0 + e) = *reinterpret_cast<const int4*>(otile + e);
          else
            *reinterpret_cast<float4*>(y + o0 + e) = *reinterpret_cast<const float4*>(otile + e);
        }
      } else {
        for (int e = tid; e < tot; e += MRS_BD) {
          const int it = (int)fdiv((uint32_t)e, fa.fd_cout);
          y[o0 + e] = otile[it * ostride + (e - it * c_out)];
        }
      }
    } else {
      for (int it = wv; it < nslots; it += MRS_BD / 64) {
        if (!sm.live(it)) continue;
        A* yr = y + rm.row(it) * c_out;
        for (int e = lane; e < c_out; e += 64) yr[e] = otile[it * ostride + e];
      }
    }
  }
  if (fa.k >= 0) {
    uint2* sel = reinterpret_cast<uint2*>(smem + fa.off_sel);   // (threshold key, last winning tie)
    uint16_t* tl_idx = lo.idx ? reinterpret_cast<uint16_t*>(smem + fa.off_lidx) : nullptr;
    TO* tl_val = reinterpret_cast<TO*>(smem + fa.off_lval);     // [slots][cap] lists of the tile
    switch (fa.kmode) {
      case 1:
        kwta_quad_items<A, TO, 8>(otile, ostride, sm, rm, c_out, fa.k, fa.shift, sel, tl_idx,
                                  tl_val, lo.cap, lo.cnt);
        break;
      case 2:
        kwta_quad_items<A, TO, 16>(otile, ostride, sm, rm, c_out, fa.k, fa.shift, sel, tl_idx,
                                   tl_val, lo.cap, lo.cnt);
        break;
      default:
        kwta_quad_items<A, TO, 32>(otile, ostride, sm, rm, c_out, fa.k, fa.shift, sel, tl_idx,
                                   tl_val, lo.cap, lo.cnt);
        break;
    }
    __syncthreads();
    if (lo.idx) {
      // the tile's lists to global memory, 4 entries per store (rows are
      // cap >= 4 entries apart, cap % 4 == 0); entries past a row's count
      // are copied too and are not part of the output
      using OV = typename ChunkVal<TO>::type;
      const int cq = lo.cap >> 2;
      for (int e = tid; e < nslots * cq; e += MRS_BD) {
        const int it = (int)fdiv((uint32_t)e, fa.fd_ochunks);
        if (!sm.live(it)) continue;
        const int j = e - it * cq;
        const int64_t g = rm.row(it) * lo.cap + 4 * j;
        *reinterpret_cast<uint2*>(lo.idx + g) = reinterpret_cast<const uint2*>(tl_idx)[it * cq + j];
        *reinterpret_cast<OV*>(static_cast<TO*>(lo.val) + g) =
            reinterpret_cast<const OV*>(tl_val)[it * cq + j];
      }
    } else {
      // dense masked output in one pass over the tile, consecutive threads on
      // consecutive channels
      const bool none = fa.k == 0;
      for (int e = tid; e < nslots * c_out; e += MRS_BD) {
        const int it = (int)fdiv((uint32_t)e, fa.fd_cout);
        if (!sm.live(it)) continue;
        const int ch = e - it * c_out;
        const A a = otile[it * ostride + ch];
        const uint2 sv = sel[it];
        const uint32_t key = order_key(a);
        const bool win = !none && (key > sv.x || (key == sv.x && ch <= (int)sv.y));
        out[rm.row(it) * c_out + ch] = win ? kwta_out<A, TO>(a, fa.shift) : TO(0);
      }
    }
  }
}

}  // namespace cs
