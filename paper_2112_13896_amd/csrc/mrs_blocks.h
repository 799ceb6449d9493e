// One fp32 layer in one kernel: Multiply, Route and Sum (Section 3.2 steps
// 3-5) with the packed table streamed through LDS in blocks of rows, then
// bias, k-WTA (Section 3.3.3) and the winners written as the next layer's
// (index, value) lists (Figure 10) or densely.
//
//  * tile: P consecutive output pixels per workgroup, complete in the channel
//    dimension (every set), so k-WTA needs no round trip through HBM;
//  * lanes: (pixel, unit of GB sets), the U = G / GB lanes of a pixel
//    adjacent (they read the same list entries);
//  * table: the augmented tensor (value + Kernel ID per slot, Section 3.3.1)
//    is staged in blocks of RB slot rows - whole taps, or a channel range of
//    one tap - as 8-byte entries {value, accumulator offset} (the Kernel ID
//    already turned into the byte offset of its accumulator row), so one LDS
//    read gives a lane its sets' weights and where their products go.  A
//    table of one block is staged once per workgroup (persistent workgroups
//    loop over tiles); larger ones are double-buffered when two blocks fit:
//    the next block's loads are in flight while the current block is used,
//    one barrier per block.  A block's slots are visited in list order (a
//    list is in ascending channel order), so a lane keeps its place in a
//    tap's list from one channel block to the next;
//  * Route / Sum: the accumulators of a lane are LDS columns acc[j*n + kid]
//    [lane] (a bank is a function of the lane only), starting at the bias.
//    fp32 has no fast LDS atomic here, so each product is a read-add-write of
//    the lane's own column; the entries of a list chunk go in pairs (both
//    reads, then the writes in entry order), and the second entry of a pair
//    whose Kernel ID equals the first's adds onto the first's new value
//    instead of the value read - the same sums, in the same order, as one
//    entry after another;
//  * epilogue, when a pixel's lanes hold all its channels in their own
//    columns: the k-WTA runs on those columns with no barrier - four lanes
//    per pixel (a quad) with the gather kernels' sorted top-8/16/32 lists and
//    bit masks, or a bit-by-bit search of the k-th largest key with group
//    counts; otherwise the sums are copied to a tile and selected there (four
//    or sixteen lanes per row).  Ties go to the lower index; the winners are
//    written as lists (non-zero values, ascending index) or densely.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_fused.h"
#include "mrs_kernels.h"
#include "wave_ops.h"

namespace cs {

constexpr int BLK_BD = 256;       // threads per workgroup
constexpr int BLK_STAGE = 8;      // 16-byte table loads per thread per block (at most)
constexpr int BLK_ENTRIES = BLK_BD * BLK_STAGE * 2;   // table entries per block (at most)

struct BlocksArgs {
  int log2U;          // lanes per pixel = G / GB (a power of two)
  int P;              // pixels per tile = BLK_BD / U
  int items;          // output pixels B * Ho * Wo (no pooling)
  int ntiles;         // tiles of P pixels; workgroups loop over them
  int RB;             // slot rows per block
  int nblocks;        // ceil(R / RB)
  int tpb;            // taps per block (RB = tpb * C), or 0: a block is a channel range
  int cblocks;        // channel blocks per tap (C / RB) when tpb == 0
  int tstride;        // 8-byte entries per staged row (G + padding)
  int nbuf;           // table buffers: 2 (the next block is stored beside the
                      // one in use) or 1 (stored after a barrier)
  int log2n;          // kernels per set n = 1 << log2n
  int log2G;          // sets G = 1 << log2G
  int k;              // k-WTA winners per row; -1: sums only
  int write_sums;     // 1: the sums (bias added) are written to y
  int kmode;          // k-WTA on a copied tile: 1/2/3 four lanes per row with
                      // top-8/16/32 lists (rows <= 128, k <= 32), 4 sixteen
                      // lanes per row; on the lanes' own columns: 5 bit by bit,
                      // 6/7/8 four lanes (a pixel's quad) with top-8/16/32 lists
  int ostride;        // row stride of the sum tile (four lanes per row)
  int kp;             // channels per lane with sixteen lanes per row (4, 8 or 16)
  int log2Us;         // on the lanes' own columns: lanes per k-WTA unit (k winners
                      // per unit of KP << log2Us channels; log2U: the whole row)
  uint32_t off_t0, off_t1;   // LDS byte offsets of the table buffers
  uint32_t off_out, off_sel, off_lidx, off_lval;       // epilogue (over the table blocks)
  FastDiv fd_wo, fd_ho, fd_kw, fd_cout, fd_ochunks;
};

// The four entries of a list chunk (indices and values), read as two vectors.
struct BChunk {
  uint2 idx;
  float4 val;
};

__device__ __forceinline__ float bchunk_val(const float4& v, int e) {
  return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w));
}
__device__ __forceinline__ int bchunk_idx(const uint2& ii, int e) {
  const uint32_t wd = e < 2 ? ii.x : ii.y;
  return (int)((e & 1) ? (wd >> 16) : (wd & 0xFFFFu));
}

// Stage table rows [r0, r1) of the augmented tensor ([R][G] {value, kid})
// into a block of rows of `tstride` 8-byte entries {value, offset}: the
// offset of (row, set s) is the byte offset of the lane's accumulator row
// (s mod GB) * n + kid, i.e. ((s mod GB) * n + kid) * BLK_BD * 4, so one LDS
// read gives a lane its sets' weights and where their products go.
template <int GB>
struct BlockStage {
  uint4 v[BLK_STAGE];
  __device__ __forceinline__ void load(const uint2* __restrict__ aug, int r0, int r1, int G) {
    const int npair = (r1 - r0) * G / 2;                 // 16-byte loads (G even)
    const uint4* src = reinterpret_cast<const uint4*>(aug + (size_t)r0 * G);
#pragma unroll
    for (int u = 0; u < BLK_STAGE; ++u) {
      const int e = u * BLK_BD + (int)threadIdx.x;
      v[u] = src[e < npair ? e : npair - 1];             // in range: npair >= 1
    }
  }
  // rows [r0, r1) as loaded, placed from staged row row0 on
  __device__ __forceinline__ void store(unsigned char* smem, uint32_t off_t, int row0, int nrows,
                                        int log2G, int tstride, int log2n) const {
    const int G = 1 << log2G;
    uint2* tab = reinterpret_cast<uint2*>(smem + off_t);
    const int npair = nrows * G / 2;
    const uint32_t nm = (1u << log2n) - 1u;                // a Kernel ID is < n
#pragma unroll
    for (int u = 0; u < BLK_STAGE; ++u) {
      const int e = u * BLK_BD + (int)threadIdx.x;
      if (e < npair) {
        const int e2 = 2 * e;
        const int row = row0 + (e2 >> log2G), s = e2 & (G - 1);   // s even: one row
        const uint32_t o0 = (((uint32_t)(s % GB) << log2n) + (v[u].y & nm)) * (BLK_BD * 4);
        const uint32_t o1 = (((uint32_t)((s + 1) % GB) << log2n) + (v[u].w & nm)) * (BLK_BD * 4);
        *reinterpret_cast<uint4*>(tab + row * tstride + s) = make_uint4(v[u].x, o0, v[u].z, o1);
      }
    }
  }
};

// One list chunk against the staged block, GB sets of the lane.  Entry e is
// live when e in [e_lo, e_hi); a dead entry reads row 0 and adds a zero.
// Route + Sum: the entries go in pairs; both reads of a pair are issued, then
// the two writes in entry order, the second entry adding onto the first's new
// value when their accumulators are the same (equal offsets <=> equal Kernel
// IDs) - the same sums, in the same order, as one entry after another.
template <int GB>
__device__ __forceinline__ void blk_chunk(const BChunk& ch, int e_lo, int e_hi, int row_add,
                                          const uint2* tab, int tstride, int set0,
                                          unsigned char* accb) {
  CS_COUNT_PRODUCTS_ADD((e_hi - e_lo) * GB);
  float x[4];
  uint2 te[4][GB];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ok = e >= e_lo && e < e_hi;
    const int r = ok ? bchunk_idx(ch.idx, e) + row_add : 0;
    x[e] = ok ? bchunk_val(ch.val, e) : 0.f;
    const uint2* tp = tab + __umul24(r, tstride) + set0;
    if constexpr (GB == 1) {
      te[e][0] = tp[0];
    } else if constexpr (GB == 2) {
      const uint4 q = *reinterpret_cast<const uint4*>(tp);
      te[e][0] = make_uint2(q.x, q.y);
      te[e][1] = make_uint2(q.z, q.w);
    } else {
      const uint4 q0 = *reinterpret_cast<const uint4*>(tp);
      const uint4 q1 = *reinterpret_cast<const uint4*>(tp + 2);
      te[e][0] = make_uint2(q0.x, q0.y);
      te[e][1] = make_uint2(q0.z, q0.w);
      te[e][2] = make_uint2(q1.x, q1.y);
      te[e][3] = make_uint2(q1.z, q1.w);
    }
  }
#pragma unroll
  for (int pr = 0; pr < 4; pr += 2) {
    float a[2][GB];
#pragma unroll
    for (int j = 0; j < GB; ++j) {
      a[0][j] = *reinterpret_cast<const float*>(accb + te[pr][j].y);
      a[1][j] = *reinterpret_cast<const float*>(accb + te[pr + 1][j].y);
    }
#pragma unroll
    for (int j = 0; j < GB; ++j) {
      const float v0 = __builtin_fmaf(x[pr], __uint_as_float(te[pr][j].x), a[0][j]);
      const float b1 = te[pr + 1][j].y == te[pr][j].y ? v0 : a[1][j];
      const float v1 = __builtin_fmaf(x[pr + 1], __uint_as_float(te[pr + 1][j].x), b1);
      *reinterpret_cast<float*>(accb + te[pr][j].y) = v0;
      *reinterpret_cast<float*>(accb + te[pr + 1][j].y) = v1;
    }
  }
}

// A tap's list count and first list entries, loaded ahead of their use.
// QD false: the lane loads the first BLK_SPEC chunks itself.  QD true (a
// pixel's lanes fill whole quads, U >= 4): the four lanes of a quad load one
// chunk each - lane p the chunk at (j0 rounded down to 4) + 4p - and pass them
// round with DPP, so a wavefront issues one load per array for sixteen
// entries of its sixteen pixels instead of one per chunk and lane.  Every
// load is issued unconditionally (a tap outside the image reads list row 0, a
// chunk past the row's capacity reads the row's last chunk, which is then
// never used), so the compiler's wait counts stay exact and a later load
// never waits for them.
constexpr int BLK_SPEC = 3;
// Whole-tap mode: the list data of the next BLK_DEPTH taps is in flight while
// a tap is processed.
constexpr int BLK_DEPTH = 1;
template <bool QD>
struct TapPre {
  int off;                 // list row offset, or -1: the tap is outside the image
  int cnt;
  BChunk ch[QD ? 1 : BLK_SPEC];
};

template <bool QD>
__device__ __forceinline__ void tap_prefetch(TapPre<QD>& tp, const uint16_t* __restrict__ lidx,
                                             const float* __restrict__ lval,
                                             const int32_t* __restrict__ lcnt, const ConvGeom& geo,
                                             bool live, int bb, int ho, int wo, int t, int j0,
                                             const FastDiv& fd_kw) {
  const int ky = (int)fdiv((uint32_t)t, fd_kw), kx = t - ky * geo.KW;
  const int hy = ho * geo.S + ky - geo.P, wx = wo * geo.S + kx - geo.P;
  const bool ok = live && t < geo.KH * geo.KW && hy >= 0 && hy < geo.H && wx >= 0 && wx < geo.W;
  const int q = ok ? (bb * geo.H + hy) * geo.W + wx : 0;   // < 2^31 (host)
  const int base = q * geo.cap;
  tp.off = ok ? base : -1;
  tp.cnt = lcnt[q];
  const int c4 = j0 & ~3;
  if constexpr (QD) {
    const int pos = min(c4 + 4 * (int)(threadIdx.x & 3), geo.cap - 4);
    tp.ch[0].idx = *reinterpret_cast<const uint2*>(lidx + base + pos);
    tp.ch[0].val = *reinterpret_cast<const float4*>(lval + base + pos);
  } else {
#pragma unroll
    for (int s2 = 0; s2 < BLK_SPEC; ++s2) {
      const int pos = min(c4 + 4 * s2, geo.cap - 4);
      tp.ch[s2].idx = *reinterpret_cast<const uint2*>(lidx + base + pos);
      tp.ch[s2].val = *reinterpret_cast<const float4*>(lval + base + pos);
    }
  }
}

// Lane s's chunk of the quad (s a constant after unrolling): a DPP broadcast
// within each quad, whose four lanes are active together (they serve one
// pixel, so they take the same branches).
__device__ __forceinline__ uint32_t quad_bcast(uint32_t v, int s) {
  switch (s) {
    case 0: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x00, 0xF, 0xF, false);
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x55, 0xF, 0xF, false);
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xAA, 0xF, 0xF, false);
    default: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xFF, 0xF, 0xF, false);
  }
}
__device__ __forceinline__ BChunk quad_bcast(const BChunk& c, int s) {
  BChunk r;
  r.idx.x = quad_bcast(c.idx.x, s);
  r.idx.y = quad_bcast(c.idx.y, s);
  r.val.x = __uint_as_float(quad_bcast(__float_as_uint(c.val.x), s));
  r.val.y = __uint_as_float(quad_bcast(__float_as_uint(c.val.y), s));
  r.val.z = __uint_as_float(quad_bcast(__float_as_uint(c.val.z), s));
  r.val.w = __uint_as_float(quad_bcast(__float_as_uint(c.val.w), s));
  return r;
}

// Entries e of chunk `ch` (list positions c4 + e) with e in [lo, m - c4) and,
// in channel mode, a channel below c_hi: processed; returns the chunk entry
// where the lane stopped (4 when it went through the chunk).
template <int GB, bool CH>
__device__ __forceinline__ int blk_chunk_upto(const BChunk& ch, int lo, int m, int c4, int c_hi,
                                              int row_add, const uint2* tab, int tstride, int set0,
                                              unsigned char* accb) {
  const int hi = m - c4 < 4 ? m - c4 : 4;
  int stop = hi;
  if constexpr (CH) {
#pragma unroll
    for (int e = 3; e >= 0; --e)
      if (e < hi && bchunk_idx(ch.idx, e) >= c_hi) stop = e;   // the list ascends
  }
  blk_chunk<GB>(ch, lo, stop, row_add, tab, tstride, set0, accb);
  return stop < hi ? stop : 4;
}

// The entries of one tap's list from position j0 on (and, in channel mode,
// below channel c_hi), the first chunks already in `tp`; the rest are read
// ahead (QD false: one chunk, QD true: the quad's next sixteen entries).
// Returns the list position where the lane stopped.
template <int GB, bool CH, bool QD>
__device__ __forceinline__ int blk_tap(const TapPre<QD>& tp, const uint16_t* __restrict__ lidx,
                                       const float* __restrict__ lval, int cap, int j0, int c_hi,
                                       int row_add, const uint2* tab, int tstride, int set0,
                                       unsigned char* accb) {
  if (tp.off < 0) return j0;
  const int m = min(tp.cnt, cap);
  int c4 = j0 & ~3;
  int lo = j0 - c4;
  const uint16_t* li = lidx + tp.off;
  const float* lv = lval + tp.off;
  if constexpr (QD) {
    BChunk mine = tp.ch[0];                              // entries g0 + 4p .. of the quad
    int g0 = c4;
    while (true) {
      const bool more = g0 + 16 < m;                     // the same in the quad
      BChunk nmine;
      if (more) {
        const int pos = min(g0 + 16 + 4 * (int)(threadIdx.x & 3), cap - 4);
        nmine.idx = *reinterpret_cast<const uint2*>(li + pos);
        nmine.val = *reinterpret_cast<const float4*>(lv + pos);
      }
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) {
        if (c4 >= m) return m;
        const BChunk cs = quad_bcast(mine, s2);
        const int st = blk_chunk_upto<GB, CH>(cs, lo, m, c4, c_hi, row_add, tab, tstride, set0,
                                              accb);
        if (st < 4) return c4 + st;
        c4 += 4;
        lo = 0;
      }
      if (!more) return m;
      mine = nmine;
      g0 += 16;
    }
  } else {
#pragma unroll
    for (int s2 = 0; s2 < BLK_SPEC; ++s2) {
      if (c4 >= m) return m;
      const int st = blk_chunk_upto<GB, CH>(tp.ch[s2], lo, m, c4, c_hi, row_add, tab, tstride,
                                            set0, accb);
      if (st < 4) return c4 + st;
      c4 += 4;
      lo = 0;
    }
    if (c4 >= m) return m;
    BChunk cur;
    cur.idx = *reinterpret_cast<const uint2*>(li + c4);
    cur.val = *reinterpret_cast<const float4*>(lv + c4);
    while (true) {
      const int pn = min(c4 + 4, cap - 4);               // next chunk, in the row
      BChunk nxt;
      nxt.idx = *reinterpret_cast<const uint2*>(li + pn);
      nxt.val = *reinterpret_cast<const float4*>(lv + pn);
      const int st = blk_chunk_upto<GB, CH>(cur, 0, m, c4, c_hi, row_add, tab, tstride, set0,
                                            accb);
      if (st < 4) return c4 + st;
      c4 += 4;
      if (c4 >= m) return m;
      cur = nxt;
    }
  }
}

// k-WTA with sixteen lanes per row (rows of up to 256 channels, any k): lane
// l of a row holds channels l*KP .. l*KP+KP-1 (read from the accumulator
// columns, bias added), the k-th largest key is found bit by bit with
// sixteen-lane counts, stopping as soon as the keys at or above the prefix
// are exactly k (their minimum is then the k-th largest); ties go to the
// lower index; winners are written as lists (non-zero values, ascending
// index) or densely.  Four rows per wavefront at a time.
template <typename TO, int GB, int KP>
__device__ __forceinline__ void blk_kwta16(const float* acc, int item0, int nrows, int P,
                                           int log2U, int log2n, int c_out, int k,
                                           int write_sums, float* __restrict__ y,
                                           TO* __restrict__ out, const ListOut& lo) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int l16 = lane & 15;
  const int n = 1 << log2n;
  for (int r0 = wv * 4; r0 < P; r0 += BLK_BD / 16) {
    const int r = r0 + (lane >> 4);
    const bool live_r = r < nrows;
    const int64_t row = (int64_t)item0 + r;
    float v[KP];
    uint32_t key[KP];
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const int o = l16 * KP + j;
      const bool ok = live_r && o < c_out;
      float sv = 0.f;
      if (ok) {
        const int g = o >> log2n, kk = o & (n - 1);
        sv = acc[((g % GB) * n + kk) * BLK_BD + (r << log2U) + g / GB];
        if (write_sums) y[row * c_out + o] = sv;
      }
      v[j] = sv;
      key[j] = ok ? order_key(sv) : 0u;                 // 0: below every real key
    }
    if (k < 0) continue;
    uint32_t thr = 0u;
    int need = 0;
    if (k > 0 && k < c_out) {
      uint32_t pre = 0u;
      int cntp = c_out;
      bool done = !live_r;
      for (int bit = 31; bit >= 0; --bit) {
        if (__ballot(!done) == 0ull) break;             // every row of the wavefront found
        const uint32_t cand = pre | (1u << bit);
        uint32_t c = 0;
#pragma unroll
        for (int j = 0; j < KP; ++j) c += key[j] >= cand ? 1u : 0u;
        c = row16_reduce(c, OpAdd{});
        if (!done) {
          if ((int)c >= k) {
            pre = cand;
            cntp = (int)c;
          }
          if (cntp == k) done = true;
        }
      }
      // the k-th largest key: the least key at or above the prefix
      uint32_t mn = 0xFFFFFFFFu;
#pragma unroll
      for (int j = 0; j < KP; ++j) mn = (key[j] >= pre && key[j] < mn) ? key[j] : mn;
      thr = row16_reduce(mn, OpMin{});
      uint32_t gt = 0;
#pragma unroll
      for (int j = 0; j < KP; ++j) gt += key[j] > thr ? 1u : 0u;
      gt = row16_reduce(gt, OpAdd{});
      need = k - (int)gt;
    }
    // ties in index order: this lane's first tie has rank (ties of the lanes before)
    int eq = 0;
#pragma unroll
    for (int j = 0; j < KP; ++j) eq += (k > 0 && k < c_out && key[j] == thr) ? 1 : 0;
    int tie_rank = row16_incl_sum(eq) - eq;
    bool win[KP];
    int wcount = 0;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const int o = l16 * KP + j;
      const bool ok = live_r && o < c_out;
      bool w;
      if (!ok || k == 0) {
        w = false;
      } else if (k >= c_out) {
        w = true;
      } else if (key[j] > thr) {
        w = true;
      } else if (key[j] == thr) {
        w = tie_rank < need;
        ++tie_rank;
      } else {
        w = false;
      }
      win[j] = w;
      wcount += (lo.idx ? (w && v[j] != 0.f) : w) ? 1 : 0;
    }
    if (lo.idx) {
      const int incl = row16_incl_sum(wcount);
      int pos = incl - wcount;
      if (live_r) {
        uint16_t* oi = lo.idx + row * lo.cap;
        TO* ov = static_cast<TO*>(lo.val) + row * lo.cap;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
          if (win[j] && v[j] != 0.f) {
            oi[pos] = (uint16_t)(l16 * KP + j);
            ov[pos] = (TO)v[j];
            ++pos;
          }
        }
        if (l16 == 15) lo.cnt[row] = incl;
      }
    } else if (live_r) {
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        const int o = l16 * KP + j;
        if (o < c_out) out[row * c_out + o] = win[j] ? (TO)v[j] : TO(0);
      }
    }
  }
}

// The epilogue on a tile copied from the accumulator columns (any lane
// layout): k-WTA with sixteen lanes per row, or with four lanes per row on a
// row-major tile (the gather kernel's selection) followed by the lists'
// copy-out; sums only when k < 0.
template <typename TO, int GB>
__device__ __forceinline__ void blk_epilogue_tile(unsigned char* smem, const float* acc,
                                                  int item0, int c_out, float* __restrict__ y,
                                                  TO* __restrict__ out, const ListOut& lo,
                                                  const BlocksArgs& ba) {
  const int tid = threadIdx.x;
  const int n = 1 << ba.log2n;
  const int nrows = min(ba.P, ba.items - item0);         // live rows of the tile
  __syncthreads();                                       // every lane's sums are in LDS
  if (ba.kmode == 4 || ba.k < 0) {
    if (ba.kp == 4)
      blk_kwta16<TO, GB, 4>(acc, item0, nrows, ba.P, ba.log2U, ba.log2n, c_out, ba.k,
                            ba.write_sums, y, out, lo);
    else if (ba.kp == 8)
      blk_kwta16<TO, GB, 8>(acc, item0, nrows, ba.P, ba.log2U, ba.log2n, c_out, ba.k,
                            ba.write_sums, y, out, lo);
    else
      blk_kwta16<TO, GB, 16>(acc, item0, nrows, ba.P, ba.log2U, ba.log2n, c_out, ba.k,
                             ba.write_sums, y, out, lo);
    return;
  }
  // four lanes per row: the sums into a row-major tile with an odd row stride
  // over the table blocks (no longer read), then the gather kernel's selection
  const int ostride = ba.ostride;
  float* otile = reinterpret_cast<float*>(smem + ba.off_out);
  for (int e = tid; e < nrows * c_out; e += BLK_BD) {
    const int r = (int)fdiv((uint32_t)e, ba.fd_cout), o = e - r * c_out;
    const int g = o >> ba.log2n, kk = o & (n - 1);
    const float sv = acc[((g % GB) * n + kk) * BLK_BD + (r << ba.log2U) + g / GB];
    otile[r * ostride + o] = sv;
    if (ba.write_sums) y[(int64_t)item0 * c_out + e] = sv;
  }
  __syncthreads();
  const FastDiv one{1u, 0u, 0u};
  const SlotMap sm{0, 1, 0, nrows, one};
  const RowMap rm{0, 1, 0, 0, 0, 0, 0, (int64_t)item0, one};
  uint2* sel = reinterpret_cast<uint2*>(smem + ba.off_sel);
  uint16_t* tl_idx = lo.idx ? reinterpret_cast<uint16_t*>(smem + ba.off_lidx) : nullptr;
  TO* tl_val = reinterpret_cast<TO*>(smem + ba.off_lval);
  if (ba.kmode == 1)
    kwta_quad_items<float, TO, 8, BLK_BD>(otile, ostride, sm, rm, c_out, ba.k, 0, sel, tl_idx,
                                          tl_val, lo.cap, lo.cnt);
  else if (ba.kmode == 2)
    kwta_quad_items<float, TO, 16, BLK_BD>(otile, ostride, sm, rm, c_out, ba.k, 0, sel, tl_idx,
                                           tl_val, lo.cap, lo.cnt);
  else
    kwta_quad_items<float, TO, 32, BLK_BD>(otile, ostride, sm, rm, c_out, ba.k, 0, sel, tl_idx,
                                           tl_val, lo.cap, lo.cnt);
  __syncthreads();
  if (lo.idx) {
    // the tile's lists, 4 entries per store (cap % 4 == 0); entries past a
    // row's count are copied too and are not part of the output
    const int cq = lo.cap >> 2;
    for (int e = tid; e < nrows * cq; e += BLK_BD) {
      const int it = (int)fdiv((uint32_t)e, ba.fd_ochunks);
      const int j = e - it * cq;
      const int64_t g = ((int64_t)item0 + it) * lo.cap + 4 * j;
      *reinterpret_cast<uint2*>(lo.idx + g) = reinterpret_cast<const uint2*>(tl_idx)[it * cq + j];
      *reinterpret_cast<float4*>(static_cast<TO*>(lo.val) + g) =
          reinterpret_cast<const float4*>(tl_val)[it * cq + j];
    }
  } else {
    const bool none = ba.k == 0;
    for (int e = tid; e < nrows * c_out; e += BLK_BD) {
      const int it = (int)fdiv((uint32_t)e, ba.fd_cout);
      const int ch = e - it * c_out;
      const float a = otile[it * ostride + ch];
      const uint2 sv = sel[it];
      const uint32_t key = order_key(a);
      const bool win = !none && (key > sv.x || (key == sv.x && ch <= (int)sv.y));
      out[(int64_t)item0 * c_out + e] = win ? (TO)a : TO(0);
    }
  }
}

// Reductions and prefix sums over aligned groups of U = 1 << log2U lanes
// (U <= 16, inside one DPP row): xor 1 and xor 2 within quads, then the
// half-row mirror (joins the two quads of an 8-lane group) and the row mirror
// (joins the two halves of a 16-lane row).  Every lane of the wavefront must
// take part; every lane of a group ends with the group's result.
template <typename Op>
__device__ __forceinline__ uint32_t group_reduce(uint32_t v, int log2U, Op op) {
  if (log2U >= 1) v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));
  if (log2U >= 2) v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));
  if (log2U >= 3) v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));
  if (log2U >= 4) v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));
  return v;
}
// Inclusive prefix sum over the group, lane position p = lane & (U - 1):
// row shifts by 1, 2, 4, 8 taken only from lanes of the same group.
__device__ __forceinline__ int group_incl_sum(int v, int log2U, int p) {
  if (log2U >= 1) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false); v += p >= 1 ? t : 0; }
  if (log2U >= 2) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false); v += p >= 2 ? t : 0; }
  if (log2U >= 3) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false); v += p >= 4 ? t : 0; }
  if (log2U >= 4) { const int t = __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false); v += p >= 8 ? t : 0; }
  return v;
}

// Clamped 16-bit subtraction, minimum and sum on two halves at once (integer
// packed operations), and 32-bit minimum and sum: written out so that the
// compiler keeps them as they are instead of turning a minimum with 1 into a
// compare (one chain through VCC) or a tree of sums into one chain.
__device__ __forceinline__ uint32_t pk_sub_sat_u16(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_pk_sub_u16 %0, %1, %2 clamp" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
__device__ __forceinline__ uint32_t pk_min_u16(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
__device__ __forceinline__ uint32_t min_u32(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_min_u32 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
__device__ __forceinline__ uint32_t add_u32(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_add_u32 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
__device__ __forceinline__ uint32_t pk_add_u16(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_pk_add_u16 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}

// How many of the 2N 16-bit values packed in h are below c16: per half,
// min(c16 -sat value, 1) is 1 exactly then; the 0/1 halves are added in a
// tree (the adds written out too, so the compiler does not turn the tree
// into one long chain of dependent adds).
template <int N>
__device__ __forceinline__ uint32_t below16(const uint32_t (&h)[N], uint32_t c16) {
  const uint32_t c2 = c16 | (c16 << 16);
  uint32_t m[N];
#pragma unroll
  for (int i = 0; i < N; ++i) m[i] = pk_min_u16(pk_sub_sat_u16(c2, h[i]), 0x00010001u);
#pragma unroll
  for (int w = 1; w < N; w *= 2)
#pragma unroll
    for (int i = 0; i + w < N; i += 2 * w) m[i] = pk_add_u16(m[i], m[i + w]);
  return (m[0] & 0xFFFFu) + (m[0] >> 16);
}

// Sum over the aligned groups of 2^log2U lanes (log2U <= 4) without
// branches: each of the four DPP steps adds its partner's value masked by
// mk[s] (all ones when the group spans that step, else zero), the masks
// made once by group_masks.
__device__ __forceinline__ void group_masks(int log2U, uint32_t (&mk)[4]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) mk[s] = log2U > s ? 0xFFFFFFFFu : 0u;
}
// In-place transpose of a 32 x 32 bit matrix held as 32 words: afterwards
// bit j of a[b] is bit b of the original a[j] (five stages of block swaps,
// each row pair by two shifts and two bit-field selects).
__device__ __forceinline__ void bit_transpose32(uint32_t (&a)[32]) {
  constexpr uint32_t M[5] = {0x0000FFFFu, 0x00FF00FFu, 0x0F0F0F0Fu, 0x33333333u, 0x55555555u};
#pragma unroll
  for (int st = 0; st < 5; ++st) {
    const int w = 16 >> st;
    const uint32_t m = M[st];
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      if (j & w) continue;
      const uint32_t x = a[j], y = a[j + w];
      a[j] = (x & m) | ((y << w) & ~m);
      a[j + w] = ((x >> w) & m) | (y & ~m);
    }
  }
}
__device__ __forceinline__ uint32_t group_min_nb(uint32_t v, const uint32_t (&mk)[4]) {
  uint32_t t;
  t = (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false) | ~mk[0];
  v = t < v ? t : v;
  t = (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false) | ~mk[1];
  v = t < v ? t : v;
  t = (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false) | ~mk[2];
  v = t < v ? t : v;
  t = (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false) | ~mk[3];
  v = t < v ? t : v;
  return v;
}
__device__ __forceinline__ uint32_t group_sum_nb(uint32_t v, const uint32_t (&mk)[4]) {
  v += (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false) & mk[0];
  v += (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false) & mk[1];
  v += (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false) & mk[2];
  v += (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false) & mk[3];
  return v;
}

// k-WTA over the U lanes of each pixel, the lanes that computed its sums: lane
// u holds channels u*KP .. u*KP+KP-1 (KP = GB * n) in its own accumulator
// column, bias included, so no other lane's data is read and no barrier is
// needed.  The row is split into units of Us = 1 << log2Us lanes (KP * Us
// channels; Us = U: the whole row), each keeping its own k winners (the k-WTA
// in units of Section 5's channel partitioning).  The k-th largest key of a
// unit is found bit by bit with group counts, stopping as soon as the keys at
// or above the prefix are exactly k (their minimum is then the k-th largest);
// the counts of the upper sixteen bits compare the keys' high halves and those
// of the lower sixteen the low halves of the keys that share the prefix's high
// half, two halves per packed instruction.  Ties go to the lower index; the
// winners of the whole row are written as one list (non-zero values,
// ascending index) or densely.
template <typename TO, int KP>
__device__ __forceinline__ void blk_kwta_own(const float* acc, int log2U, int log2Us,
                                             int64_t row, bool live, int c_out, int k,
                                             int write_sums, float* __restrict__ y,
                                             TO* __restrict__ out, const ListOut& lo) {
  const int tid = threadIdx.x;
  const int p = tid & ((1 << log2U) - 1);                // lane position in the group
  const int ps = p & ((1 << log2Us) - 1);                // lane position in its unit
  const int c_unit = KP << log2Us;                       // channels per k-WTA unit
  const int o0 = p * KP;                                 // first channel of the lane
  float v[KP];
  uint32_t key[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    v[j] = acc[j * BLK_BD + tid];
    key[j] = live ? order_key(v[j]) : 0u;                // 0: below every real key
  }
  if (write_sums && live) {
    float* yr = y + row * c_out + o0;                    // 16-byte aligned (host)
#pragma unroll
    for (int j = 0; j < KP; j += 4)
      *reinterpret_cast<float4*>(yr + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
  }
  if (k < 0) return;
  uint32_t thr = 0u;
  int need = 0;
  // KP == 32: the search leaves the winners as masks (bit j: key j) — keys
  // above the final prefix, and keys that still match it
  uint32_t gtm32 = 0u, eqm32 = 0u;
  if (k > 0 && k < c_unit) {
    uint32_t pre = 0u;
    int cntp = c_unit;
    bool done = !live;
    // one step of the search: the unit's keys at or above pre | bit, from
    // this lane's count c (every lane of a unit takes part in the reduction)
    uint32_t mk[4];
    group_masks(log2Us, mk);
    auto step = [&](uint32_t cand, uint32_t c) {
      c = group_sum_nb(c, mk);
      if (!done) {
        if ((int)c >= k) {
          pre = cand;
          cntp = (int)c;
        }
        if (cntp == k) done = true;
      }
    };
    if constexpr (KP == 32) {
      // bit-sliced: plane b holds bit b of the lane's 32 keys (bit j: key
      // j), so a step's count is the keys already above the prefix plus one
      // bit count of the planes' AND with the keys that still match it
      uint32_t sl[32];
#pragma unroll
      for (int j = 0; j < 32; ++j) sl[j] = key[j];
      bit_transpose32(sl);
      uint32_t match = 0xFFFFFFFFu, above = 0u, above_m = 0u;
      // the group masks as vector values (an AND each, instead of selects on
      // scalar conditions the compiler spills at this register pressure)
      uint32_t mv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        mv[q] = mk[q];
        asm volatile("" : "+v"(mv[q]));
      }
      // each step branch-free: a unit still searching takes bit b when at
      // least k keys are at or above the candidate, else the matching keys
      // with bit b set are above the prefix from now on (k as a vector value:
      // the scalar one is a spilled argument, reloaded every step)
      int kv = k;
      asm volatile("" : "+v"(kv));
#pragma unroll
      for (int bit = 31; bit >= 0; --bit) {
        if (__ballot(!done) == 0ull) break;              // every unit of the wavefront found
        const uint32_t hit = match & sl[bit];
        const uint32_t nh = (uint32_t)__popc(hit);
        uint32_t c = above + nh;
        if (log2Us == 3) {
          // units of eight lanes: three DPP adds with no masks
          c += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)c, 0xB1, 0xF, 0xF, false);
          c += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)c, 0x4E, 0xF, 0xF, false);
          c += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)c, 0x141, 0xF, 0xF, false);
        } else {
          c = group_sum_nb(c, mv);
        }
        const bool take = !done && (int)c >= kv;
        const bool drop = !done && (int)c < kv;
        pre = take ? (pre | (1u << bit)) : pre;
        cntp = take ? (int)c : cntp;
        match = take ? hit : (drop ? (match & ~sl[bit]) : match);
        above = drop ? above + nh : above;
        above_m = drop ? (above_m | hit) : above_m;
        done = done || cntp == kv;
      }
      // keys above the prefix are above the k-th largest; the matching ones
      // are its copies when the search ran to bit 0, else (cntp == k) keys
      // that all win
      gtm32 = above_m;
      eqm32 = match;
    } else {
    // bits 31..16 on the keys' high halves, two to a register (a candidate's
    // low half is 0 there, so key >= cand is a compare of the high halves)
    {
      uint32_t hp[KP / 2];
#pragma unroll
      for (int i = 0; i < KP / 2; ++i) hp[i] = (key[2 * i] >> 16) | (key[2 * i + 1] & 0xFFFF0000u);
      for (int bit = 31; bit >= 16; --bit) {
        if (__ballot(!done) == 0ull) break;              // every unit of the wavefront found
        const uint32_t cand = pre | (1u << bit);
        step(cand, (uint32_t)KP - below16(hp, cand >> 16));
      }
    }
    // bits 15..0: only keys whose high half is the prefix's compete, on their
    // low halves (the others hold 0, below every candidate, whose low half is
    // at least 1); keys with a larger high half count in every step
    if (__ballot(!done) != 0ull) {
      const uint32_t ph = pre >> 16;
      uint32_t lp[KP / 2];
      uint32_t above = 0;
#pragma unroll
      for (int i = 0; i < KP / 2; ++i) {
        const uint32_t k0 = key[2 * i], k1 = key[2 * i + 1];
        lp[i] = ((k0 >> 16) == ph ? (k0 & 0xFFFFu) : 0u) | ((k1 >> 16) == ph ? (k1 << 16) : 0u);
        above += ((k0 >> 16) > ph ? 1u : 0u) + ((k1 >> 16) > ph ? 1u : 0u);
      }
      for (int bit = 15; bit >= 0; --bit) {
        if (__ballot(!done) == 0ull) break;
        const uint32_t cand = pre | (1u << bit);
        step(cand, above + (uint32_t)KP - below16(lp, cand & 0xFFFFu));
      }
    }
    }
    CS_STAMP(19);
    if constexpr (KP != 32) {
    // the k-th largest key: the least key at or above the prefix.  key - pre
    // wraps the keys below the prefix above every key at or above it, so the
    // least of the differences (a tree of minima, then the group's) is the
    // least key at or above the prefix minus the prefix; the unit has cntp
    // >= k > 0 such keys
    uint32_t d[KP];
#pragma unroll
    for (int j = 0; j < KP; ++j) d[j] = key[j] - pre;
#pragma unroll
    for (int w = 1; w < KP; w *= 2)
#pragma unroll
      for (int j = 0; j + w < KP; j += 2 * w) d[j] = d[j] < d[j + w] ? d[j] : d[j + w];
    thr = group_min_nb(d[0], mk) + pre;
    // keys above the threshold: the cntp keys at or above the prefix are the
    // threshold's copies and the keys above it; the copies are counted with
    // min(key ^ thr, 1), 0 exactly for a copy (a tree of sums, no compares)
#pragma unroll
    for (int j = 0; j < KP; ++j) d[j] = min_u32(key[j] ^ thr, 1u);
#pragma unroll
    for (int w = 1; w < KP; w *= 2)
#pragma unroll
      for (int j = 0; j + w < KP; j += 2 * w) d[j] = add_u32(d[j], d[j + w]);
    const uint32_t eq_unit = group_sum_nb((uint32_t)KP - d[0], mk);
    need = k - (cntp - (int)eq_unit);
    }
  }
  uint32_t winm = 0;                                    // bit j: channel o0 + j wins
  uint32_t putm = 0;                                    // ... and has a non-zero value
  if constexpr (KP == 32) {
    // need = k minus the unit's keys above; the first `need` matching keys
    // of the unit in index order win (every lane takes part in the sums)
    uint32_t mk2[4];
    group_masks(log2Us, mk2);
    const int nabove = (int)group_sum_nb((uint32_t)__popc(gtm32), mk2);
    const int eq_l = __popc(eqm32);
    const int tie0 = group_incl_sum(eq_l, log2Us, ps) - eq_l;
    int m = k - nabove - tie0;
    m = m < 0 ? 0 : (m > eq_l ? eq_l : m);
    uint32_t tm = m >= eq_l ? eqm32 : 0u;
    if (m > 0 && m < eq_l) {                            // a tie split at this lane (rare)
      for (uint32_t e2 = eqm32; m > 0; --m) {
        const uint32_t lb = e2 & (0u - e2);
        tm |= lb;
        e2 ^= lb;
      }
    }
    winm = (!live || k == 0) ? 0u : (k >= c_unit ? 0xFFFFFFFFu : (gtm32 | tm));
    putm = winm;
    if (lo.idx) {
      // winners whose value is exactly zero are left out of the list
      for (uint32_t w = winm; w != 0u; w &= w - 1u) {
        const int j = __builtin_ctz(w);
        if (acc[j * BLK_BD + threadIdx.x] == 0.f) putm &= ~(1u << j);
      }
    }
  } else {
  // ties in index order: this lane's first tie has rank (ties of the unit's
  // lanes before)
  int eq = 0;
#pragma unroll
  for (int j = 0; j < KP; ++j) eq += (k > 0 && k < c_unit && key[j] == thr) ? 1 : 0;
  int tie_rank = group_incl_sum(eq, log2Us, ps) - eq;
#pragma unroll
  for (int j = 0; j < KP; ++j) {
    bool w;
    if (!live || k == 0) {
      w = false;
    } else if (k >= c_unit) {
      w = true;
    } else if (key[j] > thr) {
      w = true;
    } else if (key[j] == thr) {
      w = tie_rank < need;
      ++tie_rank;
    } else {
      w = false;
    }
    winm |= w ? 1u << j : 0u;
    putm |= (w && v[j] != 0.f) ? 1u << j : 0u;
  }
  }
  const int wcount = __popc(lo.idx ? putm : winm);
  CS_STAMP(20);
  if (lo.idx) {
    const int incl = group_incl_sum(wcount, log2U, p);
    int pos = incl - wcount;
    if (live) {
      uint16_t* oi = lo.idx + row * lo.cap;
      TO* ov = static_cast<TO*>(lo.val) + row * lo.cap;
      // one pass per winner of the lane (a few), the value read back from
      // the lane's own column, instead of KP predicated slots
      for (uint32_t w = putm; w != 0u; w &= w - 1u) {
        const int j = __builtin_ctz(w);
        oi[pos] = (uint16_t)(o0 + j);
        ov[pos] = (TO)acc[j * BLK_BD + threadIdx.x];
        ++pos;
      }
      if (p == (1 << log2U) - 1) lo.cnt[row] = incl;
    }
  } else if (live) {
    TO* orow = out + row * c_out + o0;
#pragma unroll
    for (int j = 0; j < KP; j += 4)
      *reinterpret_cast<float4*>(orow + j) =
          make_float4((winm >> j) & 1u ? v[j] : 0.f, (winm >> (j + 1)) & 1u ? v[j + 1] : 0.f,
                      (winm >> (j + 2)) & 1u ? v[j + 2] : 0.f, (winm >> (j + 3)) & 1u ? v[j + 3] : 0.f);
  }
}

// KP: channels per lane (GB * n) when the k-WTA runs on the lanes' own
// accumulator columns; 0: the selection of ba.kmode on a copied tile.  Up to
// 16 channels per lane the registers are held to three wavefronts per SIMD.
// QK: with the four-lane selection in place (kmode 6-8), its list length
// (8, 16 or 32); 0 otherwise.  QD: a pixel's lanes fill whole quads (U >= 4),
// whose lanes share the list loads.
template <typename TO, int GB, bool CH, int KP, int QK, bool QD>
__global__ __launch_bounds__(BLK_BD, (KP > 0 && KP <= 16) ? 3 : 2) void mrs_blocks_f32(const uint16_t* __restrict__ lidx,
                                                         const float* __restrict__ lval,
                                                         const int32_t* __restrict__ lcnt,
                                                         const uint2* __restrict__ aug,
                                                         const float* __restrict__ bias,
                                                         float* __restrict__ y,
                                                         TO* __restrict__ out, ListOut lo,
                                                         ConvGeom geo, BlocksArgs ba) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int n = 1 << ba.log2n;
  const int G = geo.G;
  const int C = geo.C;
  const int T_ = geo.KH * geo.KW;
  const int R = T_ * C;
  const int c_out = geo.c_out;
  const int U = 1 << ba.log2U;
  const int ps = tid >> ba.log2U;                        // pixel slot of the lane
  const int u = tid & (U - 1);                           // unit: sets u*GB .. u*GB+GB-1
  const int nacc = GB << ba.log2n;                       // the lane's channels u*nacc ..
  float* acc = reinterpret_cast<float*>(smem);           // [GB * n][BLK_BD]
  unsigned char* accb = smem + tid * 4;                  // this lane's column
  const bool one_block = ba.nblocks == 1;
  BlockStage<GB> st;
  auto stage_first = [&]() {
    // the first block, in passes of BLK_ENTRIES entries (a single block may
    // be larger than what one pass holds in registers)
    const int rb0 = min(R, ba.RB);
    const int rpp = BLK_ENTRIES >> ba.log2G;              // rows per pass
    for (int rs = 0; rs < rb0; rs += rpp) {
      const int re = min(rb0, rs + rpp);
      st.load(aug, rs, re, G);
      st.store(smem, ba.off_t0, rs, re - rs, ba.log2G, ba.tstride, ba.log2n);
    }
  };
  // a table of one block is staged once for all the workgroup's tiles
  if (one_block) {
    stage_first();
    __syncthreads();
  }
  // workgroups go to the eight XCDs in turn (workgroup b to XCD b mod 8), each
  // XCD with its own L2: renumber them so the workgroups of one XCD take
  // neighbouring tiles, whose windows share input rows
  const int nx = gridDim.x >> 3;
  const int wg = (gridDim.x & 7) == 0 ? (int)(blockIdx.x & 7) * nx + (int)(blockIdx.x >> 3)
                                      : (int)blockIdx.x;
  for (int tile = wg; tile < ba.ntiles; tile += gridDim.x) {
    CS_STAMP_COUNT(31);
    CS_STAMP(16);
    const int item0 = tile * ba.P;
    const int item = item0 + ps;
    const bool live = item < ba.items;
    int bb = 0, ho = 0, wo = 0;
    if (live) {
      const uint32_t t1 = fdiv((uint32_t)item, ba.fd_wo);
      wo = item - (int)(t1 * ba.fd_wo.d);
      const uint32_t t2 = fdiv(t1, ba.fd_ho);
      ho = (int)(t1 - t2 * ba.fd_ho.d);
      bb = (int)t2;
    }
    // accumulators start at the bias of their channels (KP > 0: nacc == KP):
    // the bias loads are issued together, then the first taps' list loads,
    // and only then are the accumulators written, so the two latencies
    // overlap (the wait before the writes covers the bias loads, and every
    // store issued before them: the vector memory counter counts both)
    constexpr int NJ = KP > 0 ? KP : GB * 16;
    float bv[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      bv[j] = (bias && (KP > 0 || j < nacc)) ? bias[u * nacc + j] : 0.f;
    // the first taps' counts and first chunks, then the table while they fly
    // (q[0] is the tap processed next; channel mode uses q[0] only)
    TapPre<QD> q[BLK_DEPTH];
    tap_prefetch(q[0], lidx, lval, lcnt, geo, live, bb, ho, wo, 0, 0, ba.fd_kw);
    if constexpr (!CH) {
#pragma unroll
      for (int d = 1; d < BLK_DEPTH; ++d)
        tap_prefetch(q[d], lidx, lval, lcnt, geo, live, bb, ho, wo, d, 0, ba.fd_kw);
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (KP > 0 || j < nacc) acc[j * BLK_BD + tid] = bv[j];
    if (!one_block) {
      stage_first();
      __syncthreads();
    }

    int cursor = 0;                                      // place in the current tap's list
    unsigned long long blk_time = 0;                     // stamping build: the blocks' products
    for (int blk = 0; blk < ba.nblocks; ++blk) {
      const int r0n = (blk + 1) * ba.RB;
      const bool has_next = blk + 1 < ba.nblocks;
      const bool odd = ba.nbuf == 2 && (blk & 1);
      const uint2* tab = reinterpret_cast<const uint2*>(smem + (odd ? ba.off_t1 : ba.off_t0));
      // the next table block's loads (issued after the prefetched list data)
      if (has_next) st.load(aug, r0n, min(R, r0n + ba.RB), G);
      const unsigned long long blk_t0 = CS_CLOCK();
      if constexpr (!CH) {
        // whole taps t0 .. t1-1; the taps BLK_DEPTH ahead (of this block
        // or the next ones) are in flight while one is processed
        const int t0 = blk * ba.tpb, t1 = min(T_, t0 + ba.tpb);
        for (int t = t0; t < t1; ++t) {
          TapPre<QD> nxt;
          tap_prefetch(nxt, lidx, lval, lcnt, geo, live, bb, ho, wo, t + BLK_DEPTH, 0, ba.fd_kw);
          blk_tap<GB, false, QD>(q[0], lidx, lval, geo.cap, 0, C, (t - t0) * C, tab, ba.tstride,
                             u * GB, accb);
#pragma unroll
          for (int d = 0; d + 1 < BLK_DEPTH; ++d) q[d] = q[d + 1];
          q[BLK_DEPTH - 1] = nxt;
        }
      } else {
        // one tap, the channels [c_lo, c_hi): the lane goes on in the tap's
        // list where the previous block stopped
        const int t0 = blk / ba.cblocks;
        const int c_lo = (blk - t0 * ba.cblocks) * ba.RB;
        if (c_lo == 0) cursor = 0;
        cursor = blk_tap<GB, true, QD>(q[0], lidx, lval, geo.cap, cursor, c_lo + ba.RB, -c_lo, tab,
                                   ba.tstride, u * GB, accb);
        // the next block's list data, in flight across the barrier
        const int tn = (blk + 1) / ba.cblocks;
        tap_prefetch(q[0], lidx, lval, lcnt, geo, live, bb, ho, wo, has_next ? tn : T_,
                     tn == t0 ? cursor : 0, ba.fd_kw);
      }
      blk_time += CS_CLOCK() - blk_t0;
      if (has_next) {
        if (ba.nbuf == 1) __syncthreads();               // every lane is done with the block
        st.store(smem, odd || ba.nbuf == 1 ? ba.off_t0 : ba.off_t1, 0,
                 min(R, r0n + ba.RB) - r0n, ba.log2G, ba.tstride, ba.log2n);
      }
      if (!one_block) __syncthreads();
    }

    // ---- epilogue
    CS_STAMP(17);
    CS_STAMP_ADD(21, blk_time);
    if constexpr (KP > 0) {
      // the lanes' own columns: no barrier, the next tile starts right after
      if constexpr (QK > 0) {
        // a pixel's four lanes are a quad holding its four quarters: the
        // gather kernel's four-lane selection reads them in place and writes
        // the lists straight to their rows
        const FastDiv one{1u, 0u, 0u};
        const RowMap rm{0, 1, 0, 0, 0, 0, 0, (int64_t)item0, one};
        uint2* sel = reinterpret_cast<uint2*>(smem + ba.off_sel);
        uint16_t* gi = lo.idx ? lo.idx + (int64_t)item0 * lo.cap : nullptr;
        TO* gv = lo.idx ? static_cast<TO*>(lo.val) + (int64_t)item0 * lo.cap : nullptr;
        if (c_out == 64)                                  // 16 channels per lane, known
          kwta_quad_item<float, TO, QK, BLK_BD, 64>(acc + tid, 0, ps, live, rm, c_out, ba.k, 0,
                                                    sel, gi, gv, lo.cap, lo.cnt);
        else
          kwta_quad_item<float, TO, QK, BLK_BD>(acc + tid, 0, ps, live, rm, c_out, ba.k, 0, sel,
                                                gi, gv, lo.cap, lo.cnt);
        if (live && (ba.write_sums || !lo.idx)) {
          wave_lds_order();                              // sel of this quad, written by lane 0
          const uint2 sv = sel[ps];
          const int o0 = u * KP;
          float* yr = y + (int64_t)item * c_out + o0;
          TO* orow = out + (int64_t)item * c_out + o0;
#pragma unroll
          for (int j = 0; j < KP; j += 4) {
            float a4[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) a4[e] = acc[(j + e) * BLK_BD + tid];
            if (ba.write_sums)
              *reinterpret_cast<float4*>(yr + j) = make_float4(a4[0], a4[1], a4[2], a4[3]);
            if (!lo.idx) {
              float w4[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t key = order_key(a4[e]);
                const bool win = ba.k > 0 && (key > sv.x || (key == sv.x && o0 + j + e <= (int)sv.y));
                w4[e] = win ? a4[e] : 0.f;
              }
              *reinterpret_cast<float4*>(orow + j) = make_float4(w4[0], w4[1], w4[2], w4[3]);
            }
          }
        }
      } else {
        blk_kwta_own<TO, KP>(acc, ba.log2U, ba.log2Us, (int64_t)item, live, c_out, ba.k,
                             ba.write_sums, y, out, lo);
      }
    } else {
      blk_epilogue_tile<TO, GB>(smem, acc, item0, c_out, y, out, lo, ba);
      __syncthreads();                                   // before the accumulators are reused
    }
    CS_STAMP(18);
  }
}

}  // namespace cs
