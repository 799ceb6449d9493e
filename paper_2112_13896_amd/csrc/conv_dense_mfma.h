// Sparse-dense first layer (Section 3.1: dense weights, n == 1, on a dense
// input; Section 4 runs the first layer this way because its input is dense)
// as one kernel on the matrix cores: convolution, bias, 2x2 max-pool, k-WTA,
// requantisation and the next layer's (index, value) lists (Figure 10).
//
// The convolution is a dense contraction (im2col rows x dense weights), so it
// runs as int8 MFMA 16x16x32 tiles with K = kh*kw*c_in <= 32 (zero padded):
//  * the workgroup owns TPR pooled rows of one image and stages the input rows
//    they read in LDS;
//  * an M tile is 16 im2col rows; with pooling they are 4 pooled pixels x 4
//    sub-pixels (row 4p + q), so the 4 accumulator rows a lane receives
//    (rows 4*(lane/16) .. +3, column lane%16) are the 2x2 window of one pooled
//    pixel and the max-pool is a max over the lane's own 4 values;
//  * the B operand (the 64 channels' weights, 4 N tiles of 16) stays in
//    registers for the whole workgroup; it is staged transposed ([channel][32
//    slots] bytes, zero past R), so a lane's 8 slots are one 8-byte read, and
//    the zero slots make the A operand's bytes past R irrelevant;
//  * the byte offsets of the 32 slots in the staged rows are a table built
//    once per workgroup;
//  * the pooled sums + bias go to an LDS tile [items][64 + 1]; k-WTA and the
//    output run as in the fused sparse layer (four lanes per item).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_fused.h"
#include "mrs_kernels.h"

namespace cs {

constexpr int DENSE_BD = 512;     // threads per workgroup
constexpr int DENSE_STAGE = 8;   // input bytes per thread in flight while staging

struct DenseArgs {
  int TPR;            // pooled rows per workgroup
  int tiles_img;      // workgroups per image
  int R;              // kh * kw * c_in (<= 32)
  int k;              // k-WTA winners per item; < 0: none (sums only)
  int shift;
  int kmode;          // 1/2/3: top-8/16/32 insertion
  int write_sums;
  int vec_rows;       // 1: no padding, rows of W*C bytes a multiple of 16, input 16-byte aligned
  int ostride;        // c_out + 1
  uint32_t off_w, off_out, off_sel, off_lidx, off_lval;   // LDS byte offsets (image rows at 0)
  FastDiv fd_wp;      // / pooled width
  FastDiv fd_timg;    // / tiles_img
  FastDiv fd_cout;    // / c_out
  FastDiv fd_ochunks; // / (list capacity / 4)
  FastDiv fd_rowb;    // / staged row bytes ((W + 2P) * C)
  FastDiv fd_c;       // / C
  FastDiv fd_kw;      // / KW
};

typedef int v4i_t __attribute__((ext_vector_type(4)));

// The workgroup body for workgroup index blk, BD (>= 512) threads.  KM: the
// k-WTA selection (da.kmode) fixed at compile time, or 0: chosen at run time.
template <int POOL, typename TO, int BD, int KM = 0>
__device__ __forceinline__ void dense_body(const int8_t* __restrict__ x,
                                           const uint16_t* __restrict__ aug,
                                           const int32_t* __restrict__ bias,
                                           int32_t* __restrict__ y, TO* __restrict__ out,
                                           const ListOut& lo, const ConvGeom& geo,
                                           const DenseArgs& da, uint32_t blk) {
  static_assert(BD >= 512 && BD % 64 == 0, "the weight staging takes 512 threads");
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int Hp = geo.Ho / POOL, Wp = geo.Wo / POOL;
  const int C = geo.C, W = geo.W;
  const uint32_t img = fdiv(blk, da.fd_timg);
  const int pr0 = (int)(blk - img * (uint32_t)da.tiles_img) * da.TPR;
  const int npr = min(da.TPR, Hp - pr0);
  const int nitems = npr * Wp;
  const int64_t item0 = ((int64_t)img * Hp + pr0) * Wp;

  // the input rows the tile reads, staged zero-padded (columns -P .. W+P-1,
  // rows outside the image as zeros), so that the im2col gather below needs
  // no bounds checks
  const int Wpad = W + 2 * geo.P;
  const int rowb = Wpad * C;
  const int iy0 = pr0 * POOL * geo.S - geo.P;
  const int rows_in = (npr * POOL - 1) * geo.S + geo.KH;
  const int nbytes = rows_in * rowb;                        // <= the LDS allocation (host)
  int8_t* rows = reinterpret_cast<int8_t*>(smem);

  // the weights ([R][64] 16-bit entries, value in the low byte) are staged
  // transposed, wt[channel][slot] bytes with slots R .. 31 zero: thread t
  // gathers slots 4*(t%8) .. +3 of channel t/8, loads issued together with
  // the input's
  const int g = lane >> 4, col = lane & 15;
  unsigned char* wt = smem + da.off_w;                     // [64][32] bytes
  int* offt = reinterpret_cast<int*>(smem + da.off_w + 64 * 32);   // [32] slot offsets
  int32_t bch[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) bch[nt] = bias ? bias[16 * nt + col] : 0;
  {
    // threads 0 .. 511: one per (channel, 4 slots)
    const int wch = (tid & 511) >> 3, wk0 = (tid & 7) * 4;
    uint32_t wb4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int kk = wk0 + i;
      wb4[i] = aug[(kk < da.R ? kk : 0) * 64 + wch];
    }
    const int8_t* ximg = x + (int64_t)img * geo.H * W * C;
    if (da.vec_rows && iy0 >= 0 && iy0 + rows_in <= geo.H) {
      // unpadded rows inside the image: one contiguous run, 16 bytes per load
      const uint4* src = reinterpret_cast<const uint4*>(ximg + (int64_t)iy0 * W * C);
      uint4* dst = reinterpret_cast<uint4*>(rows);
      const int n16 = nbytes / 16;                         // >= 1
      for (int b0 = 0; b0 < n16; b0 += BD * 2) {
        uint4 v[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = b0 + u * BD + tid;
          v[u] = src[e < n16 ? e : n16 - 1];               // in range: no branch
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = b0 + u * BD + tid;
          if (e < n16) dst[e] = v[u];
        }
      }
    } else
    for (int b0 = 0; b0 < nbytes; b0 += BD * DENSE_STAGE) {
      int8_t v[DENSE_STAGE];
#pragma unroll
      for (int u = 0; u < DENSE_STAGE; ++u) {
        const int e = b0 + u * BD + tid;
        const int r = (int)fdiv((uint32_t)e, da.fd_rowb);
        const int cb = e - r * rowb;
        const int px = (int)fdiv((uint32_t)cb, da.fd_c);
        const int iy = iy0 + r, ix = px - geo.P;
        const bool ok = e < nbytes && iy >= 0 && iy < geo.H && ix >= 0 && ix < W;
        v[u] = ximg[ok ? ((int64_t)iy * W + ix) * C + (cb - px * C) : 0];
        v[u] = ok ? v[u] : int8_t(0);
      }
#pragma unroll
      for (int u = 0; u < DENSE_STAGE; ++u) {
        const int e = b0 + u * BD + tid;
        if (e < nbytes) rows[e] = v[u];
      }
    }
    uint32_t w4 = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) w4 |= (wk0 + i < da.R ? wb4[i] & 0xFFu : 0u) << (8 * i);
    if (tid < 512) reinterpret_cast<uint32_t*>(wt)[tid] = w4;   // wt + wch * 32 + wk0
    if (tid < 32) {
      // slot kk = (ky * KW + kx) * C + c: byte offset from a window's corner
      const int kk = tid;
      const int t = (int)fdiv((uint32_t)kk, da.fd_c), c = kk - t * C;
      const int ky = (int)fdiv((uint32_t)t, da.fd_kw), kx = t - ky * geo.KW;
      offt[kk] = kk < da.R ? ky * rowb + kx * C + c : 0;
    }
  }
  __syncthreads();
  CS_STAMP(1);
  // B operands: lane holds channel 16*nt + lane%16, slots 8*(lane/16) .. +7
  int64_t bop[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
    bop[nt] = *reinterpret_cast<const int64_t*>(wt + (16 * nt + col) * 32 + 8 * g);
  // this lane's 8 slots of a window: byte offsets from the window's top-left
  // corner in the staged rows (slots past R read offset 0; their B is zero)
  int offs[8];
  {
    const int4 o0 = reinterpret_cast<const int4*>(offt)[2 * g];
    const int4 o1 = reinterpret_cast<const int4*>(offt)[2 * g + 1];
    offs[0] = o0.x; offs[1] = o0.y; offs[2] = o0.z; offs[3] = o0.w;
    offs[4] = o1.x; offs[5] = o1.y; offs[6] = o1.z; offs[7] = o1.w;
  }

  int32_t* otile = reinterpret_cast<int32_t*>(smem + da.off_out);
  const int ostride = da.ostride;
  constexpr int IPM = 16 / (POOL * POOL);                  // items per M tile
  const int mtiles = (nitems + IPM - 1) / IPM;
  for (int mt = wv; mt < mtiles; mt += BD / 64) {
    // this lane's im2col row: item and sub-pixel (past the tile's last item
    // the last item is gathered again; its results are not stored)
    const int r = lane & 15;
    int item = mt * IPM + r / (POOL * POOL);
    item = item < nitems ? item : nitems - 1;
    const int q = r % (POOL * POOL);
    const int pr = (int)fdiv((uint32_t)item, da.fd_wp);
    const int pc = item - pr * Wp;
    const int oyl = pr * POOL + q / POOL, ox = pc * POOL + q % POOL;   // conv row in the tile
    const unsigned char* wb = reinterpret_cast<const unsigned char*>(rows) +
                              oyl * geo.S * rowb + ox * geo.S * C;
    uint32_t lo4 = 0u, hi4 = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lo4 |= (uint32_t)wb[offs[j]] << (8 * j);
      hi4 |= (uint32_t)wb[offs[4 + j]] << (8 * j);
    }
    const uint64_t a8 = (uint64_t)lo4 | ((uint64_t)hi4 << 32);
    const v4i_t zero = {0, 0, 0, 0};
    v4i_t dd[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)   // independent products, issued back to back
      dd[nt] = __builtin_amdgcn_mfma_i32_16x16x32_i8((int64_t)a8, bop[nt], zero, 0, 0, 0);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const v4i_t d = dd[nt];
      // lane holds rows 4g .. 4g+3 of column col
      if constexpr (POOL == 2) {
        const int it = mt * IPM + g;                      // the 4 rows are its 2x2 window
        int32_t m = d[0];
        m = d[1] > m ? d[1] : m;
        m = d[2] > m ? d[2] : m;
        m = d[3] > m ? d[3] : m;
        if (it < nitems) otile[it * ostride + 16 * nt + col] = m + bch[nt];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int it = mt * IPM + 4 * g + i;
          if (it < nitems) otile[it * ostride + 16 * nt + col] = d[i] + bch[nt];
        }
      }
    }
  }
  __syncthreads();
  CS_STAMP(2);

  // ---- output: the sums, and/or k-WTA as in the fused sparse layer
  const int c_out = 64;
  if (da.write_sums) {
    const int tot = nitems * c_out;
    for (int e = tid; e < tot; e += BD) {
      const int it = (int)fdiv((uint32_t)e, da.fd_cout);
      y[item0 * c_out + e] = otile[it * ostride + (e - it * c_out)];
    }
  }
  if (da.k >= 0) {
    const SlotMap sm{0, 1, 1, nitems, FastDiv{1, 0, 0}};
    const RowMap rm{0, 1, 0, 0, 0, 0, 0, item0, FastDiv{1, 0, 0}};
    uint2* sel = reinterpret_cast<uint2*>(smem + da.off_sel);
    uint16_t* tl_idx = lo.idx ? reinterpret_cast<uint16_t*>(smem + da.off_lidx) : nullptr;
    TO* tl_val = reinterpret_cast<TO*>(smem + da.off_lval);
    switch (KM > 0 ? KM : da.kmode) {
      case 1:
        kwta_quad_items<int32_t, TO, 8, BD, 64>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel, tl_idx,
                                        tl_val, lo.cap, lo.cnt);
        break;
      case 2:
        kwta_quad_items<int32_t, TO, 16, BD, 64>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel,
                                         tl_idx, tl_val, lo.cap, lo.cnt);
        break;
      default:
        kwta_quad_items<int32_t, TO, 32, BD, 64>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel,
                                         tl_idx, tl_val, lo.cap, lo.cnt);
        break;
    }
    __syncthreads();
    CS_STAMP(3);
    if (lo.idx) {
      using OV = typename ChunkVal<TO>::type;
      const int cq = lo.cap >> 2;
      for (int e = tid; e < nitems * cq; e += BD) {
        const int it = (int)fdiv((uint32_t)e, da.fd_ochunks);
        const int j = e - it * cq;
        const int64_t gofs = (item0 + it) * lo.cap + 4 * j;
        *reinterpret_cast<uint2*>(lo.idx + gofs) = reinterpret_cast<const uint2*>(tl_idx)[it * cq + j];
        *reinterpret_cast<OV*>(static_cast<TO*>(lo.val) + gofs) =
            reinterpret_cast<const OV*>(tl_val)[it * cq + j];
      }
    } else {
      const bool none = da.k == 0;
      for (int e = tid; e < nitems * c_out; e += BD) {
        const int it = (int)fdiv((uint32_t)e, da.fd_cout);
        const int ch = e - it * c_out;
        const int32_t a = otile[it * ostride + ch];
        const uint2 sv = sel[it];
        const uint32_t key = order_key(a);
        const bool win = !none && (key > sv.x || (key == sv.x && ch <= (int)sv.y));
        out[(item0 + it) * c_out + ch] = win ? kwta_out<int32_t, TO>(a, da.shift) : TO(0);
      }
    }
  }
}

template <int POOL, typename TO>
__global__ __launch_bounds__(DENSE_BD) void conv_dense_mfma(const int8_t* __restrict__ x,
                                                       const uint16_t* __restrict__ aug,
                                                       const int32_t* __restrict__ bias,
                                                       int32_t* __restrict__ y,
                                                       TO* __restrict__ out, ListOut lo,
                                                       ConvGeom geo, DenseArgs da) {
  dense_body<POOL, TO, DENSE_BD>(x, aug, bias, y, out, lo, geo, da, blockIdx.x);
}

}  // namespace cs
