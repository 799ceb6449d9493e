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
//    registers for the whole workgroup;
//  * the pooled sums + bias go to an LDS tile [items][64 + 1]; k-WTA and the
//    output run as in the fused sparse layer (one lane per item).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "kwta_kernels.h"
#include "mrs_fused.h"
#include "mrs_kernels.h"

namespace cs {

struct DenseArgs {
  int TPR;            // pooled rows per workgroup
  int tiles_img;      // workgroups per image
  int R;              // kh * kw * c_in (<= 32)
  int k;              // k-WTA winners per item; < 0: none (sums only)
  int shift;
  int kmode;          // 1/2/3: top-8/16/32 insertion
  int write_sums;
  int ostride;        // c_out + 1
  uint32_t off_out, off_sel, off_lidx, off_lval;   // LDS byte offsets (image rows at 0)
  FastDiv fd_wp;      // / pooled width
  FastDiv fd_timg;    // / tiles_img
  FastDiv fd_cout;    // / c_out
  FastDiv fd_ochunks; // / (list capacity / 4)
};

typedef int v4i_t __attribute__((ext_vector_type(4)));

template <int POOL, typename TO>
__global__ __launch_bounds__(256) void conv_dense_mfma(const int8_t* __restrict__ x,
                                                       const uint16_t* __restrict__ aug,
                                                       const int32_t* __restrict__ bias,
                                                       int32_t* __restrict__ y,
                                                       TO* __restrict__ out, ListOut lo,
                                                       ConvGeom geo, DenseArgs da) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int Hp = geo.Ho / POOL, Wp = geo.Wo / POOL;
  const int C = geo.C, W = geo.W;
  const uint32_t img = fdiv(blockIdx.x, da.fd_timg);
  const int pr0 = (int)(blockIdx.x - img * (uint32_t)da.tiles_img) * da.TPR;
  const int npr = min(da.TPR, Hp - pr0);
  const int nitems = npr * Wp;
  const int64_t item0 = ((int64_t)img * Hp + pr0) * Wp;

  // input rows the tile reads, clipped to the image, staged whole (W * C bytes each)
  const int iy0 = pr0 * POOL * geo.S - geo.P;
  const int ry0 = max(iy0, 0);
  const int ry1 = min(((pr0 + npr) * POOL - 1) * geo.S - geo.P + geo.KH, geo.H);
  const int rowb = W * C;
  const int nbytes = max(ry1 - ry0, 0) * rowb;
  int8_t* rows = reinterpret_cast<int8_t*>(smem);
  {
    const int8_t* src = x + ((int64_t)img * geo.H + ry0) * rowb;
    for (int e = tid; e < nbytes; e += 256) rows[e] = src[e];
  }

  // B operands: lane holds channel 16*nt + lane%16, slots 8*(lane/16) .. +7
  const int g = lane >> 4, col = lane & 15;
  int64_t bop[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    uint64_t b8 = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kk = 8 * g + j;
      const uint32_t v = kk < da.R ? (uint32_t)(aug[kk * 64 + 16 * nt + col] & 0xFFu) : 0u;
      b8 |= (uint64_t)v << (8 * j);
    }
    bop[nt] = (int64_t)b8;
  }
  int32_t bch[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) bch[nt] = bias ? bias[16 * nt + col] : 0;

  // this lane's 8 slots of a window: input offset relative to the window's
  // top-left corner, or -1 past r
  int dy[8], dx[8], dc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int kk = 8 * g + j;
    const int t = kk / C, c = kk - (kk / C) * C;
    dy[j] = kk < da.R ? t / geo.KW : -1;
    dx[j] = t - (t / geo.KW) * geo.KW;
    dc[j] = c;
  }
  __syncthreads();

  int32_t* otile = reinterpret_cast<int32_t*>(smem + da.off_out);
  const int ostride = da.ostride;
  constexpr int IPM = 16 / (POOL * POOL);                  // items per M tile
  const int mtiles = (nitems + IPM - 1) / IPM;
  for (int mt = wv; mt < mtiles; mt += 4) {
    // this lane's im2col row: item and sub-pixel
    const int r = lane & 15;
    const int item = mt * IPM + r / (POOL * POOL);
    const int q = r % (POOL * POOL);
    uint64_t a8 = 0;
    if (item < nitems) {
      const int pr = (int)fdiv((uint32_t)item, da.fd_wp);
      const int pc = item - pr * Wp;
      const int oy = (pr0 + pr) * POOL + q / POOL, ox = pc * POOL + q % POOL;
      const int by = oy * geo.S - geo.P, bx = ox * geo.S - geo.P;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int iy = by + dy[j], ix = bx + dx[j];
        uint32_t v = 0u;
        if (dy[j] >= 0 && iy >= ry0 && iy < ry1 && ix >= 0 && ix < W)
          v = (uint8_t)rows[(iy - ry0) * rowb + ix * C + dc[j]];
        a8 |= (uint64_t)v << (8 * j);
      }
    }
    const v4i_t zero = {0, 0, 0, 0};
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const v4i_t d = __builtin_amdgcn_mfma_i32_16x16x32_i8((int64_t)a8, bop[nt], zero, 0, 0, 0);
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

  // ---- output: the sums, and/or k-WTA as in the fused sparse layer
  const int c_out = 64;
  if (da.write_sums) {
    const int tot = nitems * c_out;
    for (int e = tid; e < tot; e += 256) {
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
    switch (da.kmode) {
      case 1:
        kwta_quad_items<int32_t, TO, 8>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel, tl_idx,
                                        tl_val, lo.cap, lo.cnt);
        break;
      case 2:
        kwta_quad_items<int32_t, TO, 16>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel,
                                         tl_idx, tl_val, lo.cap, lo.cnt);
        break;
      default:
        kwta_quad_items<int32_t, TO, 32>(otile, ostride, sm, rm, c_out, da.k, da.shift, sel,
                                         tl_idx, tl_val, lo.cap, lo.cnt);
        break;
    }
    __syncthreads();
    if (lo.idx) {
      using OV = typename ChunkVal<TO>::type;
      const int cq = lo.cap >> 2;
      for (int e = tid; e < nitems * cq; e += 256) {
        const int it = (int)fdiv((uint32_t)e, da.fd_ochunks);
        const int j = e - it * cq;
        const int64_t gofs = (item0 + it) * lo.cap + 4 * j;
        *reinterpret_cast<uint2*>(lo.idx + gofs) = reinterpret_cast<const uint2*>(tl_idx)[it * cq + j];
        *reinterpret_cast<OV*>(static_cast<TO*>(lo.val) + gofs) =
            reinterpret_cast<const OV*>(tl_val)[it * cq + j];
      }
    } else {
      const bool none = da.k == 0;
      for (int e = tid; e < nitems * c_out; e += 256) {
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

}  // namespace cs
