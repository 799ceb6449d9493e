// Reordering the activations instead of routing the products (Section 3.2:
// for some hardware it can pay to reorder the incoming activations rather
// than route the element-wise products).  The packed kernel is read in
// Kernel-ID order: for every output o = g*n + kid, the slots i with
// kid[i][g] == kid and their values (the support of kernel o, gathered
// offline by cs_reorder_table).  Each output is then the dot product of its
// support with the activations at those slots: no product is routed, every
// sum stays in a register.  The activations are read densely (zeros
// included), so the kernel suits a layer whose input is a dense tensor (the
// first layer of a chain) at a small N, where the support is short.
//
// gfx950 mapping, fp32, stride 1, no pooling, C <= 64, c_out = 64:
//  * one wavefront per tile of 8 x 8 output pixels, one pixel per lane; the
//    tile's input halo ((8 + kh - 1) x (8 + kw - 1) pixels x C channels) is
//    staged in LDS with a pixel stride of C + 1 words, so the 64 lanes' reads
//    of one slot fall in distinct banks;
//  * the table entry (LDS byte offset of the slot in the halo, weight) is
//    wavefront-uniform: batches of 8 come by vector loads issued a batch
//    ahead, and each multiply-add is one LDS read and one FMA;
//  * the 64 outputs of the lane's pixel stay in registers for the k-WTA:
//    top-KMAX keys by bitonic sort/merge networks, ties to the lower channel,
//    the winners' list staged in LDS per lane and written with 16-byte stores.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kwta_kernels.h"
#include "mrs_fused.h"
#include "mrs_kernels.h"
#include "wave_ops.h"

namespace cs {

constexpr int RO_T = 8;         // output tile side (8 x 8 pixels: one wavefront)
constexpr int RO_COUT = 64;     // outputs per pixel

struct ReorderArgs {
  int smax;        // table entries per output (a multiple of 8)
  int tiles_w;     // tiles per output row
  int tiles_img;   // tiles per image
  int k;           // k-WTA winners (< 0: sums only)
  int write_sums;
  int vec4;        // 1: C % 4 == 0 and the input 16-byte aligned (float4 staging)
  FastDiv fd_cq;   // / staged pieces per pixel (C / 4 with vec4, else C)
  FastDiv fd_hw;   // / halo width (8 + KW - 1)
};

template <int KMAX>
__global__ __launch_bounds__(64) void conv_reorder_f32(const float* __restrict__ x,
                                                       const int2* __restrict__ tab,
                                                       const float* __restrict__ bias,
                                                       float* __restrict__ y,
                                                       float* __restrict__ out, ListOut lo,
                                                       ConvGeom geo, ReorderArgs ra) {
  extern __shared__ __align__(16) float halo[];
  const int lane = threadIdx.x;
  const int C = geo.C, H = geo.H, W = geo.W;
  const int HW = RO_T + geo.KW - 1, HH = RO_T + geo.KH - 1, CP = C + 1;
  const int img = (int)(blockIdx.x / (unsigned)ra.tiles_img);
  const int tr = (int)(blockIdx.x - (unsigned)img * ra.tiles_img);
  const int ty = tr / ra.tiles_w, tx = tr - (tr / ra.tiles_w) * ra.tiles_w;
  const int oy0 = ty * RO_T, ox0 = tx * RO_T;
  const int iy0 = oy0 - geo.P, ix0 = ox0 - geo.P;
  const float* ximg = x + (int64_t)img * H * W * C;

  // ---- the halo into LDS (zeros outside the image)
  if (ra.vec4) {
    const int c4 = C >> 2, n4 = HH * HW * c4;
    for (int e = lane; e < n4; e += 64) {
      const int p = (int)fdiv((uint32_t)e, ra.fd_cq), q = e - p * c4;
      const int hy = (int)fdiv((uint32_t)p, ra.fd_hw), hx = p - hy * HW;
      const int iy = iy0 + hy, ix = ix0 + hx;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (iy >= 0 && iy < H && ix >= 0 && ix < W)
        v = *reinterpret_cast<const float4*>(ximg + ((int64_t)iy * W + ix) * C + 4 * q);
      float* d = halo + p * CP + 4 * q;
      d[0] = v.x;
      d[1] = v.y;
      d[2] = v.z;
      d[3] = v.w;
    }
  } else {
    const int n1 = HH * HW * C;
    for (int e = lane; e < n1; e += 64) {
      const int p = (int)fdiv((uint32_t)e, ra.fd_cq), c = e - p * C;
      const int hy = (int)fdiv((uint32_t)p, ra.fd_hw), hx = p - hy * HW;
      const int iy = iy0 + hy, ix = ix0 + hx;
      float v = 0.f;
      if (iy >= 0 && iy < H && ix >= 0 && ix < W) v = ximg[((int64_t)iy * W + ix) * C + c];
      halo[p * CP + c] = v;
    }
  }
  __syncthreads();

  // ---- the dot products: output o of this lane's pixel over its support.
  // The table is one contiguous stream of c_out * smax entries (smax a
  // multiple of 8); batches of 8 entries arrive by vector loads (every lane
  // the same address), the next batch issued before the current one is used.
  // Vector loads complete in order and have a counter of their own, so the
  // LDS reads of a batch do not wait for the prefetch.
  const int py = lane >> 3, px = lane & 7;
  const unsigned char* hb = reinterpret_cast<const unsigned char*>(halo) + 4 * ((py * HW + px) * CP);
  typedef int i4_t __attribute__((ext_vector_type(4)));
  const i4_t* T4 = reinterpret_cast<const i4_t*>(tab);              // two entries per piece
  const int nb4 = ra.smax >> 1;                                     // pieces per output
  const int last4 = RO_COUT * nb4 - 4;                              // the stream's last batch
  const int vz = opaque_int(0);                                     // vector (not scalar) loads
  i4_t cur[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) cur[u] = T4[vz + u];
  float acc[RO_COUT];
#pragma unroll
  for (int o = 0; o < RO_COUT; ++o) {
    float a0 = bias != nullptr ? bias[o] : 0.f, a1 = 0.f;
    for (int s4 = 0; s4 < nb4; s4 += 4) {                           // uniform
      const int f = o * nb4 + s4 + 4;
      const int fn = f < last4 ? f : last4;
      i4_t nxt[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) nxt[u] = T4[vz + fn + u];
      float v[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[2 * u] = *reinterpret_cast<const float*>(hb + cur[u].x);
        v[2 * u + 1] = *reinterpret_cast<const float*>(hb + cur[u].z);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a0 = fmaf(v[2 * u], __int_as_float(cur[u].y), a0);
        a1 = fmaf(v[2 * u + 1], __int_as_float(cur[u].w), a1);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) cur[u] = nxt[u];
    }
    acc[o] = a0 + a1;
  }

  const int oy = oy0 + py, ox = ox0 + px;
  const bool valid = oy < geo.Ho && ox < geo.Wo;
  const int64_t row = ((int64_t)img * geo.Ho + (valid ? oy : 0)) * geo.Wo + (valid ? ox : 0);
  typedef float f4_t __attribute__((ext_vector_type(4)));
  if (ra.write_sums && valid) {
    f4_t* yr = reinterpret_cast<f4_t*>(y + row * RO_COUT);
#pragma unroll
    for (int q = 0; q < RO_COUT / 4; ++q) {
      f4_t v = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
      yr[q] = v;
    }
  }
  const int k = ra.k;
  if (k < 0) return;

  // ---- k-WTA over the lane's 64 outputs: the k-th largest key T, ties to
  // the lower channel
  uint32_t thr = 0u;
  int need = 0;
  if (k >= RO_COUT) {
    need = RO_COUT;                                                 // every key >= 0 wins
  } else if (k > 0) {
    uint32_t top[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) top[i] = order_key(acc[i]);
    bitonic_sort_desc<KMAX>(top);
#pragma unroll
    for (int b = KMAX; b < RO_COUT; b += KMAX) {
      uint32_t blk[KMAX];
#pragma unroll
      for (int i = 0; i < KMAX; ++i) blk[i] = order_key(acc[b + i]);
      bitonic_sort_desc<KMAX>(blk);
      top_merge_desc<KMAX>(top, blk);
    }
#pragma unroll
    for (int s = 0; s < KMAX; ++s) thr = (s == k - 1) ? top[s] : thr;
    int gt = 0;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) gt += (s < k && top[s] > thr) ? 1 : 0;
    need = k - gt;
  }
  if (lo.idx) {
    // the non-zero winners in channel order, staged per lane in LDS (the
    // halo is no longer read) and written as whole 16-byte pieces
    __syncthreads();
    const int cap = lo.cap;
    uint16_t* sx = reinterpret_cast<uint16_t*>(halo) + lane * cap;
    float* sv = halo + 32 * cap + lane * cap;                      // after 64 * cap u16
    int pos = 0, tr_ = 0;
#pragma unroll
    for (int o = 0; o < RO_COUT; ++o) {
      const uint32_t key = order_key(acc[o]);
      const bool tie = k > 0 && key == thr;
      const bool win = k > 0 && (key > thr || (tie && tr_ < need));
      tr_ += tie ? 1 : 0;
      if (win && acc[o] != 0.f) {
        sx[pos] = (uint16_t)o;
        sv[pos] = acc[o];
        ++pos;
      }
    }
    if (valid) {
      uint16_t* gx = lo.idx + row * cap;
      float* gv = static_cast<float*>(lo.val) + row * cap;
      for (int j = 0; j < pos; j += 4) {
        *reinterpret_cast<uint2*>(gx + j) = *reinterpret_cast<const uint2*>(sx + j);
      }
      for (int j = 0; j < pos; j += 4) {
        *reinterpret_cast<uint4*>(gv + j) = *reinterpret_cast<const uint4*>(sv + j);
      }
      lo.cnt[row] = pos;
    }
  } else if (valid) {
    f4_t* orow = reinterpret_cast<f4_t*>(out + row * RO_COUT);
    int tr_ = 0;
#pragma unroll
    for (int q = 0; q < RO_COUT / 4; ++q) {
      f4_t v;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int o = 4 * q + u;
        const uint32_t key = order_key(acc[o]);
        const bool tie = k > 0 && key == thr;
        const bool win = k > 0 && (key > thr || (tie && tr_ < need));
        tr_ += tie ? 1 : 0;
        v[u] = win ? acc[o] : 0.f;
      }
      orow[q] = v;
    }
  }
}

}  // namespace cs
