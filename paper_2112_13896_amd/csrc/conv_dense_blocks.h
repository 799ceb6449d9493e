// Sparse-dense convolution with block Complementary Sparsity (Section 3.1:
// complementary patterns made of blocks; Section 5: the stem treats the
// c_in <= 4 channel values of one input pixel as a block; Section 4: a first
// layer on dense input runs sparse-dense).  int8 activations and weights,
// int32 sums.
//
// A block is one tap's c_in channels, so a (tap, set) pair has one Kernel ID
// for its c_in products: they are summed first - one v_dot4 of the pixel's
// channels with the set's weights at that tap - and routed once, to
// accumulator g*n + kid.  Each output pixel visits its kh*kw taps; the work
// per pixel is kh*kw*G dot products and routed adds, G = c_out / n, against
// kh*kw*c_in*c_out multiply-adds for the dense layer.
//
//  * tile: P consecutive output pixels per workgroup, complete in the channel
//    dimension; lanes = (pixel, unit of GB sets), U = G / GB lanes a pixel;
//  * staging: the input rows under the tile's windows, zero-padded at the
//    sides and outside the image, one 32-bit word per pixel (its channels in
//    the low bytes), so a lane reads a tap's channels with one LDS load; the
//    table as [tap][set] {four weight bytes, accumulator byte offset};
//  * Route / Sum: the lane's accumulators are LDS columns acc[j][lane]
//    (bank = lane), j = (g mod GB)*n + kid, added with ds_add_u32 (no
//    read-back, no conflict);
//  * out: bias + sums, the lane's GB*n consecutive channels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "fastdiv.h"
#include "mrs_kernels.h"

namespace cs {

constexpr int DB_BD = 256;            // threads per workgroup
constexpr int DB_PRE = 4;             // staged input pixels per thread at most

struct DenseBlocksArgs {
  int GB;             // sets per lane (1 or 2)
  int U;              // lanes per pixel = G / GB
  int P;              // output pixels per tile (a segment of one output row) = DB_BD / U
  int nseg;           // segments per output row, ceil(Wo / P)
  int ntiles;         // B * Ho * nseg
  int SW;             // staged input columns per row: (P - 1) * S + KW
  uint32_t off_x, off_t;   // LDS byte offsets (accumulator columns at 0)
  FastDiv fd_nseg, fd_ho, fd_sw;
};

// KW: the kernel width (a tap row's loads are issued together), 0: any
// (one tap after another); GB: sets per lane; PK: c_in <= 3, so a table entry
// is one word, the accumulator index j in the fourth byte (the staged input's
// fourth byte is 0, so the dot product ignores it).  Persistent workgroups:
// the table is staged once, then the workgroup loops over tiles.
template <int KW, int GB, bool PK>
__global__ __launch_bounds__(DB_BD) void conv_dense_blocks(const int8_t* __restrict__ x,
                                                           const uint16_t* __restrict__ aug,
                                                           const uint8_t* __restrict__ kidb,
                                                           const int32_t* __restrict__ bias,
                                                           int32_t* __restrict__ y, ConvGeom geo,
                                                           DenseBlocksArgs da) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int C = geo.C, G = geo.G, n = geo.n, T = geo.KH * geo.KW;
  const int U = da.U;
  const int ps = tid / U, u = tid - ps * U;              // pixel slot, unit
  const int nacc = GB * n;                               // the lane's channels
  unsigned char* accb = smem + tid * 4;
  uint32_t* xs = reinterpret_cast<uint32_t*>(smem + da.off_x);
  using TE = typename std::conditional<PK, uint32_t, uint2>::type;
  TE* tab = reinterpret_cast<TE*>(smem + da.off_t);

  // the table: (tap t, set g) -> the block's weights (channel c in byte c)
  // and the byte offset of its accumulator column ((g mod GB)*n + kid)
  for (int e = tid; e < T * G; e += DB_BD) {
    const int t = e / G, g = e - t * G;
    uint32_t w4 = 0u;
    for (int c = 0; c < C; ++c)
      w4 |= (uint32_t)(aug[(size_t)(t * C + c) * G + g] & 0xFFu) << (8 * c);
    const int kid = kidb[e] < n ? kidb[e] : n - 1;        // < n for cs_pack_blocks output
    const uint32_t j = (uint32_t)((g % GB) * n + kid);
    if constexpr (PK)
      tab[e] = w4 | j << 24;                              // j < GB * n <= 64
    else
      tab[e] = make_uint2(w4, j * (uint32_t)(DB_BD * 4));
  }

  const int nst = geo.KH * da.SW;            // staged pixels per tile, <= DB_PRE * DB_BD (host)
  // a tile's input: rows oy*S - P + ky under its windows, columns
  // ox0*S - P .. + SW - 1, zero outside the image; each thread's pixels are
  // loaded into registers one tile ahead, so the loads overlap the previous
  // tile's products
  auto load_tile = [&](int tile, uint32_t (&v)[DB_PRE]) {
    const uint32_t r = fdiv((uint32_t)tile, da.fd_nseg);
    const int seg = tile - (int)r * da.nseg;
    const uint32_t bb = fdiv(r, da.fd_ho);
    const int oy = (int)r - (int)bb * geo.Ho;
    const int iy0 = oy * geo.S - geo.P, ix0 = seg * da.P * geo.S - geo.P;
    const int8_t* ximg = x + (size_t)bb * geo.H * geo.W * C;
#pragma unroll
    for (int q = 0; q < DB_PRE; ++q) {
      const int e = q * DB_BD + tid;
      const int ky = (int)fdiv((uint32_t)e, da.fd_sw), col = e - ky * da.SW;
      const int iy = iy0 + ky, ix = ix0 + col;
      uint32_t w = 0u;
      if (tile < da.ntiles && e < nst && iy >= 0 && iy < geo.H && ix >= 0 && ix < geo.W) {
        const int8_t* src = ximg + ((size_t)iy * geo.W + ix) * C;
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (c < C) w |= (uint32_t)(uint8_t)src[c] << (8 * c);
      }
      v[q] = w;
    }
  };
  uint32_t pre[DB_PRE];
  load_tile(blockIdx.x, pre);
  for (int tile = blockIdx.x; tile < da.ntiles; tile += gridDim.x) {
    const uint32_t r = fdiv((uint32_t)tile, da.fd_nseg);  // output row b*Ho + oy
    const int seg = tile - (int)r * da.nseg;
    const int ox0 = seg * da.P;
    __syncthreads();                                       // the previous tile is done with xs
#pragma unroll
    for (int q = 0; q < DB_PRE; ++q)
      if (q * DB_BD + tid < nst) xs[q * DB_BD + tid] = pre[q];
    // accumulators start at zero (the bias is added at the end)
    for (int j = 0; j < nacc; ++j) *reinterpret_cast<int32_t*>(accb + j * DB_BD * 4) = 0;
    __syncthreads();
    load_tile(tile + gridDim.x, pre);                     // the next tile's input, in flight

    const int ox = ox0 + ps;
    if (ps < da.P && ox < geo.Wo) {
      const uint32_t* xrow = xs + ps * geo.S;
      const TE* trow = tab + u * GB;
      auto route = [&](uint32_t xv, const TE& e) {
        uint32_t w, off;
        if constexpr (PK) {
          w = e;
          off = (e >> 24) * (uint32_t)(DB_BD * 4);
        } else {
          w = e.x;
          off = e.y;
        }
        const int p = __builtin_amdgcn_sdot4((int)xv, (int)w, 0, false);
        __hip_atomic_fetch_add(reinterpret_cast<int32_t*>(accb + off), p, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
      };
      for (int ky = 0; ky < geo.KH; ++ky) {
        const uint32_t* xr = xrow + ky * da.SW;
        const TE* tr = trow + ky * geo.KW * G;
        if constexpr (KW > 0) {
          // the row's activations and table entries first, then the products
          uint32_t xv[KW];
          TE e[KW][GB];
#pragma unroll
          for (int kx = 0; kx < KW; ++kx) {
            xv[kx] = xr[kx];
#pragma unroll
            for (int s2 = 0; s2 < GB; ++s2) e[kx][s2] = tr[kx * G + s2];
          }
#pragma unroll
          for (int kx = 0; kx < KW; ++kx)
#pragma unroll
            for (int s2 = 0; s2 < GB; ++s2) route(xv[kx], e[kx][s2]);
        } else {
          for (int kx = 0; kx < geo.KW; ++kx)
#pragma unroll
            for (int s2 = 0; s2 < GB; ++s2) route(xr[kx], tr[kx * G + s2]);
        }
      }
      // out: channels u*GB*n + j, j < GB*n, with the bias
      int32_t* yr = y + ((size_t)r * geo.Wo + ox) * geo.c_out + u * nacc;
      for (int j = 0; j < nacc; ++j) {
        const int32_t a = *reinterpret_cast<const int32_t*>(accb + j * DB_BD * 4);
        yr[j] = a + (bias ? bias[u * nacc + j] : 0);
      }
    }
  }
}

}  // namespace cs
