// Complementary Sparsity overlaid in the channel dimension (Section 3.1: the
// sets can be overlaid in the filter or in the channel dimension), int8
// dense input, int32 sums.  In every filter the n kh x kw slices of a group of
// n consecutive input channels have disjoint supports and are overlaid into
// one slice whose slots keep a weight and a channel ID; the slot (q, y, x)
// multiplies the input at tap (y, x), channel q*n + ID, and every product goes
// to the filter's own output, so nothing is routed: each output is a dot
// product of its packed slots with the input gathered at them.
//
//  * tile: 64 consecutive output pixels of one output row, one per lane;
//    the 256 lanes are four wavefronts, wavefront w computing filters
//    w*FW .. w*FW + FW - 1 of every pixel of the tile (FW = c_out / 4);
//  * staging: the tile's input rows under its windows as bytes
//    [KH][SW][CP] (SW = 63 * stride + KW pixels, a pixel's channels padded
//    to CP bytes, an odd number of words, so the 64 lanes' gathers of one
//    slot fall in different banks), zero outside the image;
//  * table: per filter its packed slots, in groups of four: the byte offsets
//    of the slots' inputs in the staged tile, then the four weights as one
//    word; read by the wavefront as uniform (scalar) values, all its lanes
//    using the same filter, the next group's loads issued before the
//    current group's products;
//  * per four slots: four LDS byte gathers packed into one word and one
//    4-way int8 dot product with the weight word; the FW sums of a lane are
//    written as consecutive words.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastdiv.h"
#include "mrs_kernels.h"

namespace cs {

constexpr int CH_BD = 256;          // threads per workgroup (four wavefronts)
constexpr int CH_P = 64;            // output pixels per tile (one per lane)

struct ChannelArgs {
  int S4;             // groups of four packed slots per filter: ceil((c_in / n) * KH * KW / 4)
  int SW;             // staged pixels per input row: 63 * stride + KW
  int CP;             // staged bytes per pixel (channels padded)
  int nseg;           // tiles per output row: ceil(Wo / 64)
  int ntiles;         // B * Ho * nseg
  FastDiv fd_nseg, fd_ho;
};

template <int FW>
__global__ __launch_bounds__(CH_BD) void conv_channels_i8(const int8_t* __restrict__ x,
                                                          const int32_t* __restrict__ table,
                                                          const int32_t* __restrict__ bias,
                                                          int32_t* __restrict__ y, ConvGeom geo,
                                                          ChannelArgs ca) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: the table loads are scalar
  const int C = geo.C;
  const int cw = C >> 2;                                  // words per pixel (C % 4 == 0, host)
  const int rw = ca.SW * cw;                              // words per staged row
  const int nw = geo.KH * rw;
  const int TS = 5 * ca.S4;                               // table words per filter
  const int32_t* tw = table + (size_t)wv * FW * TS;       // this wavefront's filters
  for (int tile = blockIdx.x; tile < ca.ntiles; tile += gridDim.x) {
    const uint32_t r = fdiv((uint32_t)tile, ca.fd_nseg);  // output row b*Ho + oy
    const int seg = tile - (int)r * ca.nseg;
    const uint32_t bb = fdiv(r, ca.fd_ho);
    const int oy = (int)r - (int)bb * geo.Ho;
    const int ox0 = seg * CH_P;
    const int iy0 = oy * geo.S - geo.P, ix0 = ox0 * geo.S - geo.P;
    const uint32_t* ximg = reinterpret_cast<const uint32_t*>(x + (size_t)bb * geo.H * geo.W * C);
    __syncthreads();                                       // the previous tile is done with it
    for (int e = tid; e < nw; e += CH_BD) {
      const int ky = e / rw, rem = e - ky * rw;
      const int px = rem / cw, cwi = rem - px * cw;
      const int iy = iy0 + ky, ix = ix0 + px;
      uint32_t v = 0u;
      if (iy >= 0 && iy < geo.H && ix >= 0 && ix < geo.W)
        v = ximg[((size_t)iy * geo.W + ix) * cw + cwi];
      *reinterpret_cast<uint32_t*>(smem + (ky * ca.SW + px) * ca.CP + cwi * 4) = v;
    }
    __syncthreads();
    const int ox = ox0 + lane;
    const uint8_t* base = smem + lane * geo.S * ca.CP;
    auto gather4 = [&](const int32_t (&o)[4]) -> int {
      const uint32_t b0 = base[o[0]], b1 = base[o[1]], b2 = base[o[2]], b3 = base[o[3]];
      return (int)(b0 | b1 << 8 | b2 << 16 | b3 << 24);
    };
    // four filters at a time: four independent sums, sixteen gathers in flight
    int32_t acc[FW];
#pragma unroll
    for (int f0 = 0; f0 < FW; f0 += 4) {
      int32_t a[4] = {0, 0, 0, 0};
      int32_t oc[4][4], onx[4][4], wc[4], wnx[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int32_t* to = tw + (f0 + k) * TS;
#pragma unroll
        for (int j = 0; j < 4; ++j) oc[k][j] = to[j];
        wc[k] = to[4 * ca.S4];
      }
      for (int g = 0; g < ca.S4; ++g) {
        const int gn = g + 1 < ca.S4 ? g + 1 : g;         // the next group's loads, in range
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int32_t* to = tw + (f0 + k) * TS;
#pragma unroll
          for (int j = 0; j < 4; ++j) onx[k][j] = to[4 * gn + j];
          wnx[k] = to[4 * ca.S4 + gn];
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) a[k] = __builtin_amdgcn_sdot4(gather4(oc[k]), wc[k], a[k], false);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
#pragma unroll
          for (int j = 0; j < 4; ++j) oc[k][j] = onx[k][j];
          wc[k] = wnx[k];
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[f0 + k] = a[k];
    }
    if (ox < geo.Wo) {
      const int o0 = wv * FW;
      int32_t* yr = y + ((size_t)r * geo.Wo + ox) * geo.c_out + o0;
#pragma unroll
      for (int f = 0; f < FW; f += 4) {
        int4 v4;
        v4.x = acc[f] + (bias ? bias[o0 + f] : 0);
        v4.y = acc[f + 1] + (bias ? bias[o0 + f + 1] : 0);
        v4.z = acc[f + 2] + (bias ? bias[o0 + f + 2] : 0);
        v4.w = acc[f + 3] + (bias ? bias[o0 + f + 3] : 0);
        *reinterpret_cast<int4*>(yr + f) = v4;
      }
    }
  }
}

}  // namespace cs
