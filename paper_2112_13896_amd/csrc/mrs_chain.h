// A whole keyword-spotting-shaped chain in one launch, one workgroup per
// image (Figure 10: every layer's winners go on with their indices; Section
// 4: the first layer runs sparse-dense on the dense input):
//  1. the dense-input first layer on the matrix cores (dense_body: conv, 2x2
//     pool, k-WTA, requantisation) over the whole image, its lists written;
//  2. after a workgroup barrier, the second layer on those lists, its k-WTA
//     lists written: output-stationary (gather_body: 64 input channels, eight
//     list slots, a square window, four sets, every output pixel in LDS) or
//     else input-stationary (scatter_body);
//  3. after another barrier, the layer whose window is the whole pooled map
//     (sample_body) on them, with the last linear layer on its winners.
// The barriers' workgroup-scope release/acquire order each phase's global
// stores before the next phase's loads; the lists come back from L2 of the
// same compute unit.  Each phase lays out the dynamic LDS its own way from
// offset 0 (the launch reserves the largest, about 62 KB).  The registers are
// held to 64 per lane (eight wavefronts per SIMD), so that two workgroups -
// two images, from one batch or from the next batch launched on another
// stream - share a compute unit and fill each other's latency-bound phases;
// a single launch is slower that way, a stream of batches faster.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "conv_dense_mfma.h"
#include "mrs_gather.h"
#include "mrs_sample.h"
#include "mrs_scatter.h"

namespace cs {

// The arguments of the three phases, passed as one value.
struct ChainArgs {
  const int8_t* x;
  const uint16_t* aug0;
  const int32_t* bias0;
  int32_t* y0;
  ListOut lo0;
  ConvGeom geo0;
  DenseArgs da;
  const uint16_t* aug;
  const int32_t* bias;
  int32_t* y;
  ListOut lo;
  ConvGeom geo;
  ScatterArgs sc;
  GatherArgs ga;
  const uint16_t* aug2;
  const int32_t* bias2;
  int32_t* y2;
  ListOut lo2;
  ConvGeom geo2;
  SampleArgs sa2;
  NextLayer nx;
};

// The kernel's argument segment, as a pointer the compiler cannot see
// through: the scalar loads of a phase's arguments stay in that phase instead
// of being hoisted to the kernel's start, where the three phases' arguments
// would all be live at once (more than the scalar registers left at eight
// wavefronts per SIMD, so they were spilled).
__device__ __forceinline__ const ChainArgs* chain_args() {
  auto p = __builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(p));
  return (const ChainArgs*)p;
}

// KM: the first layer's k-WTA selection (its kmode), fixed at compile time;
// GA: the second layer output-stationary (four sets).
template <int POOL, int KW, int KM, bool GA>
__device__ __forceinline__ void dense_chain_body() {
  CS_STAMP_COUNT(15);
  CS_STAMP(0);
  {
    const ChainArgs* a = chain_args();
    const ListOut lo0 = a->lo0;
    const ConvGeom geo0 = a->geo0;
    const DenseArgs da = a->da;
    dense_body<POOL, int8_t, SCAT_BD, KM>(a->x, a->aug0, a->bias0, a->y0, nullptr, lo0, geo0, da,
                                      blockIdx.x);
  }
  __syncthreads();
  CS_STAMP(4);
  {
    const ChainArgs* a = chain_args();
    const ListOut lo0 = a->lo0, lo = a->lo;
    const ConvGeom geo = a->geo;
    if constexpr (GA) {
      const GatherArgs ga = a->ga;
      gather_body<int8_t, KW, 4>(lo0.idx, static_cast<const int8_t*>(lo0.val), lo0.cnt, a->aug,
                                 a->bias, a->y, nullptr, lo, geo, ga, blockIdx.x);
    } else {
      const ScatterArgs sc = a->sc;
      scatter_body<int8_t, KW, 2, 1>(lo0.idx, static_cast<const int8_t*>(lo0.val), lo0.cnt,
                                     a->aug, a->bias, a->y, nullptr, lo, geo, sc, blockIdx.x);
    }
  }
  __syncthreads();
  CS_STAMP(7);
  {
    const ChainArgs* a = chain_args();
    const ListOut lo = a->lo, lo2 = a->lo2;
    const ConvGeom geo2 = a->geo2;
    const SampleArgs sa2 = a->sa2;
    const NextLayer nx = a->nx;
    sample_body<int8_t, int32_t, int8_t>(lo.idx, static_cast<const int8_t*>(lo.val), lo.cnt,
                                         a->aug2, a->bias2, a->y2, nullptr, lo2, geo2, sa2, nx,
                                         blockIdx.x);
  }
#ifdef CS_PHASE_STAMPS
  __syncthreads();
#endif
  CS_STAMP(13);
}

template <int POOL, int KW, int KM>
__global__ __launch_bounds__(SCAT_BD, 8) void dense_scatter_sample(ChainArgs) {
  dense_chain_body<POOL, KW, KM, false>();
}

template <int POOL, int KW, int KM>
__global__ __launch_bounds__(SCAT_BD, 8) void dense_gather_sample(ChainArgs) {
  dense_chain_body<POOL, KW, KM, true>();
}

}  // namespace cs
