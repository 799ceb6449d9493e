// C ABI entry points of the sparse-sparse layer (declared in include/cs.h).
// Every argument is checked on the host before the first HIP call; kernels
// are enqueued on the caller's stream and nothing is allocated, freed or
// synchronised here.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>

#include "compact_kernels.h"
#include "conv_channels.h"
#include "conv_dense_blocks.h"
#include "conv_dense_mfma.h"
#include "cs.h"
#include "kwta_kernels.h"
#include "mrs_blocks.h"
#include "mrs_chain.h"
#include "mrs_fused.h"
#include "mrs_reorder.h"
#include "mrs_kernels.h"
#include "mrs_sample.h"
#include "mrs_rows.h"
#include "mrs_scatter.h"
#include "mrs_tiled.h"

// Scratch of cs_conv2d_noalloc: the compaction lists it would otherwise take
// from a caller's workspace.  A device-side array of the code object (one copy
// per GPU, at that GPU's own address), held until the process ends; host code
// never passes its name to a kernel, only the address noalloc_scratch() looks
// up with hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[CS_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

size_t elem_size(cs_dtype t) { return t == CS_I8 ? 1 : 4; }

bool is_act_dtype(cs_dtype t) { return t == CS_I8 || t == CS_F32; }

int launch_status() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? CS_OK : CS_ERR_DEVICE;
}

int blocks_for(int64_t threads, int bd, int64_t cap = 1 << 20) {
  int64_t b = (threads + bd - 1) / bd;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

// ---------------------------------------------------------------- compaction
int device_cus(int* cus);

// The vectorised compaction's lanes per row group (log2): 16-byte rows of at
// most 16 vectors share a wavefront in power-of-two groups, longer ones take a
// wavefront each; -1 when the rows are not whole 16-byte vectors or x is not
// 16-byte aligned.
int compact_vec_lg(cs_dtype xt, const void* x, int c) {
  const int E = xt == CS_I8 ? 16 : 4;
  if (c % E != 0 || reinterpret_cast<uintptr_t>(x) % 16 != 0) return -1;
  const int nl = c / E;
  if (nl > 16) return 6;
  int lg = 0;
  while ((1 << lg) < nl) ++lg;
  return lg;
}

int compact_checked(cs_dtype xt, const void* x, int64_t rows, int c, uint16_t* idx, void* val,
                    int32_t* cnt, hipStream_t stream) {
  if (rows == 0) return CS_OK;
  const int lg = compact_vec_lg(xt, x, c);
  if (lg >= 0) {
    int cus = 0;
    const int dst = device_cus(&cus);
    if (dst != CS_OK) return dst;
    const int64_t rpw = 64 >> lg;                          // rows per wavefront (lg 6: one)
    const int64_t waves = (rows + rpw - 1) / rpw;
    int64_t blocks = (waves + 3) / 4;                      // 4 wavefronts per workgroup
    const int64_t cap = (int64_t)cus * 16;                 // at most 64 wavefronts per CU
    if (blocks > cap) blocks = cap;
    if (xt == CS_I8)
      hipLaunchKernelGGL(cs::compact_vec<int8_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                         static_cast<const int8_t*>(x), rows, c, lg, idx,
                         static_cast<int8_t*>(val), cnt);
    else
      hipLaunchKernelGGL(cs::compact_vec<float>, dim3((unsigned)blocks), dim3(256), 0, stream,
                         static_cast<const float*>(x), rows, c, lg, idx, static_cast<float*>(val),
                         cnt);
    return launch_status();
  }
  if (c >= 64) {
    const int64_t threads = rows * 64;
    const int grid = blocks_for(threads, 256, 65536);
    if (xt == CS_I8)
      hipLaunchKernelGGL(cs::compact_wide<int8_t>, dim3(grid), dim3(256), 0, stream,
                         static_cast<const int8_t*>(x), rows, c, idx, static_cast<int8_t*>(val),
                         cnt);
    else
      hipLaunchKernelGGL(cs::compact_wide<float>, dim3(grid), dim3(256), 0, stream,
                         static_cast<const float*>(x), rows, c, idx, static_cast<float*>(val),
                         cnt);
  } else {
    int s_log2 = 0;
    while ((1 << s_log2) < c) ++s_log2;
    const int64_t rows_per_wave = 64 >> s_log2;
    const int64_t threads = (rows + rows_per_wave - 1) / rows_per_wave * 64;
    const int grid = blocks_for(threads, 256, 65536);
    if (xt == CS_I8)
      hipLaunchKernelGGL(cs::compact_narrow<int8_t>, dim3(grid), dim3(256), 0, stream,
                         static_cast<const int8_t*>(x), rows, c, s_log2, idx,
                         static_cast<int8_t*>(val), cnt);
    else
      hipLaunchKernelGGL(cs::compact_narrow<float>, dim3(grid), dim3(256), 0, stream,
                         static_cast<const float*>(x), rows, c, s_log2, idx,
                         static_cast<float*>(val), cnt);
  }
  return launch_status();
}

// ---------------------------------------------------------------- MRS
int conv_geometry(int b, int h, int w, int c_in, int kh, int kw, int stride, int pad, int c_out,
                  int n, int pool, cs::ConvGeom* g) {
  if (b < 1 || h < 1 || w < 1 || c_in < 1 || kh < 1 || kw < 1 || stride < 1 || pad < 0 ||
      c_out < 1 || n < 1)
    return CS_ERR_ARG;
  if (c_in > CS_MAX_ROW || n > CS_MAX_N || c_out % n != 0) return CS_ERR_SHAPE;
  if (pool != 1 && pool != 2) return CS_ERR_ARG;
  const int64_t ho = ((int64_t)h + 2 * pad - kh) / stride + 1;
  const int64_t wo = ((int64_t)w + 2 * pad - kw) / stride + 1;
  if (h + 2 * pad < kh || w + 2 * pad < kw || ho < 1 || wo < 1) return CS_ERR_SHAPE;
  if (pool == 2 && (ho % 2 != 0 || wo % 2 != 0)) return CS_ERR_SHAPE;
  if ((int64_t)kh * kw * c_in > INT32_MAX) return CS_ERR_SHAPE;
  g->B = b; g->H = h; g->W = w; g->C = c_in;
  g->KH = kh; g->KW = kw; g->S = stride; g->P = pad;
  g->Ho = (int)ho; g->Wo = (int)wo; g->pool = pool;
  g->G = c_out / n; g->n = n; g->c_out = c_out;
  g->cap = c_in;
  return CS_OK;
}

int device_cus(int* cus) {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return CS_ERR_DEVICE;
  if (dev >= 0 && dev < 64 && cached[dev] > 0) {
    *cus = cached[dev];
    return CS_OK;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v < 1)
    return CS_ERR_DEVICE;
  if (dev >= 0 && dev < 64) cached[dev] = v;
  *cus = v;
  return CS_OK;
}

constexpr size_t kBlockLds = 64 * 1024;   // LDS budget of one workgroup
constexpr size_t kCuLds = 160 * 1024;     // LDS of one compute unit (gfx950)
// LDS is given to a workgroup in units of 1,280 bytes (measured: three
// workgroups of 53,760 bytes run together on a compute unit, three of 54,016
// bytes do not)
constexpr size_t kLdsGranule = 1280;

// Workgroups of `shmem` bytes of LDS that fit on one compute unit at once.
inline int64_t lds_wgs_per_cu(size_t shmem) {
  const size_t g = (shmem + kLdsGranule - 1) / kLdsGranule * kLdsGranule;
  return g == 0 ? 8 : (int64_t)(kCuLds / g);
}

// First version: one lane per (output item, set), packed kernels read from
// global memory.  Used when the lists cannot be read four entries at a time
// (row stride not a multiple of 4) or a table slice cannot fit in LDS.
int mrs_launch_simple(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                      const cs::ConvGeom& geo, const void* aug, const void* bias, void* y,
                      hipStream_t stream) {
  const int64_t opix = (int64_t)geo.B * (geo.Ho / geo.pool) * (geo.Wo / geo.pool);
  const int64_t total = opix * geo.G;
  const bool one = geo.n == 1;
  const int nacc = one ? 1 : geo.n;
  const size_t per_thread = (size_t)nacc * 4 * (geo.pool == 2 ? 2 : 1);
  const int bd = per_thread * 256 <= 32768 ? 256 : 128;
  const size_t shmem = per_thread * bd;
  const int64_t nblocks = (total + bd - 1) / bd;
  if (nblocks > INT32_MAX) return CS_ERR_SHAPE;
  const dim3 grid((unsigned)nblocks), block(bd);
  if (xt == CS_I8) {
    auto* lv = static_cast<const int8_t*>(lval);
    auto* pa = static_cast<const uint16_t*>(aug);
    auto* bs = static_cast<const int32_t*>(bias);
    auto* yy = static_cast<int32_t*>(y);
    if (one)
      hipLaunchKernelGGL((cs::mrs_conv<int8_t, int32_t, true>), grid, block, shmem, stream, idx,
                         lv, cnt, pa, bs, yy, geo, total);
    else
      hipLaunchKernelGGL((cs::mrs_conv<int8_t, int32_t, false>), grid, block, shmem, stream, idx,
                         lv, cnt, pa, bs, yy, geo, total);
  } else {
    auto* lv = static_cast<const float*>(lval);
    auto* pa = static_cast<const uint2*>(aug);
    auto* bs = static_cast<const float*>(bias);
    auto* yy = static_cast<float*>(y);
    if (one)
      hipLaunchKernelGGL((cs::mrs_conv<float, float, true>), grid, block, shmem, stream, idx, lv,
                         cnt, pa, bs, yy, geo, total);
    else
      hipLaunchKernelGGL((cs::mrs_conv<float, float, false>), grid, block, shmem, stream, idx,
                         lv, cnt, pa, bs, yy, geo, total);
  }
  return launch_status();
}

template <typename T, typename A, bool ONE, int GB>
void launch_tiled(dim3 grid, size_t shmem, hipStream_t stream, const uint16_t* idx,
                  const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                  void* y, const cs::ConvGeom& geo, const cs::TiledArgs& ta) {
  hipLaunchKernelGGL((cs::mrs_tiled<T, A, ONE, GB>), grid, dim3(cs::MRS_BD), shmem, stream, idx,
                     static_cast<const T*>(lval), cnt,
                     static_cast<const typename cs::Aug<T>::type*>(aug),
                     static_cast<const A*>(bias), static_cast<A*>(y), geo, ta);
}

template <typename T, typename A>
void launch_tiled_any(bool one, int gb, dim3 grid, size_t shmem, hipStream_t stream,
                      const uint16_t* idx, const void* lval, const int32_t* cnt, const void* aug,
                      const void* bias, void* y, const cs::ConvGeom& geo,
                      const cs::TiledArgs& ta) {
  if (one) {
    if (gb == 2)
      launch_tiled<T, A, true, 2>(grid, shmem, stream, idx, lval, cnt, aug, bias, y, geo, ta);
    else
      launch_tiled<T, A, true, 1>(grid, shmem, stream, idx, lval, cnt, aug, bias, y, geo, ta);
  } else {
    if (gb == 2)
      launch_tiled<T, A, false, 2>(grid, shmem, stream, idx, lval, cnt, aug, bias, y, geo, ta);
    else
      launch_tiled<T, A, false, 1>(grid, shmem, stream, idx, lval, cnt, aug, bias, y, geo, ta);
  }
}

// Sets per table slice: the largest divisor of G that is a multiple of gb and
// whose table fits the workgroup's LDS next to the accumulators; 0 if none.
int table_slice(const cs::ConvGeom& geo, size_t esz, int nacc, int gb) {
  const size_t acc_bytes = (size_t)gb * nacc * cs::MRS_BD * 4;
  if (acc_bytes >= kBlockLds) return 0;
  const size_t R = (size_t)geo.KH * geo.KW * geo.C;
  for (int gs = geo.G; gs >= gb; --gs)                 // table + bias of the slice
    if (geo.G % gs == 0 && gs % gb == 0 &&
        acc_bytes + R * esz * gs + (size_t)gs * nacc * 4 + 16 <= kBlockLds)
      return gs;
  return 0;
}

// ---------------------------------------------------------------- fused layer
constexpr size_t kFusedLds = 80 * 1024;   // two workgroups per compute unit
constexpr size_t kFusedLds3 = 53 * 1024;  // three

size_t round16(size_t v) { return (v + 15) / 16 * 16; }

bool aligned(const void* p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }   // NULL: yes

// Lists can be read 4 entries at a time: row stride a multiple of 4 and the
// arrays aligned for 8-byte index and 4- or 16-byte value loads.
bool lists_vectorisable(cs_dtype xt, const uint16_t* idx, const void* lval, int cap) {
  return cap % 4 == 0 && aligned(idx, 8) && aligned(lval, xt == CS_I8 ? 4 : 16);
}

struct FusedPlan {
  cs::FusedArgs fa;
  size_t shmem;
  int64_t blocks;
  int gb;
};

// Tiles for the fused kernel, or false when the layer does not suit it (the
// table does not fit the LDS next to the accumulators, too many lanes per
// item, misaligned operands, a row too long for the selection).
//
// Candidates (LDS budget for three or two workgroups per compute unit, tile
// shape, slices) are compared with a simple model of the time: workgroups per
// concurrently resident workgroup slot of 256 compute units, times (a fixed
// cost per workgroup for staging and the epilogue + rounds x the list chunks
// one lane walks + the group reduction).
constexpr int kPlanCus = 256;          // MI355X compute units (the model only)
constexpr double kCostFixed = 40.0;    // per workgroup, in list-chunk units
constexpr int kMaxPlanSlices = 4;

bool fused_plan(const cs::ConvGeom& geo, cs_dtype xt, const void* aug, const void* y, int k,
                int shift, int write_sums, int ocap, int osz, FusedPlan* pl) {
  const bool one = geo.n == 1;
  const int n = one ? 1 : geo.n;
  const size_t esz = xt == CS_I8 ? 2 : 8;                 // augmented entry
  const size_t chunk_b = xt == CS_I8 ? 12 : 24;           // 4 indices + 4 values
  const int T = geo.KH * geo.KW;
  const int64_t R = (int64_t)T * geo.C;
  const int64_t ntab = R * geo.G;
  if (ntab * (int64_t)esz >= INT32_MAX || geo.cap % 4 != 0 || geo.c_out % 4 != 0) return false;
  if (!aligned(aug, 16) || !aligned(y, 16)) return false;
  // k-WTA in the epilogue: one lane per item, rows of at most 128 channels
  if (k >= 0 && (geo.c_out > 128 || k > 32)) return false;
  // sets per lane: two when they split evenly and the lane's accumulators fit
  const int gb = (geo.G % 2 == 0 && 2 * n <= cs::FUSED_NACC) ? 2 : 1;
  if (gb * n > cs::FUSED_NACC) return false;
  const int units = geo.G / gb;
  const int log2Q = geo.pool == 2 ? 2 : 0;
  if ((units << log2Q) > cs::MRS_BD) return false;
  const size_t acc_b = (size_t)((gb * n + 7) & ~7) * cs::MRS_BD * 4;   // rows rounded up to 8
  const bool lists = k >= 0 && ocap > 0;
  const size_t fixed = acc_b + round16((size_t)ntab * esz) + round16((size_t)geo.c_out * 4) + 64;
  const bool lane_sel = k >= 0;
  const int ostride = lane_sel ? geo.c_out + 1 : geo.c_out;   // odd: conflict-free lane reads
  const int64_t worst_ch = geo.cap / 4;                  // chunks of a full row
  const size_t min_ch = (size_t)(worst_ch < 4 ? worst_ch : 4);   // planned per pixel, at least
  const bool mode0 = T == 1 && geo.S == 1 && geo.P == 0 && geo.pool == 1;
  const int Hp = geo.Ho / geo.pool, Wp = geo.Wo / geo.pool;
  // list chunks one lane walks for one tap, on average (unknown for dense inputs)
  const double ch_tap = (double)(worst_ch < 4 ? worst_ch : 4);
  auto tile_bytes = [&](int sl, int np, size_t chunks) {
    return fixed + round16((size_t)sl * ostride * 4) + (k >= 0 ? round16((size_t)sl * 8) : 0) +
           (lists ? round16((size_t)sl * ocap * 2) + round16((size_t)sl * ocap * osz) : 0) +
           round16((size_t)np * 8) + chunks * chunk_b + 2 * chunk_b + 32;
  };
  bool found = false;
  double best = 0.0;
  cs::FusedArgs bfa{};
  int64_t bblocks = 0;
  size_t bbudget = 0;
  auto consider = [&](size_t budget, int sl, int np, int64_t blocks, int log2S,
                      const cs::FusedArgs& f) {
    const size_t lds = tile_bytes(sl, np, (size_t)np * min_ch);
    if (lds > budget || np > cs::MRS_BD * cs::FUSED_PPT || blocks < 1 || blocks > INT32_MAX)
      return;
    const int lpi = units << (log2Q + log2S);
    if (lpi > cs::MRS_BD) return;
    const int ipr = cs::MRS_BD / lpi;
    const int rounds = (sl + ipr - 1) / ipr;
    const int S = 1 << log2S;
    const double work = T == 1 ? std::ceil(ch_tap / S) : std::ceil((double)T / S) * ch_tap;
    // the group reduction: one shuffle per accumulator and slice/sub-pixel step
    const double red = (double)gb * n * (log2S + log2Q) / 16.0;
    int bpc = (int)(kCuLds / budget);
    bpc = bpc > 8 ? 8 : (bpc < 1 ? 1 : bpc);
    double waves = (double)blocks / ((double)kPlanCus * bpc);   // fractional, at least one
    waves = waves < 1.0 ? 1.0 : waves;
    const double cost = waves * (kCostFixed + rounds * (work + red));
    if (!found || cost < best) {
      found = true;
      best = cost;
      bfa = f;
      bfa.log2S = log2S;
      bfa.LPI = lpi;
      bfa.IPR = ipr;
      bfa.npix_cap = np;
      bblocks = blocks;
      bbudget = budget;
    }
  };
  const int max_log2S_tap = [&] {
    int l = 0;
    while ((2 << l) <= T && (2 << l) <= kMaxPlanSlices && l + log2Q < 6) ++l;
    return l;
  }();
  const int max_log2S_chunk = [&] {
    int l = 0;
    while ((2 << l) <= worst_ch && (2 << l) <= kMaxPlanSlices && l + log2Q < 6) ++l;
    return l;
  }();
  const int max_log2S = T == 1 ? max_log2S_chunk : max_log2S_tap;
  for (size_t budget : {kFusedLds3, kFusedLds}) {
    if (fixed >= budget) continue;
    for (int log2S = 0; log2S <= max_log2S; ++log2S) {
      const int lpi = units << (log2Q + log2S);
      if (lpi > cs::MRS_BD) break;
      const int ipr = cs::MRS_BD / lpi;
      if (mode0) {
        const int64_t items = (int64_t)geo.B * geo.Ho * geo.Wo;
        for (int r = 1; r <= 4; ++r) {
          const int ti = ipr * r;
          cs::FusedArgs f{};
          f.tile_mode = 0;
          f.TI = ti;
          consider(budget, ti, ti, (items + ti - 1) / ti, log2S, f);
        }
      } else {
        for (int tw = Wp; tw >= 1; tw = (tw > 1 ? (tw + 1) / 2 : 0)) {
          const int iw = (tw * geo.pool - 1) * geo.S + geo.KW;
          for (int tpr = 1; tpr <= Hp; ++tpr) {
            const int ih = (tpr * geo.pool - 1) * geo.S + geo.KH;
            const int64_t np = (int64_t)ih * iw;
            if (np > cs::MRS_BD * cs::FUSED_PPT) break;
            const int sl = tpr * tw;
            if (sl > ipr * 8) break;
            cs::FusedArgs f{};
            f.tile_mode = 1;
            f.TPR = tpr;
            f.TW = tw;
            f.tiles_x = (Wp + tw - 1) / tw;
            f.tiles_img = ((Hp + tpr - 1) / tpr) * f.tiles_x;
            f.IW = iw;
            consider(budget, sl, (int)np, (int64_t)geo.B * f.tiles_img, log2S, f);
          }
          if (tw == 1) break;
        }
      }
    }
  }
  if (!found) return false;
  cs::FusedArgs fa = bfa;
  const int slots = fa.tile_mode == 0 ? fa.TI : fa.TPR * fa.TW;
  if (fa.tile_mode == 1) {
    fa.fd_tw = cs::make_fastdiv((uint32_t)fa.TW);
    fa.fd_iw = cs::make_fastdiv((uint32_t)fa.IW);
    fa.fd_tx = cs::make_fastdiv((uint32_t)fa.tiles_x);
    fa.fd_timg = cs::make_fastdiv((uint32_t)fa.tiles_img);
  }
  // list budget: what is left of the LDS, at most every chunk of every pixel
  const size_t base = tile_bytes(slots, fa.npix_cap, 0);
  if (base >= bbudget) return false;
  int64_t lc = (int64_t)((bbudget - base) / chunk_b);
  if (lc > (int64_t)fa.npix_cap * worst_ch) lc = (int64_t)fa.npix_cap * worst_ch;
  fa.units = units;
  fa.log2Q = log2Q;
  fa.list_cap = (int)lc;
  fa.k = k;
  fa.shift = shift;
  fa.write_sums = write_sums;
  fa.ostride = ostride;
  fa.kmode = k <= 8 ? 1 : (k <= 16 ? 2 : 3);               // one lane per item
  fa.fd_lpi = cs::make_fastdiv((uint32_t)fa.LPI);
  fa.fd_kw = cs::make_fastdiv((uint32_t)geo.KW);
  fa.fd_cout = cs::make_fastdiv((uint32_t)geo.c_out);
  fa.fd_ochunks = cs::make_fastdiv((uint32_t)(lists ? ocap / 4 : 1));
  // LDS layout
  size_t o = acc_b;
  fa.off_tab = (uint32_t)o;
  o += round16((size_t)ntab * esz);
  fa.off_bias = (uint32_t)o;
  o += round16((size_t)geo.c_out * 4);
  fa.off_out = (uint32_t)o;
  o += round16((size_t)slots * fa.ostride * 4);
  fa.off_sel = (uint32_t)o;
  o += k >= 0 ? round16((size_t)slots * 8) : 0;
  fa.off_lidx = (uint32_t)o;
  o += lists ? round16((size_t)slots * ocap * 2) : 0;
  fa.off_lval = (uint32_t)o;
  o += lists ? round16((size_t)slots * ocap * osz) : 0;
  fa.off_pix = (uint32_t)o;
  o += round16((size_t)fa.npix_cap * 8);
  fa.off_cidx = (uint32_t)o;                             // lc chunks + the spare slot
  o += round16((size_t)(lc + 1) * 8);
  fa.off_cval = (uint32_t)o;
  o += round16((size_t)(lc + 1) * (chunk_b - 8));
  fa.off_misc = (uint32_t)o;
  o += 64;
  if (o > bbudget) return false;
  pl->fa = fa;
  pl->shmem = o;
  pl->blocks = bblocks;
  pl->gb = gb;
  return true;
}

template <typename T, typename A, typename TO>
void launch_fused_t(const FusedPlan& pl, hipStream_t stream, const uint16_t* idx,
                    const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                    void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  const dim3 grid((unsigned)pl.blocks), block(cs::MRS_BD);
  const T* lv = static_cast<const T*>(lval);
  const auto* pa = static_cast<const typename cs::Aug<T>::type*>(aug);
  const A* bs = static_cast<const A*>(bias);
  A* yy = static_cast<A*>(y);
  TO* oo = static_cast<TO*>(out);
#define CS_FUSED(ONE_, GB_)                                                                  \
  hipLaunchKernelGGL((cs::mrs_fused<T, A, TO, ONE_, GB_>), grid, block, pl.shmem, stream, idx, \
                     lv, cnt, pa, bs, yy, oo, lo, geo, pl.fa)
  if (geo.n == 1) {
    if (pl.gb == 2) CS_FUSED(true, 2);
    else CS_FUSED(true, 1);
  } else {
    if (pl.gb == 2) CS_FUSED(false, 2);
    else CS_FUSED(false, 1);
  }
#undef CS_FUSED
}

// Launch a planned fused layer.  ot: output dtype of the k-WTA (ignored when
// fa.k < 0).
int launch_fused(const FusedPlan& pl, cs_dtype xt, cs_dtype ot, hipStream_t stream,
                 const uint16_t* idx, const void* lval, const int32_t* cnt, const void* aug,
                 const void* bias, void* y, void* out, const cs::ListOut& lo,
                 const cs::ConvGeom& geo) {
  if (xt == CS_F32)
    launch_fused_t<float, float, float>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo, geo);
  else if (ot == CS_I8)
    launch_fused_t<int8_t, int32_t, int8_t>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo,
                                           geo);
  else
    launch_fused_t<int8_t, int32_t, int32_t>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo,
                                            geo);
  return launch_status();
}

// ------------------------------------------------ fp32 layers, table in row blocks
// A fp32 layer without pooling whose sets and kernels per set are powers of
// two: tiles of pixels complete in the channel dimension, the packed table
// streamed through LDS in blocks of rows, k-WTA over rows of up to 256
// channels in the epilogue (mrs_blocks.h).
struct BlocksPlan {
  cs::BlocksArgs ba;
  int gb;
  bool own;              // k-WTA on the lanes' own accumulator columns
  int64_t blocks;
  size_t shmem;
};

int ilog2_exact(int64_t v) {                    // log2 of a power of two, else -1
  if (v < 1) return -1;
  int l = 0;
  while ((1LL << l) < v) ++l;
  return (1LL << l) == v ? l : -1;
}

// ocap: capacity of the output lists (0: dense output or sums only); lvec:
// the output lists take 8-byte index and 16-byte value stores.
// cus: compute units of the device (sizes the grid of a one-block table), or
// 0 when only planning.
// unit: channels per k-WTA unit (k winners in each), 0 or c_out: the whole row
bool blocks_plan(const cs::ConvGeom& geo, cs_dtype xt, const void* aug, const void* y,
                 const void* out, int k, int write_sums, int ocap, bool lvec, int cus,
                 BlocksPlan* pl, int unit = 0) {
  if (xt != CS_F32 || geo.pool != 1) return false;
  if (unit <= 0) unit = geo.c_out;
  const int n = geo.n, G = geo.G;
  const int log2n = ilog2_exact(n), log2G = ilog2_exact(G);
  if (log2n < 0 || log2G < 1 || n > 16 || geo.c_out > 256) return false;
  if (geo.cap % 4 != 0 || !aligned(aug, 16) || !aligned(y, 4)) return false;
  const int T = geo.KH * geo.KW;
  const int64_t R = (int64_t)T * geo.C;
  const int64_t items = (int64_t)geo.B * geo.Ho * geo.Wo;
  const int64_t in_rows = (int64_t)geo.B * geo.H * geo.W;
  if (items * geo.c_out >= INT32_MAX || in_rows * geo.cap >= INT32_MAX || R * G >= INT32_MAX)
    return false;
  // sets per lane: two (four when the lane count per pixel would pass 64)
  int gb = G >= 2 ? 2 : 1;
  while (gb < 4 && G / gb > 64) gb *= 2;
  if (gb * n > 64 || G / gb > cs::BLK_BD) return false;   // offsets fit 16 bits
  const int U = G / gb;
  // rows per block: the whole table if it fits one workgroup's share of LDS
  // (two workgroups per compute unit); else blocks of at most BLK_ENTRIES
  // entries (the next block waits in registers), double-buffered when two
  // fit, else one buffer refilled between two barriers: whole taps if a tap
  // fits, else a channel range dividing C
  const int tstride = G;                                  // 8-byte entries per row
  const size_t acc_b = (size_t)gb * n * cs::BLK_BD * 4;
  const size_t budget = kCuLds / 2;
  const size_t fixed = acc_b;
  auto lds_for = [&](int64_t rows, int nbuf) {
    return fixed + nbuf * round16((size_t)rows * tstride * 8);
  };
  const int max_rows = cs::BLK_ENTRIES / G;
  int64_t RB = 0;
  int tpb = 0, cblocks = 0, nbuf = 1;
  if (lds_for(R, 1) <= budget) {
    RB = R;
    tpb = T;
  } else if (geo.C <= max_rows && lds_for(geo.C, 1) <= budget) {
    tpb = max_rows / geo.C;
    if (tpb > T) tpb = T;
    while (tpb > 1 && lds_for((int64_t)tpb * geo.C, 1) > budget) --tpb;
    RB = (int64_t)tpb * geo.C;
    nbuf = lds_for(RB, 2) <= budget ? 2 : 1;
  } else {
    RB = geo.C < max_rows ? geo.C : max_rows;
    while (RB >= 4 && (geo.C % RB != 0 || lds_for(RB, 1) > budget)) --RB;
    if (RB < 4) return false;
    cblocks = (int)(geo.C / RB);
    nbuf = lds_for(RB, 2) <= budget ? 2 : 1;
  }
  const int64_t nblocks = (R + RB - 1) / RB;
  if (nblocks == 1) nbuf = 1;
  const size_t tb = round16((size_t)RB * tstride * 8);
  cs::BlocksArgs& ba = pl->ba;
  ba.log2U = ilog2_exact(U);
  ba.P = cs::BLK_BD / U;
  ba.items = (int)items;
  ba.RB = (int)RB;
  ba.nblocks = (int)nblocks;
  ba.tpb = tpb;
  ba.cblocks = cblocks;
  ba.tstride = tstride;
  ba.nbuf = nbuf;
  ba.log2n = log2n;
  ba.log2G = log2G;
  ba.k = k;
  ba.write_sums = write_sums;
  // k-WTA: four lanes per row (the gather kernel's selection) for rows of at
  // most 128 channels and k <= 32, else sixteen lanes per row
  const bool quad = k >= 0 && geo.c_out <= 128 && k <= 32 && (ocap == 0 || (ocap % 4 == 0 && lvec));
  ba.kmode = !quad ? 4 : (k <= 8 ? 1 : (k <= 16 ? 2 : 3));
  ba.kp = geo.c_out <= 64 ? 4 : (geo.c_out <= 128 ? 8 : 16);
  ba.ostride = geo.c_out + 1;                             // odd: conflict-free row reads
  ba.off_t0 = (uint32_t)acc_b;
  ba.off_t1 = (uint32_t)(acc_b + (nbuf - 1) * tb);
  size_t end = acc_b + nbuf * tb;
  // the four-lane epilogue's tile, selections and lists over the table blocks
  const int P = cs::BLK_BD / U;
  ba.off_out = (uint32_t)acc_b;
  ba.off_sel = ba.off_out + (uint32_t)round16((size_t)P * ba.ostride * 4);
  ba.off_lidx = ba.off_sel + (uint32_t)round16((size_t)P * 8);
  ba.off_lval = ba.off_lidx + (uint32_t)round16((size_t)P * ocap * 2);
  const size_t epi_end = ba.off_lval + round16((size_t)P * ocap * 4);
  if (quad && epi_end > end) end = epi_end;
  // k-WTA on the lanes' own accumulator columns: a pixel's lanes in one DPP
  // row (U <= 16), 4..32 channels per lane, 16-byte aligned dense rows
  const int kp_own = gb * n;
  pl->own = U <= 16 && kp_own >= 4 && kp_own <= 32 && (kp_own & (kp_own - 1)) == 0 &&
            aligned(y, 16) && aligned(out, 16);
  // k-WTA units narrower than the row: only on the lanes' own columns, a unit
  // being a power-of-two number of a pixel's lanes
  const int log2Us = unit % kp_own == 0 ? ilog2_exact(unit / kp_own) : -1;
  if (unit != geo.c_out && (!pl->own || log2Us < 0 || log2Us > ilog2_exact(U))) return false;
  ba.log2Us = pl->own ? (log2Us >= 0 ? log2Us : ilog2_exact(U)) : ilog2_exact(U);
  if (pl->own) {
    // a pixel's four lanes hold its four quarters: the four-lane selection
    // in place (a quad selection record per pixel in LDS), else bit by bit
    const bool quad_own = U == 4 && gb == 2 && tpb > 0 && k >= 0 && k <= 32 &&
                          geo.c_out == 4 * kp_own && unit == geo.c_out;
    ba.kmode = quad_own ? (k <= 8 ? 6 : (k <= 16 ? 7 : 8)) : 5;
    if (quad_own) {
      ba.off_sel = (uint32_t)round16(acc_b + nbuf * tb);
      end = ba.off_sel + round16((size_t)P * 8);
    } else {
      end = acc_b + nbuf * tb;
    }
  }
  ba.fd_wo = cs::make_fastdiv((uint32_t)geo.Wo);
  ba.fd_ho = cs::make_fastdiv((uint32_t)geo.Ho);
  ba.fd_kw = cs::make_fastdiv((uint32_t)geo.KW);
  ba.fd_cout = cs::make_fastdiv((uint32_t)geo.c_out);
  ba.fd_ochunks = cs::make_fastdiv((uint32_t)(ocap >= 4 ? ocap / 4 : 1));
  pl->gb = gb;
  pl->shmem = end;
  const int64_t ntiles = (items + ba.P - 1) / ba.P;
  ba.ntiles = (int)ntiles;
  pl->blocks = ntiles;
  if (nblocks == 1) {
    // the table is staged once per workgroup: as many workgroups as fit at
    // once (by LDS), each looping over tiles
    if (cus > 0) {
      int64_t per_cu = lds_wgs_per_cu(end);
      if (per_cu > 8) per_cu = 8;
      if (per_cu < 1) per_cu = 1;
      if (pl->blocks > per_cu * cus) pl->blocks = per_cu * cus;
    }
  }
  return pl->shmem <= kBlockLds * 2 && ntiles < INT32_MAX;
}

int launch_blocks(const BlocksPlan& pl, hipStream_t stream, const uint16_t* idx,
                  const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                  void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  const dim3 grid((unsigned)pl.blocks), block(cs::BLK_BD);
  const float* lv = static_cast<const float*>(lval);
  const uint2* pa = static_cast<const uint2*>(aug);
  const float* bs = static_cast<const float*>(bias);
  float* yy = static_cast<float*>(y);
  float* oo = static_cast<float*>(out);
#define CS_BLOCKS(GB_, CH_, KP_, QK_, QD_)                                               \
  hipLaunchKernelGGL((cs::mrs_blocks_f32<float, GB_, CH_, KP_, QK_, QD_>), grid, block, pl.shmem, \
                     stream, idx, lv, cnt, pa, bs, yy, oo, lo, geo, pl.ba)
// a pixel's lanes fill whole quads (U >= 4): the quads share the list loads
#define CS_BLOCKS_QD(GB_, CH_, KP_)                                                      \
  do {                                                                                  \
    if (pl.ba.log2U >= 2) CS_BLOCKS(GB_, CH_, KP_, 0, true);                            \
    else CS_BLOCKS(GB_, CH_, KP_, 0, false);                                            \
  } while (0)
#define CS_BLOCKS_KP(GB_, CH_)                                                           \
  do {                                                                                  \
    const int kp = pl.own ? GB_ * geo.n : 0;                                            \
    if (kp == 4) CS_BLOCKS_QD(GB_, CH_, 4);                                             \
    else if (kp == 8) CS_BLOCKS_QD(GB_, CH_, 8);                                        \
    else if (kp == 16) CS_BLOCKS_QD(GB_, CH_, 16);                                      \
    else if (kp == 32) CS_BLOCKS_QD(GB_, CH_, 32);                                      \
    else CS_BLOCKS_QD(GB_, CH_, 0);                                                     \
  } while (0)
// the four-lane selection in place: two sets per lane, whole-tap blocks, four
// lanes per pixel
#define CS_BLOCKS_QUAD(KP_)                                                              \
  do {                                                                                  \
    if (pl.ba.kmode == 6) CS_BLOCKS(2, false, KP_, 8, true);                            \
    else if (pl.ba.kmode == 7) CS_BLOCKS(2, false, KP_, 16, true);                      \
    else CS_BLOCKS(2, false, KP_, 32, true);                                            \
  } while (0)
  const bool ch = pl.ba.tpb == 0;
  if (pl.own && pl.ba.kmode >= 6) {
    const int kp = 2 * geo.n;
    if (kp == 4) CS_BLOCKS_QUAD(4);
    else if (kp == 8) CS_BLOCKS_QUAD(8);
    else if (kp == 16) CS_BLOCKS_QUAD(16);
    else CS_BLOCKS_QUAD(32);
  } else if (pl.gb == 1) {
    if (ch) CS_BLOCKS_KP(1, true); else CS_BLOCKS_KP(1, false);
  } else if (pl.gb == 2) {
    if (ch) CS_BLOCKS_KP(2, true); else CS_BLOCKS_KP(2, false);
  } else {
    if (ch) CS_BLOCKS_KP(4, true); else CS_BLOCKS_KP(4, false);
  }
#undef CS_BLOCKS_QUAD
#undef CS_BLOCKS_KP
#undef CS_BLOCKS_QD
#undef CS_BLOCKS
  return launch_status();
}

// ------------------------------------------------ one sample per workgroup
// A layer whose output is one vector per sample (a linear layer, or a
// convolution whose window is the whole unpadded input map) runs with one
// workgroup per sample, whatever the size of its table.
struct SamplePlan {
  cs::SampleArgs sa;
  size_t shmem;
};

bool sample_plan(const cs::ConvGeom& geo, cs_dtype xt, int k, int shift, int write_sums,
                 SamplePlan* pl) {
  if (geo.Ho != 1 || geo.Wo != 1 || geo.pool != 1 || geo.KH != geo.H || geo.KW != geo.W ||
      geo.P != 0)
    return false;
  const int npix = geo.H * geo.W;
  if (npix > cs::SAMPLE_BD || geo.c_out > cs::SAMPLE_MAX_ROW) return false;
  const int64_t ents = (int64_t)npix * geo.cap;
  if ((int64_t)geo.B * ents >= INT32_MAX || (int64_t)geo.B * geo.c_out >= INT32_MAX) return false;
  // all workgroups resident at once: the whole LDS of a compute unit; else
  // two workgroups per compute unit
  const size_t budget = geo.B <= kPlanCus ? kCuLds : kFusedLds;
  const size_t asz = 4;                                  // int32 / fp32 sums
  const size_t hist_b = k >= 0 ? 2 * cs::SAMPLE_BINS * 4 : 0;
  const size_t ent_b = round16((size_t)(ents + cs::SAMPLE_ENT_PAD) * 4);
  const size_t fixed = round16((size_t)geo.c_out * asz) + 2 * ent_b +
                       round16((size_t)npix * 8) + hist_b + cs::SAMPLE_MISC * 4;
  const size_t slice = round16((size_t)geo.c_out * asz);
  if (fixed + slice > budget) return false;
  int S = cs::SAMPLE_BD / geo.G;
  // int32 sums share one accumulator row (LDS atomics); fp32 slices own one each
  const int smax = xt == CS_I8 ? cs::SAMPLE_MAX_SLICES : (int)((budget - fixed) / slice);
  S = S > smax ? smax : S;
  S = S > cs::SAMPLE_MAX_SLICES ? cs::SAMPLE_MAX_SLICES : S;
  S = S < 1 ? 1 : S;
  const int acc_rows = xt == CS_I8 ? 1 : S;
  cs::SampleArgs& sa = pl->sa;
  sa.npix = npix;
  sa.S = S;
  sa.k = k;
  sa.shift = shift;
  sa.write_sums = write_sums;
  sa.fd_cap = cs::make_fastdiv((uint32_t)geo.cap);
  sa.fd_g = cs::make_fastdiv((uint32_t)geo.G);
  sa.fd_n = cs::make_fastdiv((uint32_t)geo.n);
  size_t o = (size_t)acc_rows * slice;
  sa.off_row = (uint32_t)o;
  o += round16((size_t)geo.c_out * asz);
  sa.off_ent = (uint32_t)o;
  o += ent_b;
  sa.off_val = (uint32_t)o;
  o += ent_b;
  sa.off_pix = (uint32_t)o;
  o += round16((size_t)npix * 8);
  sa.off_hist = (uint32_t)o;
  o += hist_b;
  sa.off_misc = (uint32_t)o;
  o += cs::SAMPLE_MISC * 4;
  pl->shmem = o;
  return o <= budget;
}

template <typename T, typename A, typename TO>
void launch_sample_t(const SamplePlan& pl, hipStream_t stream, const uint16_t* idx,
                     const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                     void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo,
                     const cs::NextLayer& nx) {
  using E = typename cs::Aug<T>::type;
  const size_t shmem = nx.aug ? (size_t)nx.off_acc + round16((size_t)nx.c_out * 4) : pl.shmem;
  hipLaunchKernelGGL((cs::mrs_sample<T, A, TO>), dim3(geo.B), dim3(cs::SAMPLE_BD), shmem,
                     stream, idx, static_cast<const T*>(lval), cnt, static_cast<const E*>(aug),
                     static_cast<const A*>(bias), static_cast<A*>(y), static_cast<TO*>(out), lo,
                     geo, pl.sa, nx);
}

int launch_sample(const SamplePlan& pl, cs_dtype xt, cs_dtype ot, hipStream_t stream,
                  const uint16_t* idx, const void* lval, const int32_t* cnt, const void* aug,
                  const void* bias, void* y, void* out, const cs::ListOut& lo,
                  const cs::ConvGeom& geo, const cs::NextLayer& nx = cs::NextLayer{}) {
  if (xt == CS_F32)
    launch_sample_t<float, float, float>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo, geo,
                                         nx);
  else if (ot == CS_I8)
    launch_sample_t<int8_t, int32_t, int8_t>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo,
                                             geo, nx);
  else
    launch_sample_t<int8_t, int32_t, int32_t>(pl, stream, idx, lval, cnt, aug, bias, y, out, lo,
                                              geo, nx);
  return launch_status();
}

// ------------------------------------------- input-stationary int8 layer
// An int8 convolution with stride 1 whose band of output rows (every column
// and channel, int32) fits in LDS runs input-stationary: each non-zero
// scatters its products into the band's shared accumulators.
struct ScatterPlan {
  cs::ScatterArgs sc;
  size_t shmem;
  int64_t blocks;
  int gpl, m;
};

bool scatter_plan(const cs::ConvGeom& geo, cs_dtype xt, const void* aug, int k, int shift,
                  int write_sums, ScatterPlan* pl) {
  if (xt != CS_I8 || geo.S != 1 || geo.KH > cs::SCAT_MAX_KH) return false;
  if (geo.KW != 3 && geo.KW != 5 && geo.KW != 7) return false;
  if (geo.c_out > 128 || geo.W > 255 || geo.C > 65535 || !aligned(aug, 4)) return false;
  const int64_t R = (int64_t)geo.KH * geo.KW * geo.C;
  if ((R * geo.G) % 2 != 0 || R * geo.G * 2 >= INT32_MAX) return false;
  const int gpl = geo.G % 2 == 0 ? 2 : 1;
  const int ostride = geo.c_out + 16;
  const int guard = (geo.KW * ostride + 64 + 3) & ~3;
  const size_t tab_b = round16((size_t)R * geo.G * 2);
  for (size_t budget : {kFusedLds, kCuLds}) {
    for (int BR = geo.Ho; BR >= geo.pool; BR -= geo.pool) {
      if (BR % geo.pool != 0) continue;
      const int rows_in = std::min(BR + geo.KH - 1, geo.H);
      const int64_t npix = (int64_t)rows_in * geo.W;
      if (npix > cs::SCAT_BD || rows_in > 255) continue;
      const int64_t ne = npix * geo.cap;
      if (ne >= INT32_MAX / 2) continue;
      const size_t acc_b = round16((size_t)(2 * guard + (int64_t)BR * geo.Wo * ostride) * 4);
      const size_t o_tab = acc_b;
      const size_t o_ent = o_tab + tab_b;
      const size_t o_pix = o_ent + round16((size_t)ne * 8);
      const size_t o_bias = o_pix + round16((size_t)npix * 8);
      const size_t o_misc = o_bias + round16((size_t)geo.c_out * 4);
      const size_t total = o_misc + cs::SAMPLE_MISC * 4;
      if (total > budget) continue;
      const int bands = (geo.Ho + BR - 1) / BR;
      cs::ScatterArgs& sc = pl->sc;
      sc.BR = BR;
      sc.bands = bands;
      sc.guard = guard;
      sc.ostride = ostride;
      sc.k = k;
      sc.shift = shift;
      sc.write_sums = write_sums;
      sc.off_tab = (uint32_t)o_tab;
      sc.off_ent = (uint32_t)o_ent;
      sc.off_pix = (uint32_t)o_pix;
      sc.off_bias = (uint32_t)o_bias;
      sc.off_misc = (uint32_t)o_misc;
      sc.fd_gpc = cs::make_fastdiv((uint32_t)(geo.G / gpl));
      sc.fd_bands = cs::make_fastdiv((uint32_t)bands);
      sc.fd_wp = cs::make_fastdiv((uint32_t)(geo.Wo / geo.pool));
      sc.fd_cap = cs::make_fastdiv((uint32_t)geo.cap);
      sc.fd_w = cs::make_fastdiv((uint32_t)geo.W);
      pl->shmem = total;
      pl->blocks = (int64_t)geo.B * bands;
      pl->gpl = gpl;
      pl->m = geo.c_out > 64 ? 2 : 1;
      return pl->blocks <= INT32_MAX;
    }
  }
  return false;
}

template <typename TO, int KW, int GPL, int M>
void launch_scatter_t(const ScatterPlan& pl, hipStream_t stream, const uint16_t* idx,
                      const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                      void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  hipLaunchKernelGGL((cs::mrs_scatter<TO, KW, GPL, M>), dim3((unsigned)pl.blocks),
                     dim3(cs::SCAT_BD), pl.shmem, stream, idx, static_cast<const int8_t*>(lval),
                     cnt, static_cast<const uint16_t*>(aug), static_cast<const int32_t*>(bias),
                     static_cast<int32_t*>(y), static_cast<TO*>(out), lo, geo, pl.sc);
}

template <typename TO, int KW>
void launch_scatter_kw(const ScatterPlan& pl, hipStream_t s, const uint16_t* idx, const void* lval,
                       const int32_t* cnt, const void* aug, const void* bias, void* y, void* out,
                       const cs::ListOut& lo, const cs::ConvGeom& geo) {
  if (pl.gpl == 2) {
    if (pl.m == 1) launch_scatter_t<TO, KW, 2, 1>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
    else launch_scatter_t<TO, KW, 2, 2>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  } else {
    if (pl.m == 1) launch_scatter_t<TO, KW, 1, 1>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
    else launch_scatter_t<TO, KW, 1, 2>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  }
}

template <typename TO>
void launch_scatter_to(const ScatterPlan& pl, hipStream_t s, const uint16_t* idx,
                       const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                       void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  switch (geo.KW) {
    case 3: launch_scatter_kw<TO, 3>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    case 5: launch_scatter_kw<TO, 5>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    default: launch_scatter_kw<TO, 7>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
  }
}

int launch_scatter(const ScatterPlan& pl, cs_dtype ot, hipStream_t s, const uint16_t* idx,
                   const void* lval, const int32_t* cnt, const void* aug, const void* bias,
                   void* y, void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  if (ot == CS_I8)
    launch_scatter_to<int8_t>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  else
    launch_scatter_to<int32_t>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  return launch_status();
}

// ------------------------------------------------- one wavefront per item
// A one-tap layer (1x1 conv with stride 1, or linear) with many items, a
// table that fits LDS and a k-WTA over long rows: each wavefront takes whole
// items.
constexpr int64_t kRowsMinItems = 4096;   // fewer items: too few wavefronts to fill the chip
constexpr size_t kRowsTabLds = 48 * 1024;

struct RowsPlan {
  cs::RowsArgs ra;
  size_t shmem, tab_b;
  int64_t blocks, items;
  int cpl, waves;
};

// LDS bytes of the row kernel with w wavefronts per workgroup
size_t rows_shmem(const RowsPlan& pl, int w, int c_out) {
  return round16(pl.tab_b) + (size_t)w * (pl.ra.acc_words * 4 + cs::ROWS_ENT_STRIDE * 8) +
         round16((size_t)c_out * 4);
}

// w wavefronts per workgroup, wcu of them resident per compute unit: LDS
// offsets, and as many workgroups as fit the chip at once, each with an even
// share of the items
bool rows_layout(RowsPlan* pl, int w, int wcu, int c_out) {
  if (wcu < w) return false;
  cs::RowsArgs& ra = pl->ra;
  ra.off_acc = (uint32_t)round16(pl->tab_b);
  ra.off_bias = ra.off_acc + w * ra.acc_words * 4;
  ra.off_ent = ra.off_bias + (uint32_t)round16((size_t)c_out * 4);
  pl->shmem = rows_shmem(*pl, w, c_out);
  pl->waves = w;
  const int64_t wgs = std::min<int64_t>((int64_t)kPlanCus * (wcu / w), (pl->items + w - 1) / w);
  ra.per_wg = (pl->items + wgs - 1) / wgs;
  pl->blocks = (pl->items + ra.per_wg - 1) / ra.per_wg;
  return pl->shmem <= kCuLds;
}

// channels per lane of the row kernel's k-WTA (odd, 64 * cpl >= c_out)
int rows_cpl(int c_out) {
  for (int cpl : {3, 5, 9, 17, 33})
    if (64 * cpl >= c_out) return cpl;
  return 0;
}

bool rows_plan(const cs::ConvGeom& geo, cs_dtype xt, const void* aug, int k, int shift,
               int write_sums, RowsPlan* pl) {
  if (xt != CS_I8) return false;
  if (geo.KH != 1 || geo.KW != 1 || geo.S != 1 || geo.P != 0 || geo.pool != 1) return false;
  // sums only, or a k-WTA the fused kernel's epilogue cannot take (rows over
  // 128 or k over 32), which would otherwise need its own kernel and the sums in HBM
  if (k >= 0 && geo.c_out <= 128 && k <= 32) return false;
  if (k < 0 && !write_sums) return false;
  if (geo.c_out > 2048 || !aligned(aug, 16)) return false;
  const int64_t items = (int64_t)geo.B * geo.H * geo.W;
  if (items < kRowsMinItems || items * geo.cap >= INT32_MAX * 4LL) return false;
  const size_t tab_b = (size_t)geo.C * geo.G * 2;
  if (tab_b > kRowsTabLds || (int64_t)geo.C * geo.G >= (1 << 24)) return false;
  const int cpl = rows_cpl(geo.c_out);
  if (cpl == 0) return false;
  cs::RowsArgs& ra = pl->ra;
  ra.k = k;
  ra.shift = shift;
  ra.write_sums = write_sums;
  // groups of 64 sets with wavefront-uniform entries; a rest of at most 32
  // sets as slices, a larger rest as one more (partial) group
  int qf = geo.G / 64, rest = geo.G % 64;
  ra.gbase = 64 * qf;
  if (rest > 32) {
    ++qf;
    rest = 0;
  }
  ra.qf = qf;
  ra.S = rest > 0 ? 64 / rest : 0;
  ra.acc_words = (uint32_t)std::max(64 * cpl, cs::ROWS_HIST);
  ra.acc_words = (ra.acc_words + 3) & ~3u;
  ra.fd_g = cs::make_fastdiv((uint32_t)(rest > 0 ? rest : 1));
  pl->items = items;
  pl->tab_b = tab_b;
  // an estimate for the plan report (LDS only); the launch sizes the
  // workgroups and the grid from the kernel's actual occupancy
  pl->cpl = cpl;
  for (int w : {16, 8, 4}) {
    const size_t sh = rows_shmem(*pl, w, geo.c_out);
    if (sh <= kCuLds)
      return rows_layout(pl, w, std::min<int>(32, (int)lds_wgs_per_cu(sh) * w), geo.c_out);
  }
  return false;
}

// Resident workgroups per compute unit of a kernel at a block size and LDS
// size (0 when the query fails).
int occupancy(const void* kern, int threads, size_t shmem) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, threads, shmem) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return nb;
}

template <typename TO, int CPL>
void launch_rows_c(RowsPlan pl, hipStream_t s, const uint16_t* idx, const void* lval,
                   const int32_t* cnt, const void* aug, const void* bias, void* y, void* out,
                   const cs::ListOut& lo, const cs::ConvGeom& geo) {
  auto go = [&](auto kern) {
    // the workgroup size with the most resident wavefronts per compute unit
    // (registers and LDS), the larger on a tie
    // resident workgroups per LDS size class, cached per kernel (-1: not yet asked)
    static std::atomic<int> occ_cache[3][2] = {{{-1}, {-1}}, {{-1}, {-1}}, {{-1}, {-1}}};
    int best_w = 0, best_cu = 0;
    int wi = 0;
    for (int w : {16, 8, 4}) {
      const size_t sh = rows_shmem(pl, w, geo.c_out);
      const int slot = wi++;
      if (sh > kCuLds) continue;
      int occ = -1;
      if ((size_t)occ_cache[slot][0].load() == sh) occ = occ_cache[slot][1].load();
      if (occ < 0) {
        occ = occupancy(reinterpret_cast<const void*>(kern), 64 * w, sh);
        occ_cache[slot][1].store(occ);
        occ_cache[slot][0].store((int)sh);
      }
      const int wcu = occ * w;
      if (wcu > best_cu) {
        best_cu = wcu;
        best_w = w;
      }
    }
    if (best_w > 0) rows_layout(&pl, best_w, best_cu, geo.c_out);   // else the plan's layout
    hipLaunchKernelGGL(kern, dim3((unsigned)pl.blocks), dim3(64 * pl.waves), pl.shmem, s, idx,
                       static_cast<const int8_t*>(lval), cnt, static_cast<const uint16_t*>(aug),
                       static_cast<const int32_t*>(bias), static_cast<int32_t*>(y),
                       static_cast<TO*>(out), lo, geo, pl.ra, pl.items);
  };
  if (geo.c_out == 64 * CPL)
    go(cs::mrs_rows<TO, CPL, true>);
  else
    go(cs::mrs_rows<TO, CPL, false>);
}

template <typename TO>
void launch_rows_t(const RowsPlan& pl, hipStream_t s, const uint16_t* idx, const void* lval,
                   const int32_t* cnt, const void* aug, const void* bias, void* y, void* out,
                   const cs::ListOut& lo, const cs::ConvGeom& geo) {
  switch (pl.cpl) {
    case 3: launch_rows_c<TO, 3>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    case 5: launch_rows_c<TO, 5>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    case 9: launch_rows_c<TO, 9>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    case 17: launch_rows_c<TO, 17>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
    default: launch_rows_c<TO, 33>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo); break;
  }
}

int launch_rows(const RowsPlan& pl, cs_dtype ot, hipStream_t s, const uint16_t* idx,
                const void* lval, const int32_t* cnt, const void* aug, const void* bias, void* y,
                void* out, const cs::ListOut& lo, const cs::ConvGeom& geo) {
  if (ot == CS_I8)
    launch_rows_t<int8_t>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  else
    launch_rows_t<int32_t>(pl, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  return launch_status();
}

int mrs_launch_tiled(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                     const cs::ConvGeom& geo, const void* aug, const void* bias, void* y,
                     hipStream_t stream);

// Sums of a layer: one workgroup per sample for a linear layer, else the fused
// kernel (lists staged in LDS) when the layer suits it, else the table-slice
// kernel, else the one-lane-per-output kernel.
int mrs_launch(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
               const cs::ConvGeom& geo, const void* aug, const void* bias, void* y,
               hipStream_t stream) {
  SamplePlan sp;
  if (sample_plan(geo, xt, -1, 0, 1, &sp))
    return launch_sample(sp, xt, xt, stream, idx, lval, cnt, aug, bias, y, nullptr,
                         cs::ListOut{nullptr, nullptr, nullptr, 0}, geo);
  ScatterPlan scp;
  if (scatter_plan(geo, xt, aug, -1, 0, 1, &scp))
    return launch_scatter(scp, CS_I32, stream, idx, lval, cnt, aug, bias, y, nullptr,
                          cs::ListOut{nullptr, nullptr, nullptr, 0}, geo);
  RowsPlan rp;
  if (rows_plan(geo, xt, aug, -1, 0, 1, &rp))
    return launch_rows(rp, CS_I32, stream, idx, lval, cnt, aug, bias, y, nullptr,
                       cs::ListOut{nullptr, nullptr, nullptr, 0}, geo);
  if (lists_vectorisable(xt, idx, lval, geo.cap)) {
    BlocksPlan bp;
    int cus = 0;
    const int dst = device_cus(&cus);
    if (dst != CS_OK) return dst;
    if (blocks_plan(geo, xt, aug, y, nullptr, -1, 1, 0, false, cus, &bp))
      return launch_blocks(bp, stream, idx, lval, cnt, aug, bias, y, nullptr,
                           cs::ListOut{nullptr, nullptr, nullptr, 0}, geo);
    FusedPlan fp;
    if (fused_plan(geo, xt, aug, y, -1, 0, 1, 0, 0, &fp))
      return launch_fused(fp, xt, xt, stream, idx, lval, cnt, aug, bias, y, nullptr,
                          cs::ListOut{nullptr, nullptr, nullptr, 0}, geo);
  }
  return mrs_launch_tiled(xt, idx, lval, cnt, geo, aug, bias, y, stream);
}

int mrs_launch_tiled(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                     const cs::ConvGeom& geo, const void* aug, const void* bias, void* y,
                     hipStream_t stream) {
  const bool one = geo.n == 1;
  const int nacc = one ? 1 : geo.n;
  const int T = geo.KH * geo.KW;
  const int64_t R = (int64_t)T * geo.C;
  const size_t esz = xt == CS_I8 ? 2 : 8;               // augmented entry bytes
  // two sets per lane when they split evenly and fit; else one
  int gb = 2;
  int Gs = geo.G % 2 == 0 ? table_slice(geo, esz, nacc, 2) : 0;
  if (Gs < 2) {
    gb = 1;
    Gs = table_slice(geo, esz, nacc, 1);
  }
  cs::TiledArgs ta;
  ta.chunk_mode = T == 1 ? 1 : 0;
  ta.log2Q = geo.pool == 2 ? 2 : 0;
  // tap mode: each lane walks at most MRS_TAPS taps
  int log2S = 0;
  if (!ta.chunk_mode)
    while (((T + (1 << log2S) - 1) >> log2S) > cs::MRS_TAPS) ++log2S;
  const int64_t items = (int64_t)geo.B * (geo.Ho / geo.pool) * (geo.Wo / geo.pool);
  const int64_t in_rows = (int64_t)geo.B * geo.H * geo.W;
  // 32-bit offsets inside the kernel: element offsets and lane counts below 2^31
  const bool fits32 = in_rows * geo.cap < INT32_MAX && items * geo.c_out < INT32_MAX &&
                      R * geo.G < INT32_MAX && items * geo.G * 64 < INT32_MAX;
  if (!lists_vectorisable(xt, idx, lval, geo.cap) || Gs < 1 || log2S + ta.log2Q > 6 || !fits32)
    return mrs_launch_simple(xt, idx, lval, cnt, geo, aug, bias, y, stream);
  int cus = 0;
  const int st = device_cus(&cus);
  if (st != CS_OK) return st;
  ta.Gs = Gs;
  ta.gslices = geo.G / Gs;
  ta.items = (int)items;
  ta.vec_stage = ta.gslices == 1 && (R * Gs * esz) % 16 == 0 &&
                 reinterpret_cast<uintptr_t>(aug) % 16 == 0;
  ta.fd_gs = cs::make_fastdiv((uint32_t)Gs);
  ta.fd_units = cs::make_fastdiv((uint32_t)(Gs / gb));
  ta.fd_wp = cs::make_fastdiv((uint32_t)(geo.Wo / geo.pool));
  ta.fd_hp = cs::make_fastdiv((uint32_t)(geo.Ho / geo.pool));
  ta.fd_kw = cs::make_fastdiv((uint32_t)geo.KW);
  const size_t tab_bytes = ((size_t)R * Gs * esz + 15) / 16 * 16;
  const size_t shmem = (size_t)gb * nacc * cs::MRS_BD * 4 + tab_bytes + (size_t)Gs * nacc * 4;
  int bpc = (int)lds_wgs_per_cu(shmem);
  bpc = bpc < 1 ? 1 : (bpc > 8 ? 8 : bpc);              // 8 x 256 threads fill a compute unit
  const int64_t grid_lanes = (int64_t)cus * bpc * cs::MRS_BD;
  const int64_t units = items * (geo.G / gb);
  // more slices while the grid is not covered twice: up to one slice per tap
  // (tap mode) or per 64 list slots (chunk mode), and 64 lanes per group
  const int64_t max_s = ta.chunk_mode ? (geo.C >= 128 ? geo.C / 64 : 1) : T;
  while (log2S + ta.log2Q < 6 && (2LL << log2S) <= max_s &&
         units * ((int64_t)1 << (log2S + ta.log2Q)) < 2 * grid_lanes)
    ++log2S;
  ta.log2S = log2S;
  ta.S = 1 << log2S;
  const int64_t lanes_per_slice = items * (Gs / gb) * ((int64_t)1 << (log2S + ta.log2Q));
  int64_t blocks_per_slice = (lanes_per_slice + cs::MRS_BD - 1) / cs::MRS_BD;
  const int64_t cap_blocks = ((int64_t)cus * bpc + ta.gslices - 1) / ta.gslices;
  if (blocks_per_slice > cap_blocks) blocks_per_slice = cap_blocks;
  if (blocks_per_slice < 1) blocks_per_slice = 1;
  const dim3 grid((unsigned)(blocks_per_slice * ta.gslices));
  if (xt == CS_I8)
    launch_tiled_any<int8_t, int32_t>(one, gb, grid, shmem, stream, idx, lval, cnt, aug, bias,
                                      y, geo, ta);
  else
    launch_tiled_any<float, float>(one, gb, grid, shmem, stream, idx, lval, cnt, aug, bias, y,
                                   geo, ta);
  return launch_status();
}

struct WsLayout {
  size_t idx_off, val_off, cnt_off, total;
};

WsLayout ws_layout(cs_dtype xt, int64_t rows, int c_in) {
  WsLayout l;
  l.idx_off = 0;
  l.val_off = align_up((size_t)rows * c_in * 2);
  l.cnt_off = l.val_off + align_up((size_t)rows * c_in * elem_size(xt));
  l.total = l.cnt_off + align_up((size_t)rows * 4);
  return l;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char* g_scratch[kMaxDevices] = {};

// The device address of the current device's scratch, looked up on the first
// call with that device current and kept per device.
int noalloc_scratch(unsigned char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return CS_ERR_DEVICE;
  }
  if (dev < 0 || dev >= kMaxDevices) return CS_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return CS_ERR_DEVICE;
    }
    if (reinterpret_cast<uintptr_t>(p) % kAlign != 0) return CS_ERR_DEVICE;
    g_scratch[dev] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch[dev];
  return CS_OK;
}

// ---------------------------------------------------------------- k-WTA
template <typename TI, typename TO>
int kwta_dispatch(const TI* in, int64_t rows, int c, int k, TO* out, int shift,
                  hipStream_t stream, cs::ListOut lo = cs::ListOut{nullptr, nullptr, nullptr, 0}) {
  if (c <= 64 && k <= 32) {
    const int64_t nb = (rows + cs::KWTA_LANE_ROWS - 1) / cs::KWTA_LANE_ROWS;
    if (nb > INT32_MAX) return CS_ERR_SHAPE;
    const size_t shmem = (size_t)cs::KWTA_LANE_ROWS * (c + 1) * 4;
    const dim3 grid((unsigned)nb), block(cs::KWTA_LANE_ROWS);
    const cs::FastDiv fd_c = cs::make_fastdiv((uint32_t)c);
    if (k <= 8)
      hipLaunchKernelGGL((cs::kwta_lane<TI, TO, 8>), grid, block, shmem, stream, in, rows, c, k,
                         out, shift, fd_c, lo);
    else if (k <= 16)
      hipLaunchKernelGGL((cs::kwta_lane<TI, TO, 16>), grid, block, shmem, stream, in, rows, c, k,
                         out, shift, fd_c, lo);
    else
      hipLaunchKernelGGL((cs::kwta_lane<TI, TO, 32>), grid, block, shmem, stream, in, rows, c, k,
                         out, shift, fd_c, lo);
    return launch_status();
  }
  const int m = (c + 63) / 64;
  const int64_t nb64 = (rows + cs::KWTA_WAVE_WAVES - 1) / cs::KWTA_WAVE_WAVES;
  const int nb = (int)(nb64 < 65536 ? nb64 : 65536);
  const dim3 grid(nb), block(64 * cs::KWTA_WAVE_WAVES);
#define CS_KWTA_WAVE(MM)                                                                  \
  hipLaunchKernelGGL((cs::kwta_wave<TI, TO, MM>), grid, block,                                  \
                     (size_t)cs::KWTA_WAVE_WAVES * cs::WAVE_HIST * 4, stream, in, rows, c, k, out, \
                     shift, lo)
  if (m <= 1) CS_KWTA_WAVE(1);
  else if (m <= 2) CS_KWTA_WAVE(2);
  else if (m <= 4) CS_KWTA_WAVE(4);
  else if (m <= 8) CS_KWTA_WAVE(8);
  else if (m <= 16) CS_KWTA_WAVE(16);
  else CS_KWTA_WAVE(32);
#undef CS_KWTA_WAVE
  return launch_status();
}

}  // namespace

extern "C" {

int cs_compact(cs_dtype xt, const void* x, int64_t rows, int c, uint16_t* idx, void* val,
               int32_t* cnt, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  if (rows < 0 || c < 1) return CS_ERR_ARG;
  if (c > CS_MAX_ROW) return CS_ERR_SHAPE;
  if (rows > 0 && (!x || !idx || !val || !cnt)) return CS_ERR_ARG;
  return compact_checked(xt, x, rows, c, idx, val, cnt, static_cast<hipStream_t>(stream));
}

int cs_mrs_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt, int cap,
                  int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                  const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                  void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (cap < 1) return CS_ERR_SHAPE;
  if (!idx || !lval || !cnt || !aug || !y) return CS_ERR_ARG;
  geo.cap = cap;
  return mrs_launch(xt, idx, lval, cnt, geo, aug, bias, y, static_cast<hipStream_t>(stream));
}

int cs_mrs_kwta_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, void* out, uint16_t* oidx,
                       void* oval, int32_t* ocnt, int ocap, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  const cs_dtype at = xt == CS_I8 ? CS_I32 : CS_F32;
  if (!(ot == at || (xt == CS_I8 && ot == CS_I8))) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (cap < 1) return CS_ERR_SHAPE;
  if (!idx || !lval || !cnt || !aug || !y) return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0 || shift < 0 || shift > 31) return CS_ERR_ARG;
  if (k > c_out || c_out > CS_MAX_KWTA_ROW) return CS_ERR_SHAPE;
  const bool lists = oidx != nullptr;
  if (lists == (out != nullptr)) return CS_ERR_ARG;        // exactly one output form
  if (lists && (!oval || !ocnt || ocap < 1)) return CS_ERR_ARG;
  if (lists && ocap < k) return CS_ERR_SHAPE;
  geo.cap = cap;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const cs::ListOut lo{oidx, oval, ocnt, lists ? ocap : 0};
  // the fused kernel writes lists 4 entries at a time
  const int osz = ot == CS_I8 ? 1 : 4;
  const bool lists_ok = !lists || (ocap % 4 == 0 && aligned(oidx, 8) && aligned(oval, osz * 4));
  {
    SamplePlan sp;
    if (sample_plan(geo, xt, k, shift, keep_sums, &sp))
      return launch_sample(sp, xt, ot, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
    ScatterPlan scp;
    if (scatter_plan(geo, xt, aug, k, shift, keep_sums, &scp))
      return launch_scatter(scp, ot, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
    RowsPlan rp;
    if (rows_plan(geo, xt, aug, k, shift, keep_sums, &rp))
      return launch_rows(rp, ot, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  }
  if (lists_vectorisable(xt, idx, lval, cap)) {
    BlocksPlan bp;
    const bool lvec = lists && aligned(oidx, 8) && aligned(oval, 16);
    int cus = 0;
    if (xt == CS_F32) {
      const int dst = device_cus(&cus);
      if (dst != CS_OK) return dst;
    }
    if (blocks_plan(geo, xt, aug, y, out, k, keep_sums, lists ? ocap : 0, lvec, cus, &bp))
      return launch_blocks(bp, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  }
  if (lists_ok && lists_vectorisable(xt, idx, lval, cap)) {
    FusedPlan fp;
    if (fused_plan(geo, xt, aug, y, k, shift, keep_sums, lists ? ocap : 0, osz, &fp))
      return launch_fused(fp, xt, ot, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  }
  // two kernels: the sums into y, then k-WTA from y
  st = mrs_launch(xt, idx, lval, cnt, geo, aug, bias, y, s);
  if (st != CS_OK) return st;
  const int64_t rows = (int64_t)b * (geo.Ho / pool) * (geo.Wo / pool);
  if (xt == CS_F32)
    return kwta_dispatch(static_cast<const float*>(y), rows, c_out, k, static_cast<float*>(out),
                         0, s, lo);
  if (ot == CS_I8)
    return kwta_dispatch(static_cast<const int32_t*>(y), rows, c_out, k,
                         static_cast<int8_t*>(out), shift, s, lo);
  return kwta_dispatch(static_cast<const int32_t*>(y), rows, c_out, k, static_cast<int32_t*>(out),
                       0, s, lo);
}

int cs_mrs_kwta_units_conv2d(cs_dtype xt, const uint16_t* idx, const void* lval,
                             const int32_t* cnt, int cap, int b, int h, int w, int c_in, int kh,
                             int kw, int stride, int pad, const void* aug, int c_out, int n,
                             const void* bias, int pool, void* y, int keep_sums, int k, int unit,
                             void* out, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap,
                             void* stream) {
  if (unit == c_out)
    return cs_mrs_kwta_conv2d(xt, idx, lval, cnt, cap, b, h, w, c_in, kh, kw, stride, pad, aug,
                              c_out, n, bias, pool, y, keep_sums, k,
                              xt == CS_I8 ? CS_I32 : CS_F32, 0, out, oidx, oval, ocnt, ocap,
                              stream);
  if (xt != CS_F32) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (cap < 1 || unit < 1 || c_out % unit != 0) return CS_ERR_SHAPE;
  if (!idx || !lval || !cnt || !aug || !y) return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0) return CS_ERR_ARG;
  if (k > unit || unit > CS_MAX_KWTA_ROW) return CS_ERR_SHAPE;
  const bool lists = oidx != nullptr;
  if (lists == (out != nullptr)) return CS_ERR_ARG;        // exactly one output form
  if (lists && (!oval || !ocnt || ocap < 1)) return CS_ERR_ARG;
  const int kall = k * (c_out / unit);                      // winners per output pixel
  if (lists && ocap < kall) return CS_ERR_SHAPE;
  geo.cap = cap;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const cs::ListOut lo{oidx, oval, ocnt, lists ? ocap : 0};
  if (lists_vectorisable(xt, idx, lval, cap)) {
    BlocksPlan bp;
    const bool lvec = lists && aligned(oidx, 8) && aligned(oval, 16);
    int cus = 0;
    const int dst = device_cus(&cus);
    if (dst != CS_OK) return dst;
    if (blocks_plan(geo, xt, aug, y, out, k, keep_sums, lists ? ocap : 0, lvec, cus, &bp, unit))
      return launch_blocks(bp, s, idx, lval, cnt, aug, bias, y, out, lo, geo);
  }
  // two kernels: the sums into y, then k-WTA on the [rows * c_out / unit][unit]
  // view of y (dense output only)
  if (lists) return CS_ERR_SHAPE;
  st = mrs_launch(xt, idx, lval, cnt, geo, aug, bias, y, s);
  if (st != CS_OK) return st;
  const int64_t rows = (int64_t)b * (geo.Ho / pool) * (geo.Wo / pool) * (c_out / unit);
  return kwta_dispatch(static_cast<const float*>(y), rows, unit, k, static_cast<float*>(out), 0, s,
                       cs::ListOut{nullptr, nullptr, nullptr, 0});
}

int cs_mrs_plan(cs_dtype xt, int cap, int b, int h, int w, int c_in, int kh, int kw, int stride,
                int pad, int c_out, int n, int pool, int k, int64_t* info) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  if (!info) return CS_ERR_ARG;
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (cap < 1 || k < -1 || k > c_out) return CS_ERR_SHAPE;
  geo.cap = cap;
  for (int i = 0; i < 11; ++i) info[i] = 0;
  SamplePlan sp;
  if (sample_plan(geo, xt, k, 0, 1, &sp)) {
    info[0] = 3;
    info[6] = geo.B;
    info[7] = (int64_t)sp.shmem;
    info[8] = sp.sa.S;
    return CS_OK;
  }
  ScatterPlan scp;
  if (scatter_plan(geo, xt, nullptr, k, 0, 1, &scp)) {
    info[0] = 4;
    info[2] = scp.sc.BR;
    info[6] = scp.blocks;
    info[7] = (int64_t)scp.shmem;
    info[8] = scp.gpl;
    return CS_OK;
  }
  RowsPlan rp;
  if (rows_plan(geo, xt, nullptr, k, 0, 1, &rp)) {
    info[0] = 5;
    info[6] = rp.blocks;
    info[7] = (int64_t)rp.shmem;
    info[8] = rp.cpl;
    return CS_OK;
  }
  BlocksPlan bp;
  if (cap % 4 == 0 && blocks_plan(geo, xt, nullptr, nullptr, nullptr, k, 1,
                                  k >= 0 ? (k + 3) / 4 * 4 : 0, true, 0, &bp)) {
    info[1] = bp.ba.kmode;
    info[0] = 6;
    info[2] = bp.ba.RB;
    info[3] = bp.ba.nblocks;
    info[6] = bp.blocks;
    info[7] = (int64_t)bp.shmem;
    info[8] = bp.gb;
    return CS_OK;
  }
  FusedPlan fp;
  const int ocap = k >= 0 ? (k + 3) / 4 * 4 : 0;        // lists as the k-WTA emits them
  bool fused = cap % 4 == 0 && fused_plan(geo, xt, nullptr, nullptr, k, 0, 1,
                                          ocap < 4 ? 4 : ocap, xt == CS_I8 ? 1 : 4, &fp);
  if (!fused && k >= 0 && cap % 4 == 0) {
    // the sums in the fused kernel, k-WTA in its own kernel
    fused = fused_plan(geo, xt, nullptr, nullptr, -1, 0, 1, 0, 0, &fp);
    info[10] = 1;
  } else if (k >= 0 && !fused) {
    info[10] = 1;
  }
  if (fused) {
    info[0] = 2;
    info[1] = fp.fa.tile_mode;
    info[2] = fp.fa.tile_mode == 0 ? fp.fa.TI : fp.fa.TPR;
    info[3] = fp.fa.tile_mode == 0 ? 0 : fp.fa.TW;
    info[4] = fp.fa.list_cap;
    info[5] = fp.fa.npix_cap;
    info[6] = fp.blocks;
    info[7] = (int64_t)fp.shmem;
    info[8] = fp.fa.log2S;
    info[9] = fp.fa.kmode;
  } else {
    info[0] = cap % 4 == 0 ? 1 : 0;
  }
  return CS_OK;
}

int cs_conv2d(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
              int stride, int pad, const void* aug, int c_out, int n, const void* bias,
              int pool, void* y, void* ws, size_t ws_bytes, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (!x || !aug || !y) return CS_ERR_ARG;
  const int64_t rows = (int64_t)b * h * w;
  const WsLayout l = ws_layout(xt, rows, c_in);
  if (!ws || ws_bytes < l.total) return CS_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return CS_ERR_WORKSPACE;
  auto* base = static_cast<unsigned char*>(ws);
  auto* idx = reinterpret_cast<uint16_t*>(base + l.idx_off);
  void* lv = base + l.val_off;
  auto* cnt = reinterpret_cast<int32_t*>(base + l.cnt_off);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int r = compact_checked(xt, x, rows, c_in, idx, lv, cnt, s);
  if (r != CS_OK) return r;
  return mrs_launch(xt, idx, lv, cnt, geo, aug, bias, y, s);
}

int cs_conv2d_noalloc(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                      int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                      int pool, void* y, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (!x || !aug || !y) return CS_ERR_ARG;
  const int64_t rows = (int64_t)b * h * w;
  const WsLayout l = ws_layout(xt, rows, c_in);
  if (l.total > CS_NOALLOC_SCRATCH_BYTES) return CS_ERR_WORKSPACE;
  unsigned char* base = nullptr;
  const int sst = noalloc_scratch(&base);
  if (sst != CS_OK) return sst;
  auto* idx = reinterpret_cast<uint16_t*>(base + l.idx_off);
  void* lv = base + l.val_off;
  auto* cnt = reinterpret_cast<int32_t*>(base + l.cnt_off);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int r = compact_checked(xt, x, rows, c_in, idx, lv, cnt, s);
  if (r != CS_OK) return r;
  return mrs_launch(xt, idx, lv, cnt, geo, aug, bias, y, s);
}

int cs_conv2d_channels(const int8_t* x, int b, int h, int w, int c_in, int kh, int kw, int stride,
                       int pad, const int32_t* table, int c_out, int n, const int32_t* bias,
                       int32_t* y, void* stream) {
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, 1, 1, &geo);
  if (st != CS_OK) return st;
  if (!x || !table || !y || n < 1) return CS_ERR_ARG;
  if (n > CS_MAX_N || c_in % n != 0 || c_in % 4 != 0) return CS_ERR_SHAPE;
  if (c_out != 16 && c_out != 32 && c_out != 64 && c_out != 128) return CS_ERR_SHAPE;
  if (!aligned(x, 4) || !aligned(y, 16)) return CS_ERR_ARG;
  cs::ChannelArgs ca;
  ca.S4 = ((c_in / n) * kh * kw + 3) / 4;
  ca.SW = 63 * stride + kw;
  ca.CP = (c_in / 4) % 2 == 1 ? c_in : c_in + 4;
  const size_t shmem = round16((size_t)kh * ca.SW * ca.CP);
  if (shmem > kBlockLds) return CS_ERR_SHAPE;
  ca.nseg = (geo.Wo + cs::CH_P - 1) / cs::CH_P;
  const int64_t ntiles = (int64_t)b * geo.Ho * ca.nseg;
  if (ntiles >= INT32_MAX || (int64_t)b * h * w * c_in >= ((int64_t)1 << 40)) return CS_ERR_SHAPE;
  ca.ntiles = (int)ntiles;
  ca.fd_nseg = cs::make_fastdiv((uint32_t)ca.nseg);
  ca.fd_ho = cs::make_fastdiv((uint32_t)geo.Ho);
  int cus = 0;
  const int dst = device_cus(&cus);
  if (dst != CS_OK) return dst;
  int64_t per_cu = lds_wgs_per_cu(shmem);
  if (per_cu > 8) per_cu = 8;
  const int64_t nb = ntiles < per_cu * cus ? ntiles : per_cu * cus;
  const hipStream_t s = static_cast<hipStream_t>(stream);
#define CS_CH(FW_)                                                                        \
  hipLaunchKernelGGL((cs::conv_channels_i8<FW_>), dim3((unsigned)nb), dim3(cs::CH_BD), shmem, s, \
                     x, table, bias, y, geo, ca)
  if (c_out == 16) CS_CH(4);
  else if (c_out == 32) CS_CH(8);
  else if (c_out == 64) CS_CH(16);
  else CS_CH(32);
#undef CS_CH
  return launch_status();
}

int cs_conv2d_dense_blocks(const int8_t* x, int b, int h, int w, int c_in, int kh, int kw,
                           int stride, int pad, const uint16_t* aug, const uint8_t* kidb,
                           int c_out, int n, const int32_t* bias, int32_t* y, void* stream) {
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, 1, &geo);
  if (st != CS_OK) return st;
  if (!x || !aug || !kidb || !y) return CS_ERR_ARG;
  if (c_in > 4) return CS_ERR_SHAPE;                       // a block is one v_dot4
  const int G = c_out / n;
  const int GB = G % 2 == 0 ? 2 : 1;
  const int U = G / GB;
  if (U > cs::DB_BD) return CS_ERR_SHAPE;
  const int P = cs::DB_BD / U;
  const int64_t items64 = (int64_t)b * geo.Ho * geo.Wo;
  if (items64 * c_out >= ((int64_t)1 << 40) || items64 >= INT32_MAX ||
      (int64_t)b * h >= INT32_MAX)
    return CS_ERR_SHAPE;
  cs::DenseBlocksArgs da;
  da.GB = GB;
  da.U = U;
  da.P = P;
  da.nseg = (geo.Wo + P - 1) / P;
  const int64_t ntiles = (int64_t)b * geo.Ho * da.nseg;
  if (ntiles >= INT32_MAX) return CS_ERR_SHAPE;
  da.ntiles = (int)ntiles;
  da.SW = (P - 1) * stride + kw;
  if ((int64_t)kh * da.SW > (int64_t)cs::DB_PRE * cs::DB_BD) return CS_ERR_SHAPE;
  const size_t acc_b = (size_t)GB * n * cs::DB_BD * 4;
  const size_t xs_b = round16((size_t)kh * da.SW * 4);
  const bool pk = c_in <= 3;                                // one-word table entries
  const size_t tab_b = (size_t)kh * kw * G * (pk ? 4 : 8);
  da.off_x = (uint32_t)acc_b;
  da.off_t = (uint32_t)(acc_b + xs_b);
  const size_t shmem = acc_b + xs_b + tab_b;
  if (shmem > kBlockLds) return CS_ERR_SHAPE;
  da.fd_nseg = cs::make_fastdiv((uint32_t)da.nseg);
  da.fd_ho = cs::make_fastdiv((uint32_t)geo.Ho);
  da.fd_sw = cs::make_fastdiv((uint32_t)da.SW);
  // persistent: as many workgroups as fit at once (LDS and 32 wavefronts per CU)
  int cus = 0;
  const int dst = device_cus(&cus);
  if (dst != CS_OK) return dst;
  int64_t per_cu = lds_wgs_per_cu(shmem);
  if (per_cu > 8) per_cu = 8;
  if (per_cu < 1) per_cu = 1;
  const int64_t nb = ntiles < per_cu * cus ? ntiles : per_cu * cus;
  const hipStream_t s = static_cast<hipStream_t>(stream);
#define CS_DB3(KW_, GB_, PK_)                                                               \
  hipLaunchKernelGGL((cs::conv_dense_blocks<KW_, GB_, PK_>), dim3((unsigned)nb),             \
                     dim3(cs::DB_BD), shmem, s, x, aug, kidb, bias, y, geo, da)
#define CS_DB(KW_, GB_)         \
  do {                          \
    if (pk) CS_DB3(KW_, GB_, true); \
    else CS_DB3(KW_, GB_, false);   \
  } while (0)
  if (GB == 2) {
    if (kw == 7) CS_DB(7, 2);
    else if (kw == 5) CS_DB(5, 2);
    else if (kw == 3) CS_DB(3, 2);
    else CS_DB(0, 2);
  } else {
    if (kw == 7) CS_DB(7, 1);
    else if (kw == 5) CS_DB(5, 1);
    else if (kw == 3) CS_DB(3, 1);
    else CS_DB(0, 1);
  }
#undef CS_DB
#undef CS_DB3
  return launch_status();
}

int cs_conv2d_dense(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                    int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                    int pool, void* y, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  const int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (!x || !aug || !y) return CS_ERR_ARG;
  const int R = kh * kw * c_in;
  const int ph = (pool - 1) * stride + kh, pw = (pool - 1) * stride + kw;
  if (n != 1 || c_out != 64 || R > 32 || (int64_t)ph * pw * c_in > 64) return CS_ERR_SHAPE;
  const int64_t items64 = (int64_t)b * (geo.Ho / pool) * (geo.Wo / pool);
  if (items64 * 64 >= INT32_MAX || (int64_t)b * h * w * c_in >= INT32_MAX) return CS_ERR_SHAPE;
  const int items = (int)items64;
  const cs::FastDiv fd_wp = cs::make_fastdiv((uint32_t)(geo.Wo / pool));
  const cs::FastDiv fd_hp = cs::make_fastdiv((uint32_t)(geo.Ho / pool));
  int cus = 0;
  const int dst = device_cus(&cus);
  if (dst != CS_OK) return dst;
  const int64_t nb64 = (items64 + 3) / 4;                  // 4 wavefronts per block
  const int64_t cap = (int64_t)cus * 8;                    // persistent: 32 wavefronts per CU
  const int nb = (int)(nb64 < cap ? nb64 : cap);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const bool gsc = kh == 5 && kw == 5 && c_in == 1 && stride == 1 && pool == 2;
  if (xt == CS_I8) {
    auto* xx = static_cast<const int8_t*>(x);
    auto* pv = static_cast<const uint16_t*>(aug);
    auto* bs = static_cast<const int32_t*>(bias);
    auto* yy = static_cast<int32_t*>(y);
    if (gsc)
      hipLaunchKernelGGL((cs::conv_dense_n1<int8_t, int32_t, 5, 5, 1, 1, 2>), dim3(nb), dim3(256),
                         0, s, xx, pv, bs, yy, geo, items, fd_wp, fd_hp);
    else
      hipLaunchKernelGGL((cs::conv_dense_n1_rt<int8_t, int32_t>), dim3(nb), dim3(256), 0, s, xx,
                         pv, bs, yy, geo, items, fd_wp, fd_hp);
  } else {
    auto* xx = static_cast<const float*>(x);
    auto* pv = static_cast<const uint2*>(aug);
    auto* bs = static_cast<const float*>(bias);
    auto* yy = static_cast<float*>(y);
    if (gsc)
      hipLaunchKernelGGL((cs::conv_dense_n1<float, float, 5, 5, 1, 1, 2>), dim3(nb), dim3(256), 0,
                         s, xx, pv, bs, yy, geo, items, fd_wp, fd_hp);
    else
      hipLaunchKernelGGL((cs::conv_dense_n1_rt<float, float>), dim3(nb), dim3(256), 0, s, xx, pv,
                         bs, yy, geo, items, fd_wp, fd_hp);
  }
  return launch_status();
}

// LDS layout and arguments of the first-layer matrix-core kernel for
// workgroups of tpr pooled rows (fewer while the layout exceeds budget); the
// layer is int8, n == 1, c_out == 64, kh*kw*c_in <= 32, k <= 32 (checked by
// the callers).  ocap: list capacity, 0 for dense output.
bool dense_plan(const cs::ConvGeom& geo, const void* x, int w, int pad, int k, int shift,
                int keep_sums, int ocap, int osz, int tpr, size_t budget, cs::DenseArgs* pda,
                size_t* shmem) {
  const int pool = geo.pool, Hp = geo.Ho / pool, Wp = geo.Wo / pool;
  const int c_in = geo.C, kh = geo.KH, kw = geo.KW, stride = geo.S;
  const bool lists = ocap > 0;
  cs::DenseArgs& da = *pda;
  da = cs::DenseArgs{};
  for (; tpr >= 1; --tpr) {
    const int rows_in = (tpr * pool - 1) * stride + kh;
    const size_t items_t = (size_t)tpr * Wp;
    size_t o = round16((size_t)rows_in * (w + 2 * pad) * c_in);   // zero-padded rows
    da.off_w = (uint32_t)o;
    o += 64 * 32 + 32 * 4;                              // weights [64][32] bytes, slot offsets
    da.off_out = (uint32_t)o;
    o += round16(items_t * 65 * 4);
    da.off_sel = (uint32_t)o;
    o += round16(items_t * 8);
    da.off_lidx = (uint32_t)o;
    o += lists ? round16(items_t * ocap * 2) : 0;
    da.off_lval = (uint32_t)o;
    o += lists ? round16(items_t * ocap * osz) : 0;
    if (o <= budget) {
      *shmem = o;
      break;
    }
  }
  if (tpr < 1) return false;
  da.TPR = tpr;
  da.tiles_img = (Hp + tpr - 1) / tpr;
  da.R = kh * kw * c_in;
  da.k = k;
  da.shift = shift;
  da.kmode = k <= 8 ? 1 : (k <= 16 ? 2 : 3);
  da.write_sums = keep_sums;
  da.ostride = 65;
  da.fd_wp = cs::make_fastdiv((uint32_t)Wp);
  da.fd_timg = cs::make_fastdiv((uint32_t)da.tiles_img);
  da.fd_cout = cs::make_fastdiv(64u);
  da.fd_ochunks = cs::make_fastdiv((uint32_t)(lists ? ocap / 4 : 1));
  da.fd_rowb = cs::make_fastdiv((uint32_t)((w + 2 * pad) * c_in));
  da.vec_rows = pad == 0 && (w * c_in) % 16 == 0 && aligned(x, 16) ? 1 : 0;
  da.fd_c = cs::make_fastdiv((uint32_t)c_in);
  da.fd_kw = cs::make_fastdiv((uint32_t)kw);
  return true;
}

int cs_conv2d_dense_kwta(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw,
                         int stride, int pad, const void* aug, int c_out, int n, const void* bias,
                         int pool, void* y, int keep_sums, int k, cs_dtype ot, int shift, void* out,
                         uint16_t* oidx, void* oval, int32_t* ocnt, int ocap, void* stream) {
  if (!is_act_dtype(xt)) return CS_ERR_DTYPE;
  const cs_dtype at = xt == CS_I8 ? CS_I32 : CS_F32;
  if (!(ot == at || (xt == CS_I8 && ot == CS_I8))) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (!x || !aug || !y) return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0 || shift < 0 || shift > 31) return CS_ERR_ARG;
  if (k > c_out || c_out > CS_MAX_KWTA_ROW) return CS_ERR_SHAPE;
  const bool lists = oidx != nullptr;
  if (lists == (out != nullptr)) return CS_ERR_ARG;
  if (lists && (!oval || !ocnt || ocap < 1)) return CS_ERR_ARG;
  if (lists && ocap < k) return CS_ERR_SHAPE;
  const int R = kh * kw * c_in;
  if (n != 1 || c_out != 64 || R > 32) return CS_ERR_SHAPE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int osz = ot == CS_I8 ? 1 : 4;
  const cs::ListOut lo{oidx, oval, ocnt, lists ? ocap : 0};
  const int Hp = geo.Ho / pool, Wp = geo.Wo / pool;
  const int64_t items = (int64_t)b * Hp * Wp;
  const bool lists_ok = !lists || (ocap % 4 == 0 && aligned(oidx, 8) && aligned(oval, osz * 4));
  if (xt == CS_I8 && k <= 32 && lists_ok && aligned(aug, 16) && items * 64 < INT32_MAX) {
    // matrix-core kernel: pooled rows per workgroup for about 512 workgroups
    int tiles = (int)((512 + b - 1) / b);
    tiles = tiles < 1 ? 1 : (tiles > Hp ? Hp : tiles);
    cs::DenseArgs da{};
    size_t shmem = 0;
    if (dense_plan(geo, x, w, pad, k, shift, keep_sums, lists ? ocap : 0, osz,
                   (Hp + tiles - 1) / tiles, kFusedLds, &da, &shmem)) {
      const int64_t nb = (int64_t)b * da.tiles_img;
      if (nb < INT32_MAX) {
        const dim3 grid((unsigned)nb), block(cs::DENSE_BD);
        const auto* xx = static_cast<const int8_t*>(x);
        const auto* pa = static_cast<const uint16_t*>(aug);
        const auto* bs = static_cast<const int32_t*>(bias);
        auto* yy = static_cast<int32_t*>(y);
        if (pool == 2) {
          if (ot == CS_I8)
            hipLaunchKernelGGL((cs::conv_dense_mfma<2, int8_t>), grid, block, shmem, s, xx, pa, bs,
                               yy, static_cast<int8_t*>(out), lo, geo, da);
          else
            hipLaunchKernelGGL((cs::conv_dense_mfma<2, int32_t>), grid, block, shmem, s, xx, pa,
                               bs, yy, static_cast<int32_t*>(out), lo, geo, da);
        } else {
          if (ot == CS_I8)
            hipLaunchKernelGGL((cs::conv_dense_mfma<1, int8_t>), grid, block, shmem, s, xx, pa, bs,
                               yy, static_cast<int8_t*>(out), lo, geo, da);
          else
            hipLaunchKernelGGL((cs::conv_dense_mfma<1, int32_t>), grid, block, shmem, s, xx, pa,
                               bs, yy, static_cast<int32_t*>(out), lo, geo, da);
        }
        return launch_status();
      }
    }
  }
  // two kernels: the sums into y (pooled window of at most 64 values), then k-WTA from y
  st = cs_conv2d_dense(xt, x, b, h, w, c_in, kh, kw, stride, pad, aug, c_out, n, bias, pool, y,
                       stream);
  if (st != CS_OK) return st;
  if (xt == CS_F32)
    return kwta_dispatch(static_cast<const float*>(y), items, c_out, k, static_cast<float*>(out),
                         0, s, lo);
  if (ot == CS_I8)
    return kwta_dispatch(static_cast<const int32_t*>(y), items, c_out, k,
                         static_cast<int8_t*>(out), shift, s, lo);
  return kwta_dispatch(static_cast<const int32_t*>(y), items, c_out, k, static_cast<int32_t*>(out),
                       0, s, lo);
}

int cs_linear(cs_dtype xt, const void* x, int batch, int d_in, const void* aug, int d_out, int n,
              const void* bias, void* y, void* ws, size_t ws_bytes, void* stream) {
  return cs_conv2d(xt, x, batch, 1, 1, d_in, 1, 1, 1, 0, aug, d_out, n, bias, 1, y, ws, ws_bytes,
                   stream);
}

int cs_kwta(cs_dtype it, const void* in, int64_t rows, int c, int k, cs_dtype ot, int shift,
            void* out, void* stream) {
  if (it != CS_I32 && it != CS_F32) return CS_ERR_DTYPE;
  if (!(ot == it || (it == CS_I32 && ot == CS_I8))) return CS_ERR_DTYPE;
  if (rows < 0 || c < 1 || k < 0) return CS_ERR_ARG;
  if (k > c || c > CS_MAX_KWTA_ROW) return CS_ERR_SHAPE;
  if (shift < 0 || shift > 31) return CS_ERR_ARG;
  if (rows > 0 && (!in || !out)) return CS_ERR_ARG;
  if (rows == 0) return CS_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (it == CS_F32)
    return kwta_dispatch(static_cast<const float*>(in), rows, c, k, static_cast<float*>(out), 0,
                         s);
  if (ot == CS_I8)
    return kwta_dispatch(static_cast<const int32_t*>(in), rows, c, k, static_cast<int8_t*>(out),
                         shift, s);
  return kwta_dispatch(static_cast<const int32_t*>(in), rows, c, k, static_cast<int32_t*>(out), 0,
                       s);
}

int cs_kwta_lists(cs_dtype it, const void* in, int64_t rows, int c, int k, cs_dtype ot, int shift,
                  uint16_t* idx, void* val, int32_t* cnt, int cap, void* stream) {
  if (it != CS_I32 && it != CS_F32) return CS_ERR_DTYPE;
  if (!(ot == it || (it == CS_I32 && ot == CS_I8))) return CS_ERR_DTYPE;
  if (rows < 0 || c < 1 || k < 0 || cap < 1) return CS_ERR_ARG;
  if (k > c || c > CS_MAX_KWTA_ROW || cap < k) return CS_ERR_SHAPE;
  if (shift < 0 || shift > 31) return CS_ERR_ARG;
  if (rows > 0 && (!in || !idx || !val || !cnt)) return CS_ERR_ARG;
  if (rows == 0) return CS_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const cs::ListOut lo{idx, val, cnt, cap};
  if (it == CS_F32)
    return kwta_dispatch(static_cast<const float*>(in), rows, c, k, static_cast<float*>(nullptr),
                         0, s, lo);
  if (ot == CS_I8)
    return kwta_dispatch(static_cast<const int32_t*>(in), rows, c, k,
                         static_cast<int8_t*>(nullptr), shift, s, lo);
  return kwta_dispatch(static_cast<const int32_t*>(in), rows, c, k, static_cast<int32_t*>(nullptr),
                       0, s, lo);
}

size_t cs_workspace_bytes(int op, cs_dtype xt, int64_t rows, int c_in) {
  if ((op != 0 && op != 1) || !is_act_dtype(xt) || rows < 0 || c_in < 1 || c_in > CS_MAX_ROW)
    return 0;
  return ws_layout(xt, rows, c_in).total;
}

}  // extern "C"

int cs_conv2d_reorder_kwta(cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh,
                           int kw, int pad, const int32_t* table, int smax, int c_out,
                           const void* bias, void* y, int keep_sums, int k, cs_dtype ot,
                           void* out, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap,
                           void* stream) {
  if (xt != CS_F32 || ot != CS_F32) return CS_ERR_DTYPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, 1, pad, c_out, 1, 1, &geo);
  if (st != CS_OK) return st;
  if (!x || !table || !y || smax < 1) return CS_ERR_ARG;
  if (smax % 8 != 0) return CS_ERR_SHAPE;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0) return CS_ERR_ARG;
  if (c_out != cs::RO_COUT || c_in > 64 || k > c_out || (k > 32 && k != c_out)) return CS_ERR_SHAPE;
  const bool lists = oidx != nullptr;
  if (lists == (out != nullptr)) return CS_ERR_ARG;
  if (lists && (!oval || !ocnt || ocap < 1)) return CS_ERR_ARG;
  if (lists && (ocap < k || ocap % 4 != 0 || !aligned(oidx, 8) || !aligned(oval, 16)))
    return CS_ERR_SHAPE;
  if (!aligned(y, 16) || !aligned(out, 16)) return CS_ERR_ARG;
  const int tiles_w = (geo.Wo + cs::RO_T - 1) / cs::RO_T, tiles_h = (geo.Ho + cs::RO_T - 1) / cs::RO_T;
  const int64_t nb = (int64_t)b * tiles_w * tiles_h;
  if (nb >= INT32_MAX || (int64_t)smax * c_out * 2 >= INT32_MAX) return CS_ERR_SHAPE;
  // the input tile, reused afterwards for the per-lane list staging
  const size_t halo = (size_t)(cs::RO_T + kh - 1) * (cs::RO_T + kw - 1) * (c_in + 1) * 4;
  const size_t stage = lists ? (size_t)64 * ocap * 6 : 0;
  const size_t shmem = round16(std::max(halo, stage));
  if (shmem > kCuLds) return CS_ERR_SHAPE;
  cs::ReorderArgs ra{};
  ra.smax = smax;
  ra.tiles_w = tiles_w;
  ra.tiles_img = tiles_w * tiles_h;
  ra.k = k;
  ra.write_sums = keep_sums;
  ra.vec4 = (c_in % 4 == 0 && aligned(x, 16)) ? 1 : 0;
  ra.fd_cq = cs::make_fastdiv((uint32_t)(ra.vec4 ? c_in / 4 : c_in));
  ra.fd_hw = cs::make_fastdiv((uint32_t)(cs::RO_T + kw - 1));
  const cs::ListOut lo{oidx, oval, ocnt, lists ? ocap : 0};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3((unsigned)nb), dim3(64), shmem, s, static_cast<const float*>(x),
                       reinterpret_cast<const int2*>(table), static_cast<const float*>(bias),
                       static_cast<float*>(y), static_cast<float*>(out), lo, geo, ra);
  };
  if (k <= 8)
    go(cs::conv_reorder_f32<8>);
  else if (k <= 16)
    go(cs::conv_reorder_f32<16>);
  else
    go(cs::conv_reorder_f32<32>);
  return launch_status();
}

int cs_mrs_kwta_chain2(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, uint16_t* oidx, void* oval,
                       int32_t* ocnt, int ocap, const void* aug2, int c_out2, int n2,
                       const void* bias2, void* y2, void* stream) {
  if (xt != CS_I8 || ot != CS_I8) return CS_ERR_DTYPE;
  if (!aug2 || !y2 || !oidx) return CS_ERR_ARG;
  if (c_out2 < 1 || n2 < 1) return CS_ERR_ARG;
  if (n2 > CS_MAX_N || c_out2 % n2 != 0) return CS_ERR_SHAPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  // the first layer as cs_mrs_kwta_conv2d checks it, the second as a linear
  // layer over the first one's output vector (one per sample when the first
  // layer's map is 1 x 1)
  const bool vec = geo.Ho / pool == 1 && geo.Wo / pool == 1;
  if (!vec) return CS_ERR_SHAPE;
  if (cap < 1) return CS_ERR_SHAPE;
  if (!idx || !lval || !cnt || !aug || !y || !oval || !ocnt || ocap < 1) return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0 || shift < 0 || shift > 31) return CS_ERR_ARG;
  if (k > c_out || c_out > CS_MAX_KWTA_ROW || ocap < k) return CS_ERR_SHAPE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  geo.cap = cap;
  SamplePlan sp;
  if (sample_plan(geo, xt, k, shift, keep_sums, &sp)) {
    // one kernel: the first layer's winners feed the second layer in LDS
    cs::NextLayer nx{static_cast<const uint16_t*>(aug2), static_cast<const int32_t*>(bias2),
                     static_cast<int32_t*>(y2), c_out2 / n2, n2, c_out2,
                     (uint32_t)round16(sp.shmem)};
    if ((size_t)nx.off_acc + round16((size_t)c_out2 * 4) <= kCuLds) {
      const cs::ListOut lo{oidx, oval, ocnt, ocap};
      return launch_sample(sp, xt, ot, s, idx, lval, cnt, aug, bias, y, nullptr, lo, geo, nx);
    }
  }
  // two launches: the layer with its lists, then the linear layer on them
  st = cs_mrs_kwta_conv2d(xt, idx, lval, cnt, cap, b, h, w, c_in, kh, kw, stride, pad, aug, c_out,
                          n, bias, pool, y, keep_sums, k, ot, shift, nullptr, oidx, oval, ocnt,
                          ocap, stream);
  if (st != CS_OK) return st;
  return cs_mrs_conv2d(CS_I8, oidx, oval, ocnt, ocap, b, 1, 1, c_out, 1, 1, 1, 0, aug2, c_out2, n2,
                       bias2, 1, y2, stream);
}

template <int KW, int GPL, int M>
void launch_scatter_sample_t(const ScatterPlan& scp, const SamplePlan& sp, size_t shmem,
                             hipStream_t s, const uint16_t* idx, const void* lval,
                             const int32_t* cnt, const void* aug, const void* bias, void* y,
                             const cs::ListOut& lo, const cs::ConvGeom& geo, const void* aug2,
                             const void* bias2, void* y2, const cs::ListOut& lo2,
                             const cs::ConvGeom& geo2, const cs::NextLayer& nx) {
  hipLaunchKernelGGL((cs::mrs_scatter_sample<KW, GPL, M>), dim3((unsigned)scp.blocks),
                     dim3(cs::SCAT_BD), shmem, s, idx, static_cast<const int8_t*>(lval), cnt,
                     static_cast<const uint16_t*>(aug), static_cast<const int32_t*>(bias),
                     static_cast<int32_t*>(y), lo, geo, scp.sc,
                     static_cast<const uint16_t*>(aug2), static_cast<const int32_t*>(bias2),
                     static_cast<int32_t*>(y2), lo2, geo2, sp.sa, nx);
}

template <int KW>
void launch_scatter_sample_kw(const ScatterPlan& scp, const SamplePlan& sp, size_t shmem,
                              hipStream_t s, const uint16_t* idx, const void* lval,
                              const int32_t* cnt, const void* aug, const void* bias, void* y,
                              const cs::ListOut& lo, const cs::ConvGeom& geo, const void* aug2,
                              const void* bias2, void* y2, const cs::ListOut& lo2,
                              const cs::ConvGeom& geo2, const cs::NextLayer& nx) {
#define CS_SCS(GPL_, M_)                                                                       \
  launch_scatter_sample_t<KW, GPL_, M_>(scp, sp, shmem, s, idx, lval, cnt, aug, bias, y, lo, geo, \
                                        aug2, bias2, y2, lo2, geo2, nx)
  if (scp.gpl == 2) {
    if (scp.m == 1) CS_SCS(2, 1);
    else CS_SCS(2, 2);
  } else {
    if (scp.m == 1) CS_SCS(1, 1);
    else CS_SCS(1, 2);
  }
#undef CS_SCS
}

int cs_mrs_kwta_chain3(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
                       int cap, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
                       const void* aug, int c_out, int n, const void* bias, int pool, void* y,
                       int keep_sums, int k, cs_dtype ot, int shift, uint16_t* oidx, void* oval,
                       int32_t* ocnt, int ocap, const void* aug2, int c_out2, int n2,
                       const void* bias2, void* y2, int k2, int shift2, uint16_t* oidx2,
                       void* oval2, int32_t* ocnt2, int ocap2, const void* aug3, int c_out3,
                       int n3, const void* bias3, void* y3, void* stream) {
  if (xt != CS_I8 || ot != CS_I8) return CS_ERR_DTYPE;
  if (!idx || !lval || !cnt || !aug || !y || !oidx || !oval || !ocnt) return CS_ERR_ARG;
  if (!aug2 || !y2 || !oidx2 || !oval2 || !ocnt2 || !aug3 || !y3) return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0 || shift < 0 || shift > 31 || k2 < 0 ||
      shift2 < 0 || shift2 > 31)
    return CS_ERR_ARG;
  if (cap < 1 || ocap < 1 || ocap2 < 1 || c_out2 < 1 || n2 < 1 || c_out3 < 1 || n3 < 1)
    return CS_ERR_SHAPE;
  cs::ConvGeom geo;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo);
  if (st != CS_OK) return st;
  if (k > c_out || c_out > CS_MAX_KWTA_ROW || ocap < k) return CS_ERR_SHAPE;
  // the second layer: a window over the whole pooled map of the first
  const int hp = geo.Ho / pool, wp = geo.Wo / pool;
  cs::ConvGeom geo2;
  st = conv_geometry(b, hp, wp, c_out, hp, wp, 1, 0, c_out2, n2, 1, &geo2);
  if (st != CS_OK) return st;
  if (k2 > c_out2 || c_out2 > CS_MAX_KWTA_ROW || ocap2 < k2) return CS_ERR_SHAPE;
  if (n3 > CS_MAX_N || c_out3 % n3 != 0) return CS_ERR_SHAPE;
  geo.cap = cap;
  geo2.cap = ocap;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // one kernel when the first layer runs one workgroup per image (its band
  // is the whole image) and the second one workgroup per sample
  ScatterPlan scp;
  SamplePlan sp;
  if (!sample_plan(geo, xt, k, shift, keep_sums, &sp) &&
      scatter_plan(geo, xt, aug, k, shift, keep_sums, &scp) && scp.sc.bands == 1 &&
      scp.blocks == b && sample_plan(geo2, xt, k2, shift2, keep_sums, &sp)) {
    const cs::NextLayer nx{static_cast<const uint16_t*>(aug3), static_cast<const int32_t*>(bias3),
                           static_cast<int32_t*>(y3), c_out3 / n3, n3, c_out3,
                           (uint32_t)round16(sp.shmem)};
    const size_t shmem2 = (size_t)nx.off_acc + round16((size_t)c_out3 * 4);
    const size_t shmem = std::max(scp.shmem, shmem2);
    if (shmem <= kCuLds) {
      const cs::ListOut lo{oidx, oval, ocnt, ocap};
      const cs::ListOut lo2{oidx2, oval2, ocnt2, ocap2};
      switch (geo.KW) {
        case 3:
          launch_scatter_sample_kw<3>(scp, sp, shmem, s, idx, lval, cnt, aug, bias, y, lo, geo,
                                      aug2, bias2, y2, lo2, geo2, nx);
          break;
        case 5:
          launch_scatter_sample_kw<5>(scp, sp, shmem, s, idx, lval, cnt, aug, bias, y, lo, geo,
                                      aug2, bias2, y2, lo2, geo2, nx);
          break;
        default:
          launch_scatter_sample_kw<7>(scp, sp, shmem, s, idx, lval, cnt, aug, bias, y, lo, geo,
                                      aug2, bias2, y2, lo2, geo2, nx);
          break;
      }
      return launch_status();
    }
  }
  // otherwise: the first layer, then the two-layer tail on its lists
  st = cs_mrs_kwta_conv2d(xt, idx, lval, cnt, cap, b, h, w, c_in, kh, kw, stride, pad, aug, c_out,
                          n, bias, pool, y, keep_sums, k, ot, shift, nullptr, oidx, oval, ocnt,
                          ocap, stream);
  if (st != CS_OK) return st;
  return cs_mrs_kwta_chain2(xt, oidx, oval, ocnt, ocap, b, hp, wp, c_out, hp, wp, 1, 0, aug2,
                            c_out2, n2, bias2, 1, y2, keep_sums, k2, ot, shift2, oidx2, oval2,
                            ocnt2, ocap2, aug3, c_out3, n3, bias3, y3, stream);
}

// The output-stationary second layer of the dense chain: 64 input channels
// with eight list slots each, a square 3x3 or 5x5 window at stride 1, four
// sets (c_out = 4n <= 64), the whole output map in LDS as blocks of 64
// pixels, one wavefront per (tap row, block).
struct GatherPlan {
  cs::GatherArgs ga;
  size_t shmem;
};

bool gather_plan(const cs::ConvGeom& geo, const void* aug, int k, int shift, int write_sums,
                 GatherPlan* pl) {
  if (geo.C != cs::GATH_C || geo.cap != cs::GATH_CAP || geo.S != 1 || geo.KH != geo.KW) return false;
  if ((geo.KW != 3 && geo.KW != 5) || geo.G != 4 || geo.c_out > 64 || !aligned(aug, 16)) return false;
  if (geo.pool != 1 && geo.pool != 2) return false;
  const int64_t npix = (int64_t)geo.H * geo.W;
  const int64_t nout = (int64_t)geo.Ho * geo.Wo;
  if (npix < 1 || npix > cs::GATH_BD || nout < 1) return false;
  const int NH = (int)((nout + 63) / 64);
  if (geo.KW * NH > cs::GATH_BD / 64) return false;
  const int nitems = (geo.Ho / geo.pool) * (geo.Wo / geo.pool);
  if (nitems < 1) return false;
  const size_t o_tab = (size_t)NH * cs::GATH_BLK_B;
  const size_t o_ent = o_tab + (size_t)(geo.G / 2) * geo.KW * geo.KW * cs::GATH_C * 4;
  const size_t o_cnt = o_ent + (size_t)npix * cs::GATH_CAP * 2;
  const size_t o_bias = o_cnt + round16((size_t)npix * 4);
  const size_t o_pt = o_bias + round16((size_t)geo.c_out * 4);
  const size_t total = o_pt + round16((size_t)nitems * (geo.c_out + 1) * 4);
  if (total > kCuLds) return false;
  cs::GatherArgs& ga = pl->ga;
  ga.NH = NH;
  ga.nitems = nitems;
  ga.k = k;
  ga.shift = shift;
  ga.write_sums = write_sums;
  ga.off_tab = (uint32_t)o_tab;
  ga.off_ent = (uint32_t)o_ent;
  ga.off_cnt = (uint32_t)o_cnt;
  ga.off_bias = (uint32_t)o_bias;
  ga.off_pt = (uint32_t)o_pt;
  ga.fd_wo = cs::make_fastdiv((uint32_t)geo.Wo);
  ga.fd_wp = cs::make_fastdiv((uint32_t)(geo.Wo / geo.pool));
  ga.fd_items = cs::make_fastdiv((uint32_t)nitems);
  pl->shmem = total;
  return true;
}

template <int POOL, int KW, int KM, bool GA>
void launch_dense_chain(const cs::DenseArgs& da, const ScatterPlan& scp, const GatherPlan& gp,
                        const SamplePlan& sp,
                        size_t shmem, hipStream_t s, const void* x, const void* aug0,
                        const void* bias0, void* y0, const cs::ListOut& lo0,
                        const cs::ConvGeom& geo0, const void* aug, const void* bias, void* y,
                        const cs::ListOut& lo, const cs::ConvGeom& geo, const void* aug2,
                        const void* bias2, void* y2, const cs::ListOut& lo2,
                        const cs::ConvGeom& geo2, const cs::NextLayer& nx) {
  const cs::ChainArgs a{static_cast<const int8_t*>(x),
                        static_cast<const uint16_t*>(aug0),
                        static_cast<const int32_t*>(bias0),
                        static_cast<int32_t*>(y0),
                        lo0,
                        geo0,
                        da,
                        static_cast<const uint16_t*>(aug),
                        static_cast<const int32_t*>(bias),
                        static_cast<int32_t*>(y),
                        lo,
                        geo,
                        scp.sc,
                        gp.ga,
                        static_cast<const uint16_t*>(aug2),
                        static_cast<const int32_t*>(bias2),
                        static_cast<int32_t*>(y2),
                        lo2,
                        geo2,
                        sp.sa,
                        nx};
  if constexpr (GA)
    hipLaunchKernelGGL((cs::dense_gather_sample<POOL, KW, KM>), dim3((unsigned)geo0.B),
                       dim3(cs::GATH_BD), shmem, s, a);
  else
    hipLaunchKernelGGL((cs::dense_scatter_sample<POOL, KW, KM>), dim3((unsigned)geo0.B),
                       dim3(cs::SCAT_BD), shmem, s, a);
}

int cs_conv2d_dense_kwta_chain3(
    cs_dtype xt, const void* x, int b, int h, int w, int c_in, int kh, int kw, int stride, int pad,
    const void* aug, int c_out, int n, const void* bias, int pool, void* y, int keep_sums, int k,
    cs_dtype ot, int shift, uint16_t* oidx, void* oval, int32_t* ocnt, int ocap, int kh2, int kw2,
    int stride2, int pad2, const void* aug2, int c_out2, int n2, const void* bias2, int pool2,
    void* y2, int k2, int shift2, uint16_t* oidx2, void* oval2, int32_t* ocnt2, int ocap2,
    const void* aug3, int c_out3, int n3, const void* bias3, void* y3, int k3, int shift3,
    uint16_t* oidx3, void* oval3, int32_t* ocnt3, int ocap3, const void* aug4, int c_out4, int n4,
    const void* bias4, void* y4, void* stream) {
  if (xt != CS_I8 || ot != CS_I8) return CS_ERR_DTYPE;
  if (!x || !aug || !y || !oidx || !oval || !ocnt) return CS_ERR_ARG;
  if (!aug2 || !y2 || !oidx2 || !oval2 || !ocnt2 || !aug3 || !y3 || !oidx3 || !oval3 || !ocnt3 ||
      !aug4 || !y4)
    return CS_ERR_ARG;
  if ((keep_sums != 0 && keep_sums != 1) || k < 0 || shift < 0 || shift > 31 || k2 < 0 ||
      shift2 < 0 || shift2 > 31 || k3 < 0 || shift3 < 0 || shift3 > 31)
    return CS_ERR_ARG;
  if (ocap < 1 || ocap2 < 1 || ocap3 < 1 || c_out2 < 1 || n2 < 1 || c_out3 < 1 || n3 < 1 ||
      c_out4 < 1 || n4 < 1)
    return CS_ERR_SHAPE;
  cs::ConvGeom geo0;
  int st = conv_geometry(b, h, w, c_in, kh, kw, stride, pad, c_out, n, pool, &geo0);
  if (st != CS_OK) return st;
  if (k > c_out || ocap < k) return CS_ERR_SHAPE;
  const int R = kh * kw * c_in;
  if (n != 1 || c_out != 64 || R > 32) return CS_ERR_SHAPE;
  const int hp0 = geo0.Ho / pool, wp0 = geo0.Wo / pool;
  cs::ConvGeom geo;
  st = conv_geometry(b, hp0, wp0, c_out, kh2, kw2, stride2, pad2, c_out2, n2, pool2, &geo);
  if (st != CS_OK) return st;
  if (k2 > c_out2 || c_out2 > CS_MAX_KWTA_ROW || ocap2 < k2) return CS_ERR_SHAPE;
  const int hp = geo.Ho / pool2, wp = geo.Wo / pool2;
  cs::ConvGeom geo2;
  st = conv_geometry(b, hp, wp, c_out2, hp, wp, 1, 0, c_out3, n3, 1, &geo2);
  if (st != CS_OK) return st;
  if (k3 > c_out3 || c_out3 > CS_MAX_KWTA_ROW || ocap3 < k3) return CS_ERR_SHAPE;
  if (n4 > CS_MAX_N || c_out4 % n4 != 0) return CS_ERR_SHAPE;
  geo.cap = ocap;
  geo2.cap = ocap2;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // one kernel: each phase one workgroup per image (the first layer's tile
  // and the second's band are the whole image), within one compute unit's LDS
  const bool lists_ok = ocap % 4 == 0 && aligned(oidx, 8) && aligned(oval, 4);
  cs::DenseArgs da{};
  size_t sh0 = 0;
  ScatterPlan scp{};
  GatherPlan gp{};
  SamplePlan sp;
  bool ga = false;
  if (k <= 32 && lists_ok && aligned(aug, 16) && (pool == 1 || pool == 2) &&
      (int64_t)b * hp0 * wp0 * 64 < INT32_MAX &&
      dense_plan(geo0, x, w, pad, k, shift, keep_sums, ocap, 1, hp0, kCuLds, &da, &sh0) &&
      da.tiles_img == 1 && !sample_plan(geo, xt, k2, shift2, keep_sums, &sp) &&
      ((ga = pool == 2 && gather_plan(geo, aug2, k2, shift2, keep_sums, &gp)) ||
       (scatter_plan(geo, xt, aug2, k2, shift2, keep_sums, &scp) && scp.sc.bands == 1 &&
        scp.blocks == b && scp.gpl == 2 && scp.m == 1)) &&
      sample_plan(geo2, xt, k3, shift3, keep_sums, &sp)) {
    const cs::NextLayer nx{static_cast<const uint16_t*>(aug4), static_cast<const int32_t*>(bias4),
                           static_cast<int32_t*>(y4), c_out4 / n4, n4, c_out4,
                           (uint32_t)round16(sp.shmem)};
    const size_t sh2 = (size_t)nx.off_acc + round16((size_t)c_out4 * 4);
    const size_t shmem = std::max(sh0, std::max(ga ? gp.shmem : scp.shmem, sh2));
    if (shmem <= kCuLds) {
      const cs::ListOut lo0{oidx, oval, ocnt, ocap};
      const cs::ListOut lo{oidx2, oval2, ocnt2, ocap2};
      const cs::ListOut lo2{oidx3, oval3, ocnt3, ocap3};
#define CS_DC4(P_, K_, M_, G_)                                                                  \
  launch_dense_chain<P_, K_, M_, G_>(da, scp, gp, sp, shmem, s, x, aug, bias, y, lo0, geo0, aug2, \
                                     bias2, y2, lo, geo, aug3, bias3, y3, lo2, geo2, nx)
#define CS_DC3(P_, K_, M_)                                              \
  do {                                                                  \
    if (P_ == 2 && K_ <= 5 && ga) CS_DC4(P_, K_, M_, (P_ == 2 && K_ <= 5)); \
    else CS_DC4(P_, K_, M_, false);                                     \
  } while (0)
#define CS_DC(P_, K_)                                   \
  do {                                                  \
    if (da.kmode == 1) CS_DC3(P_, K_, 1);               \
    else if (da.kmode == 2) CS_DC3(P_, K_, 2);          \
    else CS_DC3(P_, K_, 3);                             \
  } while (0)
      if (pool == 2) {
        if (geo.KW == 3) CS_DC(2, 3);
        else if (geo.KW == 5) CS_DC(2, 5);
        else CS_DC(2, 7);
      } else {
        if (geo.KW == 3) CS_DC(1, 3);
        else if (geo.KW == 5) CS_DC(1, 5);
        else CS_DC(1, 7);
      }
#undef CS_DC
#undef CS_DC3
#undef CS_DC4
      return launch_status();
    }
  }
  // otherwise: the first layer, then the three-layer tail on its lists
  st = cs_conv2d_dense_kwta(xt, x, b, h, w, c_in, kh, kw, stride, pad, aug, c_out, n, bias, pool, y,
                            keep_sums, k, ot, shift, nullptr, oidx, oval, ocnt, ocap, stream);
  if (st != CS_OK) return st;
  return cs_mrs_kwta_chain3(xt, oidx, oval, ocnt, ocap, b, hp0, wp0, c_out, kh2, kw2, stride2, pad2,
                            aug2, c_out2, n2, bias2, pool2, y2, keep_sums, k2, ot, shift2, oidx2,
                            oval2, ocnt2, ocap2, aug3, c_out3, n3, bias3, y3, k3, shift3, oidx3,
                            oval3, ocnt3, ocap3, aug4, c_out4, n4, bias4, y4, stream);
}

extern "C" int cs_phase_stamps(unsigned long long* acc, int n, int reset, int* clock_khz) {
#ifdef CS_PHASE_STAMPS
  if (n < 0 || n > 32 || (n > 0 && !acc)) return CS_ERR_ARG;
  unsigned long long v[32] = {0};
  int dev = 0;
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpyFromSymbol(v, HIP_SYMBOL(cs_phase_acc), sizeof(v), 0, hipMemcpyDeviceToHost) !=
          hipSuccess ||
      hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return CS_ERR_DEVICE;
  }
  for (int i = 0; i < n; ++i) acc[i] = v[i];
  if (clock_khz &&
      hipDeviceGetAttribute(clock_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) {
    (void)hipGetLastError();
    return CS_ERR_DEVICE;
  }
  if (reset) {
    const unsigned long long zero[32] = {0};
    if (hipMemcpyToSymbol(HIP_SYMBOL(cs_phase_acc), zero, sizeof(zero), 0,
                          hipMemcpyHostToDevice) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess) {
      (void)hipGetLastError();
      return CS_ERR_DEVICE;
    }
  }
  return CS_OK;
#else
  (void)acc;
  (void)n;
  (void)reset;
  if (clock_khz) *clock_khz = 0;
  return CS_ERR_UNSUPPORTED;
#endif
}

extern "C" int cs_product_count(unsigned long long* count, int reset) {
#ifdef CS_COUNT_PRODUCTS
  unsigned long long v = 0;
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpyFromSymbol(&v, HIP_SYMBOL(cs_products_formed), sizeof(v), 0,
                          hipMemcpyDeviceToHost) != hipSuccess) {
    (void)hipGetLastError();
    return CS_ERR_DEVICE;
  }
  if (count) *count = v;
  if (reset) {
    const unsigned long long zero = 0;
    if (hipMemcpyToSymbol(HIP_SYMBOL(cs_products_formed), &zero, sizeof(zero), 0,
                          hipMemcpyHostToDevice) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess) {
      (void)hipGetLastError();
      return CS_ERR_DEVICE;
    }
  }
  return CS_OK;
#else
  if (count) *count = 0;
  (void)reset;
  return CS_ERR_UNSUPPORTED;
#endif
}
