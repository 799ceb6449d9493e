// C ABI entry points of the sparse-sparse layer (declared in include/cs.h).
// Every argument is checked on the host before the first HIP call; kernels
// are enqueued on the caller's stream and nothing is allocated, freed or
// synchronised here.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "compact_kernels.h"
#include "cs.h"
#include "kwta_kernels.h"
#include "mrs_kernels.h"
#include "mrs_tiled.h"

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
int compact_checked(cs_dtype xt, const void* x, int64_t rows, int c, uint16_t* idx, void* val,
                    int32_t* cnt, hipStream_t stream) {
  if (rows == 0) return CS_OK;
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

int mrs_launch(cs_dtype xt, const uint16_t* idx, const void* lval, const int32_t* cnt,
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
  if (geo.cap % 4 != 0 || Gs < 1 || log2S + ta.log2Q > 6 || !fits32)
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
  int bpc = (int)(kCuLds / shmem);
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
  hipLaunchKernelGGL((cs::kwta_wave<TI, TO, MM>), grid, block, 0, stream, in, rows, c, k, out, \
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
