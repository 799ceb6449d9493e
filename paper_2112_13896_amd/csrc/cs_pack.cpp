// cs_pack: Combine step of Complementary Sparsity (Sections 3.1 and 3.2,
// step 1; Figure 7).  N kernels whose supports do not collide are overlaid
// into one packed kernel; every slot keeps the weight value and the Kernel ID
// of the kernel that owns it (Section 3.3.1), the ID being local to the set
// (Section 3.3.2).  Host memory only; no HIP call.
#include <cstdint>
#include <cstring>

#include "cs.h"

namespace {

inline void put(uint16_t* aug, int64_t s, int8_t v, int kid) {
  aug[s] = (uint16_t)((uint8_t)v | ((uint16_t)kid << 8));
}
inline void put(cs_aug_f32* aug, int64_t s, float v, int kid) {
  aug[s].value = v;
  aug[s].kid = (uint32_t)kid;
}

template <typename T, typename E>
int pack_impl(const T* w, int d_out, int r, int n, E* aug, int64_t* holes, int* bad_g,
              int* bad_i) {
  const int G = d_out / n;
  int64_t nholes = 0;
  for (int g = 0; g < G; ++g) {
    for (int i = 0; i < r; ++i) {
      int owner = -1;
      for (int j = 0; j < n; ++j) {
        const T v = w[(int64_t)(g * n + j) * r + i];
        if (v != T(0)) {
          if (owner >= 0) {
            if (bad_g) *bad_g = g;
            if (bad_i) *bad_i = i;
            return CS_ERR_COLLISION;
          }
          owner = j;
        }
      }
      const int64_t s = (int64_t)i * G + g;
      if (owner < 0) {
        put(aug, s, T(0), 0);
        ++nholes;
      } else {
        put(aug, s, w[(int64_t)(g * n + owner) * r + i], owner);
      }
    }
  }
  if (holes) *holes = nholes;
  return CS_OK;
}

}  // namespace

extern "C" int cs_pack(cs_dtype wt, const void* w, int d_out, int r, int n, void* aug,
                       int64_t* holes, int* bad_g, int* bad_i) {
  if (bad_g) *bad_g = -1;
  if (bad_i) *bad_i = -1;
  if (holes) *holes = 0;
  if (!w || !aug || d_out < 1 || r < 1 || n < 1) return CS_ERR_ARG;
  if (n > CS_MAX_N || d_out % n != 0) return CS_ERR_SHAPE;
  switch (wt) {
    case CS_I8:
      return pack_impl(static_cast<const int8_t*>(w), d_out, r, n, static_cast<uint16_t*>(aug),
                       holes, bad_g, bad_i);
    case CS_F32:
      return pack_impl(static_cast<const float*>(w), d_out, r, n, static_cast<cs_aug_f32*>(aug),
                       holes, bad_g, bad_i);
    default:
      return CS_ERR_DTYPE;
  }
}

extern "C" int cs_reorder_table(const void* aug, int kh, int kw, int c_in, int c_out, int n,
                                int* smax, int32_t* table) {
  if (!aug || !smax || kh < 1 || kw < 1 || c_in < 1 || c_out < 1 || n < 1) return CS_ERR_ARG;
  if (n > CS_MAX_N || c_out % n != 0) return CS_ERR_SHAPE;
  if ((int64_t)kh * kw * c_in > CS_MAX_ROW) return CS_ERR_SHAPE;
  const int G = c_out / n, R = kh * kw * c_in;
  const cs_aug_f32* a = static_cast<const cs_aug_f32*>(aug);
  // the support of every kernel: its non-zero slots (holes and zero weights
  // add nothing and are left out)
  int longest = 0;
  for (int o = 0; o < c_out; ++o) {
    const int g = o / n, kid = o - g * n;
    int cnt = 0;
    for (int i = 0; i < R; ++i) {
      const cs_aug_f32& e = a[(int64_t)i * G + g];
      if (e.kid >= (uint32_t)n) return CS_ERR_ARG;
      cnt += (e.value != 0.f && (int)e.kid == kid) ? 1 : 0;
    }
    longest = cnt > longest ? cnt : longest;
  }
  const int sm = longest > 0 ? longest : 1;
  if (!table) {
    *smax = sm;
    return CS_OK;
  }
  if (*smax < sm) return CS_ERR_SHAPE;
  const int hw = CS_REORDER_TILE + kw - 1, cp = c_in + 1;
  for (int o = 0; o < c_out; ++o) {
    const int g = o / n, kid = o - g * n;
    int32_t* t = table + (int64_t)o * *smax * 2;
    int j = 0;
    for (int i = 0; i < R; ++i) {
      const cs_aug_f32& e = a[(int64_t)i * G + g];
      if (e.value == 0.f || (int)e.kid != kid) continue;
      // slot i = (ky * kw + kx) * c_in + c -> byte offset in the input tile
      const int tap = i / c_in, c = i - tap * c_in;
      const int ky = tap / kw, kx = tap - ky * kw;
      t[2 * j] = 4 * ((ky * hw + kx) * cp + c);
      std::memcpy(&t[2 * j + 1], &e.value, 4);
      ++j;
    }
    for (; j < *smax; ++j) {                                      // padding: offset 0, weight 0
      t[2 * j] = 0;
      t[2 * j + 1] = 0;
    }
  }
  return CS_OK;
}

extern "C" int cs_pack_blocks(cs_dtype wt, const void* w, int d_out, int r, int n, int b,
                              void* aug, uint8_t* kidb, int64_t* holes, int* bad_g, int* bad_i) {
  if (bad_g) *bad_g = -1;
  if (bad_i) *bad_i = -1;
  if (holes) *holes = 0;
  if (!w || !aug || !kidb || d_out < 1 || r < 1 || n < 1 || b < 1) return CS_ERR_ARG;
  if (wt != CS_I8 && wt != CS_F32) return CS_ERR_DTYPE;
  if (n > CS_MAX_N || d_out % n != 0 || r % b != 0) return CS_ERR_SHAPE;
  const int nb = r / b, G = d_out / n;
  const size_t es = wt == CS_I8 ? 1 : 4;
  auto nz = [&](int o, int i) {
    const unsigned char* p = static_cast<const unsigned char*>(w) + ((int64_t)o * r + i) * es;
    if (wt == CS_I8) return *reinterpret_cast<const int8_t*>(p) != 0;
    float v;
    std::memcpy(&v, p, 4);
    return v != 0.f;
  };
  // every support a union of whole blocks
  for (int o = 0; o < d_out; ++o)
    for (int j = 0; j < nb; ++j) {
      int c = 0;
      for (int t = 0; t < b; ++t) c += nz(o, j * b + t) ? 1 : 0;
      if (c != 0 && c != b) {
        if (bad_g) *bad_g = o;
        if (bad_i) *bad_i = j;
        return CS_ERR_SHAPE;
      }
    }
  // complementary block by block: one Kernel ID per (block, set)
  int64_t nh = 0;
  for (int g = 0; g < G; ++g)
    for (int j = 0; j < nb; ++j) {
      int owner = -1;
      for (int k = 0; k < n; ++k) {
        if (nz(g * n + k, j * b)) {
          if (owner >= 0) {
            if (bad_g) *bad_g = g;
            if (bad_i) *bad_i = j;
            return CS_ERR_COLLISION;
          }
          owner = k;
        }
      }
      kidb[(int64_t)j * G + g] = (uint8_t)(owner >= 0 ? owner : 0);
      nh += owner < 0 ? 1 : 0;
    }
  if (holes) *holes = nh;
  // the per-slot augmented tensor every layer kernel reads
  return cs_pack(wt, w, d_out, r, n, aug, nullptr, nullptr, nullptr);
}

extern "C" int cs_pack_channels(cs_dtype wt, const void* w, int c_out, int kh, int kw, int c_in,
                                int n, void* packed, int64_t* holes, int* bad_o, int* bad_i) {
  if (bad_o) *bad_o = -1;
  if (bad_i) *bad_i = -1;
  if (holes) *holes = 0;
  if (!w || !packed || c_out < 1 || kh < 1 || kw < 1 || c_in < 1 || n < 1) return CS_ERR_ARG;
  if (wt != CS_F32 && wt != CS_I8) return CS_ERR_DTYPE;
  if (n > CS_MAX_N || c_in % n != 0) return CS_ERR_SHAPE;
  const int Q = c_in / n;
  int64_t nh = 0;
  for (int o = 0; o < c_out; ++o)
    for (int q = 0; q < Q; ++q)
      for (int y = 0; y < kh; ++y)
        for (int x = 0; x < kw; ++x) {
          const int64_t wi = (((int64_t)o * kh + y) * kw + x) * c_in + q * n;
          int owner = -1;
          for (int j = 0; j < n; ++j) {
            const bool nz = wt == CS_F32 ? static_cast<const float*>(w)[wi + j] != 0.f
                                         : static_cast<const int8_t*>(w)[wi + j] != 0;
            if (nz) {
              if (owner >= 0) {
                if (bad_o) *bad_o = o;
                if (bad_i) *bad_i = (q * kh + y) * kw + x;
                return CS_ERR_COLLISION;
              }
              owner = j;
            }
          }
          const int64_t pi = (((int64_t)o * Q + q) * kh + y) * kw + x;
          if (wt == CS_F32) {
            cs_aug_f32& e = static_cast<cs_aug_f32*>(packed)[pi];
            e.value = owner >= 0 ? static_cast<const float*>(w)[wi + owner] : 0.f;
            e.kid = owner >= 0 ? (uint32_t)owner : 0u;
          } else {
            const uint8_t v = owner >= 0 ? (uint8_t)static_cast<const int8_t*>(w)[wi + owner] : 0;
            static_cast<uint16_t*>(packed)[pi] =
                (uint16_t)(v | (owner >= 0 ? (uint32_t)owner << 8 : 0u));
          }
          nh += owner < 0 ? 1 : 0;
        }
  if (holes) *holes = nh;
  return CS_OK;
}

extern "C" int cs_channel_table(const uint16_t* packed, int kh, int kw, int c_in, int c_out, int n,
                                int stride, int32_t* table) {
  if (!packed || !table || kh < 1 || kw < 1 || c_in < 1 || c_out < 1 || n < 1 || stride < 1)
    return CS_ERR_ARG;
  if (n > CS_MAX_N || c_in % n != 0 || c_in % 4 != 0) return CS_ERR_SHAPE;
  const int Q = c_in / n, S = Q * kh * kw, S4 = (S + 3) / 4;
  const int64_t sw = (int64_t)63 * stride + kw;            // staged pixels per row
  const int64_t cp = (c_in / 4) % 2 == 1 ? c_in : c_in + 4; // staged bytes per pixel
  if ((int64_t)kh * sw * cp >= ((int64_t)1 << 23)) return CS_ERR_SHAPE;
  for (int o = 0; o < c_out; ++o) {
    int32_t* row = table + (int64_t)o * 5 * S4;             // offsets [4*S4], weights [S4]
    for (int i = 0; i < 5 * S4; ++i) row[i] = 0;            // padding slots: offset 0, weight 0
    for (int q = 0; q < Q; ++q)
      for (int y = 0; y < kh; ++y)
        for (int x = 0; x < kw; ++x) {
          const int si = (q * kh + y) * kw + x;
          const uint16_t e = packed[(int64_t)o * S + si];
          const int cid = e >> 8;
          if (cid >= n) return CS_ERR_ARG;
          row[si] = (int32_t)((y * sw + x) * cp + q * n + cid);
          row[4 * S4 + si / 4] |= (int32_t)((uint32_t)(e & 0xFFu) << (8 * (si % 4)));
        }
  }
  return CS_OK;
}

extern "C" int cs_reorder_table_channels(const void* packed, int kh, int kw, int c_in, int c_out,
                                         int n, int* smax, int32_t* table) {
  if (!packed || !smax || kh < 1 || kw < 1 || c_in < 1 || c_out < 1 || n < 1) return CS_ERR_ARG;
  if (n > CS_MAX_N || c_in % n != 0) return CS_ERR_SHAPE;
  if ((int64_t)kh * kw * c_in > CS_MAX_ROW) return CS_ERR_SHAPE;
  const cs_aug_f32* P = static_cast<const cs_aug_f32*>(packed);
  const int Q = c_in / n, S = Q * kh * kw;                        // packed slots per filter
  int longest = 0;
  for (int o = 0; o < c_out; ++o) {
    int cnt = 0;
    for (int i = 0; i < S; ++i) {
      const cs_aug_f32& e = P[(int64_t)o * S + i];
      if (e.kid >= (uint32_t)n) return CS_ERR_ARG;
      cnt += e.value != 0.f ? 1 : 0;
    }
    longest = cnt > longest ? cnt : longest;
  }
  const int sm = longest > 0 ? longest : 1;
  if (!table) {
    *smax = sm;
    return CS_OK;
  }
  if (*smax < sm) return CS_ERR_SHAPE;
  const int hw = CS_REORDER_TILE + kw - 1, cp = c_in + 1;
  for (int o = 0; o < c_out; ++o) {
    int32_t* t = table + (int64_t)o * *smax * 2;
    int j = 0;
    // packed slot (q, y, x) with channel ID cid reads channel q*n + cid at tap (y, x)
    for (int q = 0; q < Q; ++q)
      for (int y = 0; y < kh; ++y)
        for (int x = 0; x < kw; ++x) {
          const cs_aug_f32& e = P[(((int64_t)o * Q + q) * kh + y) * kw + x];
          if (e.value == 0.f) continue;
          const int c = q * n + (int)e.kid;
          t[2 * j] = 4 * ((y * hw + x) * cp + c);
          std::memcpy(&t[2 * j + 1], &e.value, 4);
          ++j;
        }
    for (; j < *smax; ++j) {
      t[2 * j] = 0;
      t[2 * j + 1] = 0;
    }
  }
  return CS_OK;
}

extern "C" const char* cs_status_str(int status) {
  switch (status) {
    case CS_OK: return "ok";
    case CS_ERR_ARG: return "invalid argument (null pointer, size or enum)";
    case CS_ERR_SHAPE: return "inconsistent or unsupported shape";
    case CS_ERR_DTYPE: return "unsupported dtype";
    case CS_ERR_COLLISION: return "two kernels of one packed set share a slot";
    case CS_ERR_WORKSPACE: return "workspace missing or too small";
    case CS_ERR_DEVICE: return "HIP device error";
    case CS_ERR_UNSUPPORTED: return "not available in this build of the library";
    default: return "unknown status";
  }
}
