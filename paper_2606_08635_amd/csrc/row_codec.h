// Per-lane pieces of the symmetric absmax row quantizer ("standard symmetric",
// Sec. 8), shared by pack, unpack and the precision upgrade.  A row of d
// binary16 values is held by d/8 lanes, 8 values (16 bytes) per lane.
#pragma once

#include "device_util.h"

namespace skv {

// The lane's 8 codes of one INT8 (Q = 127) or INT4 (Q = 7) row.
struct LaneCodes {
  float scale;      // RN32(a / Q); NaN if the row holds an infinity or NaN; 0 for a zero row
  uint32_t c[8];    // 0x4B400000 + code: the low byte / nibble is the two's-complement code
  bool nonfinite;
};

// amax: the row's largest magnitude pattern (bits & 0x7FFF, reduced over the
// row's lanes).  code = clamp(rne(RN32(x * RN32(Q / a))), -Q, Q).
__device__ __forceinline__ LaneCodes quantize_lane(u32x4 x, uint32_t amax, int Q) {
  LaneCodes out;
  out.nonfinite = amax >= 0x7C00u;
  int32_t lo = 0x4B400000, hi = 0x4B400000;  // clamp window around 1.5 * 2^23
  if (out.nonfinite) {
    out.scale = __builtin_bit_cast(float, 0x7FC00000u);
  } else if (amax == 0u) {
    out.scale = 0.0f;
  } else {
    const float Qf = static_cast<float>(Q);
    const float a = half_lo(amax);
    out.scale = a / Qf;  // correctly rounded binary32 division
    const float rcp = Qf / a;
    lo -= Q;
    hi += Q;
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // RN32(x * r), then rounding to an integer (nearest-even) by adding
      // 1.5 * 2^23: the low mantissa bits of the sum are the code
      const float y0 = half_lo(w[i]) * rcp;
      const float y1 = half_hi(w[i]) * rcp;
      out.c[2 * i] = static_cast<uint32_t>(min(max(__builtin_bit_cast(int32_t, y0 + 12582912.0f), lo), hi));
      out.c[2 * i + 1] = static_cast<uint32_t>(min(max(__builtin_bit_cast(int32_t, y1 + 12582912.0f), lo), hi));
    }
    return out;
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) out.c[i] = static_cast<uint32_t>(lo);  // code 0
  return out;
}

// 8 INT8 codes as 8 bytes, element order.
__device__ __forceinline__ u32x2 pack_int8(const LaneCodes& q) {
  u32x2 out;
  out.x = (q.c[0] & 0xFFu) | ((q.c[1] & 0xFFu) << 8) | ((q.c[2] & 0xFFu) << 16) | (q.c[3] << 24);
  out.y = (q.c[4] & 0xFFu) | ((q.c[5] & 0xFFu) << 8) | ((q.c[6] & 0xFFu) << 16) | (q.c[7] << 24);
  return out;
}

// 8 INT4 codes as 4 bytes: element 2i in the low nibble of byte i.
__device__ __forceinline__ uint32_t pack_int4(const LaneCodes& q) {
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) out |= (q.c[i] & 0xFu) << (4 * i);
  return out;
}

// 8 signed codes times the row scale, rounded to binary32 and then to binary16.
__device__ __forceinline__ u32x4 dequant_int8(u32x2 c, float s) {
  const uint32_t w[2] = {c.x, c.y};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float f0 = static_cast<float>(static_cast<int32_t>(w[i] << 24) >> 24) * s;
    const float f1 = static_cast<float>(static_cast<int32_t>(w[i] << 16) >> 24) * s;
    const float f2 = static_cast<float>(static_cast<int32_t>(w[i] << 8) >> 24) * s;
    const float f3 = static_cast<float>(static_cast<int32_t>(w[i]) >> 24) * s;
    o[2 * i] = pack_half2(f0, f1);
    o[2 * i + 1] = pack_half2(f2, f3);
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

__device__ __forceinline__ u32x4 dequant_int4(uint32_t w, float s) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float f0 = static_cast<float>(static_cast<int32_t>(w << (28 - 8 * i)) >> 28) * s;
    const float f1 = static_cast<float>(static_cast<int32_t>(w << (24 - 8 * i)) >> 28) * s;
    o[i] = pack_half2(f0, f1);
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

constexpr uint32_t kNaNHalf2 = 0x7E007E00u;

// The lane's 8 reconstructed values of a row held at tier tr (what unpack
// writes): FP16 verbatim, DROP zeros, INT8/INT4 dequantized, NaN scale -> 0x7E00.
__device__ __forceinline__ u32x4 held_lane(int tr, u32x4 x, uint32_t amax) {
  if (tr == kFP16) return x;
  if (tr == kDROP) return u32x4{0u, 0u, 0u, 0u};
  const LaneCodes q = quantize_lane(x, amax, tr == kINT8 ? 127 : 7);
  if (q.nonfinite) return u32x4{kNaNHalf2, kNaNHalf2, kNaNHalf2, kNaNHalf2};
  return tr == kINT8 ? dequant_int8(pack_int8(q), q.scale) : dequant_int4(pack_int4(q), q.scale);
}

}  // namespace skv
