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

// RN32(a / Q) and RN32(Q / a) for a positive finite binary16 magnitude a
// (held in binary32) and Q in {7, 127}, without a full division: the quotient
// from the constant RN32(1/Q), respectively the hardware reciprocal of a, plus
// one Newton-Raphson correction (Markstein's scheme: residual by a fused
// multiply-add, then a fused correction).  Checked exhaustively in exact
// arithmetic to give the correctly rounded quotient for every such a and for
// any reciprocal within 2 ulp of 1/a.
__device__ __forceinline__ float scale_of(float a, float Qf, float inv_q) {
  const float s0 = a * inv_q;
  const float e = __builtin_fmaf(-s0, Qf, a);
  return __builtin_fmaf(e, inv_q, s0);
}
__device__ __forceinline__ float recip_scale_of(float a, float Qf) {
  const float r0 = __builtin_amdgcn_rcpf(a);
  const float q0 = Qf * r0;
  const float e = __builtin_fmaf(-q0, a, Qf);
  return __builtin_fmaf(e, r0, q0);
}
// RN32(Qf / a) for any positive normal binary32 a and Qf in {15, 255}: the
// sequence above after one refinement of the reciprocal (checked exhaustively
// over every binary32 significand and any hardware reciprocal within 2 ulp;
// without the refinement a few binary32 a round wrongly).
__device__ __forceinline__ float recip_scale_of_f32(float a, float Qf) {
  const float r0 = __builtin_amdgcn_rcpf(a);
  const float y = __builtin_fmaf(__builtin_fmaf(-a, r0, 1.0f), r0, r0);
  const float q0 = Qf * y;
  const float e = __builtin_fmaf(-q0, a, Qf);
  return __builtin_fmaf(e, y, q0);
}

// amax: the row's largest magnitude pattern (bits & 0x7FFF, reduced over the
// row's lanes).  code = clamp(rne(RN32(x * RN32(Q / a))), -Q, Q); for a finite
// row |RN32(x r)| < Q + 1/2 (checked exhaustively over a), so the clamp never
// binds and is not executed.  Rounding to an integer adds 1.5 * 2^23: the low
// mantissa bits of the sum hold the code in two's complement.
__device__ __forceinline__ LaneCodes quantize_lane(u32x4 x, uint32_t amax, int Q) {
  LaneCodes out;
  out.nonfinite = amax >= 0x7C00u;
  if (out.nonfinite || amax == 0u) {
    out.scale = out.nonfinite ? __builtin_bit_cast(float, 0x7FC00000u) : 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) out.c[i] = 0x4B400000u;  // code 0
    return out;
  }
  const float Qf = static_cast<float>(Q);
  const float inv_q = Q == 127 ? 1.0f / 127.0f : 1.0f / 7.0f;  // RN32(1/Q), folded at compile time
  const float a = half_lo(amax);
  out.scale = scale_of(a, Qf, inv_q);
  const float rcp = recip_scale_of(a, Qf);
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out.c[2 * i] = __builtin_bit_cast(uint32_t, half_lo(w[i]) * rcp + 12582912.0f);
    out.c[2 * i + 1] = __builtin_bit_cast(uint32_t, half_hi(w[i]) * rcp + 12582912.0f);
  }
  return out;
}

// 8 INT8 codes as 8 bytes, element order (byte 0 of each code word).
__device__ __forceinline__ u32x2 pack_int8(const LaneCodes& q) {
  // perm selector 0x0c0c0400: bytes [lo.b0, hi.b0, 0, 0]; 0x05040100 joins two halves
  const uint32_t p01 = __builtin_amdgcn_perm(q.c[1], q.c[0], 0x0c0c0400u);
  const uint32_t p23 = __builtin_amdgcn_perm(q.c[3], q.c[2], 0x0c0c0400u);
  const uint32_t p45 = __builtin_amdgcn_perm(q.c[5], q.c[4], 0x0c0c0400u);
  const uint32_t p67 = __builtin_amdgcn_perm(q.c[7], q.c[6], 0x0c0c0400u);
  return u32x2{__builtin_amdgcn_perm(p23, p01, 0x05040100u), __builtin_amdgcn_perm(p67, p45, 0x05040100u)};
}

// 8 INT4 codes as 4 bytes: element 2i in the low nibble of byte i.
__device__ __forceinline__ uint32_t pack_int4(const LaneCodes& q) {
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) out |= (q.c[i] & 0xFu) << (4 * i);
  return out;
}

// 8 signed codes times the row scale, rounded to binary32 and then to binary16.
// code * s rounded to binary32 (the value the binary16 conversion then
// rounds).  The register pin keeps the product a binary32 value: left free,
// the backend folds multiply and conversion into one mixed-precision FMA that
// rounds the exact product straight to binary16.  The two agree for every
// scale the quantizer produces (RN32(a / Q), checked exhaustively over a and
// the codes), but not for arbitrary scales, such as a payload's corrupted or
// externally written ones.
__device__ __forceinline__ float scaled(float code, float s) {
  float p = code * s;
  asm("" : "+v"(p));
  return p;
}

__device__ __forceinline__ u32x4 dequant_int8(u32x2 c, float s) {
  const uint32_t w[2] = {c.x, c.y};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float f0 = scaled(static_cast<float>(static_cast<int32_t>(w[i] << 24) >> 24), s);
    const float f1 = scaled(static_cast<float>(static_cast<int32_t>(w[i] << 16) >> 24), s);
    const float f2 = scaled(static_cast<float>(static_cast<int32_t>(w[i] << 8) >> 24), s);
    const float f3 = scaled(static_cast<float>(static_cast<int32_t>(w[i]) >> 24), s);
    o[2 * i] = pack_half2(f0, f1);
    o[2 * i + 1] = pack_half2(f2, f3);
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

__device__ __forceinline__ u32x4 dequant_int4(uint32_t w, float s) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float f0 = scaled(static_cast<float>(static_cast<int32_t>(w << (28 - 8 * i)) >> 28), s);
    const float f1 = scaled(static_cast<float>(static_cast<int32_t>(w << (24 - 8 * i)) >> 28), s);
    o[i] = pack_half2(f0, f1);
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

constexpr uint32_t kNaNHalf2 = 0x7E007E00u;

// A pair of binary16 values with every NaN replaced by the canonical 0x7E00
// (the hardware's NaN from an invalid product, 0 * inf, has its sign set).
__device__ __forceinline__ uint32_t canon_nan_half2(uint32_t w) {
  const uint32_t lo = w & 0xFFFFu, hi = w >> 16;
  return ((lo & 0x7FFFu) > 0x7C00u ? 0x7E00u : lo) | (((hi & 0x7FFFu) > 0x7C00u ? 0x7E00u : hi) << 16);
}
__device__ __forceinline__ u32x4 canon_nan_lane(u32x4 o) {
  return u32x4{canon_nan_half2(o.x), canon_nan_half2(o.y), canon_nan_half2(o.z), canon_nan_half2(o.w)};
}

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
