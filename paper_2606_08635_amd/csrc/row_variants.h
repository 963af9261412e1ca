// Per-tier quantizer variants (any scheme may run inside a tier: Sec. 6.10,
// Sec. 8; KIVI-style asymmetric quantization, Sec. 8 and Sec. 10): scale
// groups of 64 or 32 elements, asymmetric min/max codes with the group
// minimum as zero point, binary16 metadata.  A descriptor per quantized tier:
//   bits 0-1  elements per group: 0 the row (d), 1 64, 2 32 (capped at d)
//   bit 2     asymmetric: codes 0..M (M = 255 / 15), x^ = code * s + lo
//   bit 3     s (and lo) stored as binary16
// Per group, symmetric: s = RN32(a/Q), r = RN32(Q/a) (a = max |x|); with
// binary16 metadata s = RN16(RN32(a/Q)), r = RN32(1/s) and codes clamped to
// +-Q.  Asymmetric: lo, hi the group's minimum and maximum (-0 below +0),
// range = RN32(hi - lo), s = RN32(range/M), r = RN32(M/range) (binary16:
// s = RN16(RN32(range/M)), r = RN32(1/s)), code = clamp(rne(RN32(RN32(x - lo) r)),
// 0, M).  A group holding an inf/NaN gets NaN metadata and zero codes; a zero
// a or range (or a binary16 s that underflows to 0) gives zero codes.
// Metadata of a quantized row: per group s (then lo), fp32 or binary16,
// located at a byte offset carried by the chunk index (third word) plus a
// block scan; it is accessed in 16-bit pieces because binary16 entries make
// the offsets only 2-byte aligned.
#pragma once

#include "device_util.h"
#include "row_codec.h"
#include "row_stream.h"
#include "skv_internal.h"

namespace skv {

constexpr int32_t kQuantAsym = 4, kQuantFp16 = 8;

struct VarCfg {
  int32_t q8, q4;  // descriptors of the INT8 and INT4 tiers
  uint32_t e8, e4;  // metadata bytes of an INT8 / INT4 row
};

__device__ __forceinline__ int var_group_lanes(int32_t q, int D) {
  const int gs = (q & 3) == 0 ? D : (q & 3) == 1 ? 64 : 32;
  return (gs < D ? gs : D) / 8;
}

// Sort key of a binary16 pattern: finite values in numeric order, -0 below +0.
__device__ __forceinline__ uint32_t order_key16(uint32_t h) {
  return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
}
__device__ __forceinline__ uint32_t key_to_half(uint32_t k) {
  return (k & 0x8000u) ? (k & 0x7FFFu) : (~k & 0xFFFFu);
}

// Reduction over aligned groups of gl lanes (gl a power of two <= LPR); every
// lane of the wavefront must call it.
template <int LPR, bool MAX>
__device__ __forceinline__ uint32_t group_reduce(uint32_t v, int gl) {
#pragma unroll
  for (int o = 1; o < LPR; o <<= 1) {
    const uint32_t p = static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), o));
    if (o < gl) v = MAX ? max(v, p) : min(v, p);
  }
  return v;
}

__device__ __forceinline__ void store_u32_as_halves(uint8_t* p, uint32_t v) {
  reinterpret_cast<uint16_t*>(p)[0] = static_cast<uint16_t>(v);
  reinterpret_cast<uint16_t*>(p)[1] = static_cast<uint16_t>(v >> 16);
}
__device__ __forceinline__ uint32_t load_u32_from_halves(const uint8_t* p) {
  return static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[0]) |
         (static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[1]) << 16);
}

// Quantizes the lane's 8 elements of a row at tier tr under descriptor q and
// writes the group's metadata at meta (the row's metadata) from the group's
// first lane.  All lanes of the wavefront call it (reductions).
template <int LPR>
__device__ __forceinline__ LaneCodes quantize_lane_var(u32x4 x, int tr, int32_t q, int lane, uint8_t* meta,
                                                       bool write_meta) {
  constexpr int D = LPR * 8;
  const int gl = var_group_lanes(q, D);
  const bool asym = (q & kQuantAsym) != 0, f16 = (q & kQuantFp16) != 0;
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t kmin = 0xFFFFu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t k0 = order_key16(w[i] & 0xFFFFu), k1 = order_key16(w[i] >> 16);
    kmin = min(kmin, min(k0, k1));
    kmax = max(kmax, max(k0, k1));
  }
  const uint32_t lane_amax = absmax_bits8(x);
  const uint32_t amax = group_reduce<LPR, true>(lane_amax, gl);
  kmin = group_reduce<LPR, false>(kmin, gl);
  kmax = group_reduce<LPR, true>(kmax, gl);
  const bool bad = amax >= 0x7C00u;  // this group holds an inf/NaN

  LaneCodes out;
  out.nonfinite = group_max<LPR>(lane_amax) >= 0x7C00u;  // some group of the row does
  const int Q = tr == kINT8 ? 127 : 7, M = tr == kINT8 ? 255 : 15;
  float scale = 0.0f, r = 0.0f, lo = 0.0f;
  uint32_t s16 = 0, lo16 = key_to_half(kmin);
  bool zero = false;
  if (bad) {
    scale = __builtin_bit_cast(float, 0x7FC00000u);
    lo = scale;
    s16 = lo16 = 0x7E00u;
    zero = true;
  } else if (!asym) {
    if (amax == 0u) {
      zero = true;
    } else {
      const float a = half_lo(amax);
      scale = scale_of(a, static_cast<float>(Q), Q == 127 ? 1.0f / 127.0f : 1.0f / 7.0f);
      if (f16) {
        s16 = __builtin_bit_cast(uint16_t, static_cast<_Float16>(scale));
        scale = half_lo(s16);
        zero = s16 == 0u;
        r = zero ? 0.0f : 1.0f / scale;  // correctly rounded division
      } else {
        r = recip_scale_of(a, static_cast<float>(Q));
      }
    }
  } else {
    lo = half_lo(lo16);
    const float range = half_lo(key_to_half(kmax)) - lo;
    if (range == 0.0f) {
      zero = true;
    } else {
      scale = range / static_cast<float>(M);
      if (f16) {
        s16 = __builtin_bit_cast(uint16_t, static_cast<_Float16>(scale));
        scale = half_lo(s16);
        zero = s16 == 0u;
        r = zero ? 0.0f : 1.0f / scale;
      } else {
        r = static_cast<float>(M) / range;
      }
    }
  }
  out.scale = scale;
  const int32_t base = 0x4B400000;
  const int32_t cmin = asym ? base : base - Q, cmax = asym ? base + M : base + Q;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float y0, y1;
    if (asym) {
      y0 = (half_lo(w[i]) - lo) * r;
      y1 = (half_hi(w[i]) - lo) * r;
    } else {
      y0 = half_lo(w[i]) * r;
      y1 = half_hi(w[i]) * r;
    }
    const int32_t c0 = min(max(__builtin_bit_cast(int32_t, y0 + 12582912.0f), cmin), cmax);
    const int32_t c1 = min(max(__builtin_bit_cast(int32_t, y1 + 12582912.0f), cmin), cmax);
    out.c[2 * i] = static_cast<uint32_t>(zero ? base : c0);
    out.c[2 * i + 1] = static_cast<uint32_t>(zero ? base : c1);
  }
  if (write_meta && (lane % gl) == 0) {
    uint8_t* e = meta + (lane / gl) * (asym ? 2 : 1) * (f16 ? 2 : 4);
    if (f16) {
      reinterpret_cast<uint16_t*>(e)[0] = static_cast<uint16_t>(s16);
      if (asym) reinterpret_cast<uint16_t*>(e)[1] = static_cast<uint16_t>(lo16);
    } else {
      store_u32_as_halves(e, __builtin_bit_cast(uint32_t, scale));
      if (asym) store_u32_as_halves(e + 4, __builtin_bit_cast(uint32_t, lo));
    }
  }
  return out;
}

// Row-width units and metadata bytes of one token (scan value of the variant
// layout: units | metadata bytes << 12).
__device__ __forceinline__ uint32_t var_scan_value(int tr, const VarCfg& v) {
  if (tr == kAbsent) return 0u;
  const uint32_t eb = tr == kINT8 ? v.e8 : tr == kINT4 ? v.e4 : 0u;
  return tier_units(tr) | (eb << 12);
}

// chunk_layout for the variant layout: s.q receives the byte offset of the
// row's metadata inside its segment's metadata.  cidx_entry: {units, quantized
// rows, metadata bytes, 0} of the chunk.  Contains __syncthreads().
template <int D>
__device__ __forceinline__ void chunk_layout_var(ChunkLds& s, int tr, const uint32_t* cidx_entry, const VarCfg& v) {
  uint32_t total;
  const uint32_t ex = block_exclusive_scan_256(var_scan_value(tr, v), s.scan, &total);
  s.tier[threadIdx.x] = static_cast<uint8_t>(tr);
  s.off[threadIdx.x] = (cidx_entry[0] + (ex & 0xFFFu)) * static_cast<uint32_t>(D / 2);
  s.q[threadIdx.x] = cidx_entry[2] + (ex >> 12);
}

template <int D, int ROWS_IN_FLIGHT, bool NT>
__device__ __forceinline__ void pack_chunk_var(const ChunkLds& s, const uint16_t* __restrict__ src,
                                               uint8_t* __restrict__ dst, uint8_t* __restrict__ meta,
                                               uint32_t* nonfinite, int t0, int n, const VarCfg& v) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = (it + u) * RPI + rsub;
      const int t = t0 + row;
      x[u] = u32x4{0u, 0u, 0u, 0u};
      if (t < n && s.tier[row] != kDROP) x[u] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = (it + u) * RPI + rsub;
      const int tr = s.tier[row];
      const bool quant = tr == kINT8 || tr == kINT4;
      const LaneCodes q = quantize_lane_var<LPR>(x[u], tr, tr == kINT8 ? v.q8 : v.q4, lane, meta + s.q[row], quant);
      if (tr == kFP16) {
        store16<NT>(dst + s.off[row] + lane * 16, x[u]);
      } else if (quant) {
        if (q.nonfinite && lane == 0) atomicAdd(nonfinite, 1u);
        uint8_t* out_row = dst + s.off[row];
        if (tr == kINT8) store8<NT>(out_row + lane * 8, pack_int8(q));
        else store4<NT>(out_row + lane * 4, pack_int4(q));
      }
    }
  }
}

// The lane's 8 outputs of a quantized row under descriptor q.
template <int LPR>
__device__ __forceinline__ u32x4 decode_lane_var(int tr, int32_t q, u32x4 raw, const uint8_t* meta, int lane) {
  constexpr int D = LPR * 8;
  const int gl = var_group_lanes(q, D);
  const bool asym = (q & kQuantAsym) != 0, f16 = (q & kQuantFp16) != 0;
  const uint8_t* e = meta + (lane / gl) * (asym ? 2 : 1) * (f16 ? 2 : 4);
  float s, lo = 0.0f;
  if (f16) {
    s = half_lo(reinterpret_cast<const uint16_t*>(e)[0]);
    if (asym) lo = half_lo(reinterpret_cast<const uint16_t*>(e)[1]);
  } else {
    s = __builtin_bit_cast(float, load_u32_from_halves(e));
    if (asym) lo = __builtin_bit_cast(float, load_u32_from_halves(e + 4));
  }
  if (__builtin_isnan(s)) return u32x4{kNaNHalf2, kNaNHalf2, kNaNHalf2, kNaNHalf2};
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int32_t code;
    if (tr == kINT8) {
      const uint32_t b = ((i < 4 ? raw.x : raw.y) >> (8 * (i & 3))) & 0xFFu;
      code = asym ? static_cast<int32_t>(b) : static_cast<int32_t>(static_cast<int8_t>(b));
    } else {
      const uint32_t nib = (raw.x >> (4 * i)) & 0xFu;
      code = asym ? static_cast<int32_t>(nib) : (static_cast<int32_t>(nib << 28) >> 28);
    }
    f[i] = static_cast<float>(code) * s;
    if (asym) f[i] = f[i] + lo;
  }
  return u32x4{pack_half2(f[0], f[1]), pack_half2(f[2], f[3]), pack_half2(f[4], f[5]), pack_half2(f[6], f[7])};
}

template <int D, int ROWS_IN_FLIGHT, bool NT>
__device__ __forceinline__ void unpack_chunk_var(const ChunkLds& s, const uint8_t* __restrict__ src,
                                                 const uint8_t* __restrict__ meta, uint16_t* __restrict__ cache,
                                                 int H, const VarCfg& v) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s.tier[r];
      const uint8_t* row = src + s.off[r];
      raw[u] = u32x4{0u, 0u, 0u, 0u};
      if (tr == kFP16) {
        raw[u] = ld_nt16(row + lane * 16);
      } else if (tr == kINT8) {
        const u32x2 c = ld_nt8(row + lane * 8);
        raw[u].x = c.x;
        raw[u].y = c.y;
      } else if (tr == kINT4) {
        raw[u].x = ld_nt4(row + lane * 4);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s.tier[r];
      if (tr == kAbsent) continue;
      u32x4 o = raw[u];  // FP16 verbatim, DROP zeros
      if (tr == kINT8 || tr == kINT4) o = decode_lane_var<LPR>(tr, tr == kINT8 ? v.q8 : v.q4, raw[u], meta + s.q[r], lane);
      store16<NT>(cache + static_cast<size_t>(s.pos[r]) * H * D + lane * 8, o);
    }
  }
}

}  // namespace skv
