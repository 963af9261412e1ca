// Per-tier quantizer variants (any scheme may run inside a tier: Sec. 6.10,
// Sec. 8; KIVI-style asymmetric quantization, Sec. 8 and Sec. 10): scale
// groups of 64 or 32 elements, asymmetric min/max codes with the group
// minimum as zero point, binary16 metadata.  A descriptor per quantized tier:
//   bits 0-1  elements per group: 0 the row (d), 1 64, 2 32 (capped at d)
//   bit 2     asymmetric: codes 0..M (M = 255 / 15), x^ = code * s + lo
//   bit 3     s (and lo) stored as binary16
//   bit 4     per-channel K (KIVI-style key quantization): the K rows of the
//             tier inside a 256-token chunk form one group per channel, with
//             bits 2-3; V rows keep the per-row groups of bits 0-3
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

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int32_t kQuantAsym = 4, kQuantFp16 = 8, kQuantChannel = 16;

struct VarCfg {
  int32_t q8, q4;  // descriptors of the INT8 and INT4 tiers
  uint32_t e8, e4;  // per-row metadata bytes of an INT8 / INT4 row of this segment
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

// Reduction over aligned groups of gl lanes (gl a power of two, 4 <= gl <=
// LPR, uniform over the wavefront); every lane of each group must be active.
// Quad butterfly and row mirrors as in group_max, chosen by gl.
template <int LPR, bool MAX>
__device__ __forceinline__ uint32_t group_reduce(uint32_t v, int gl) {
  auto op = [](uint32_t a, uint32_t b) { return MAX ? max(a, b) : min(a, b); };
  v = op(v, dpp_mov<0xB1>(v));  // quad_perm [1,0,3,2]
  v = op(v, dpp_mov<0x4E>(v));  // quad_perm [2,3,0,1]
  if constexpr (LPR >= 8) {
    if (gl >= 8) v = op(v, dpp_mov<0x141>(v));  // row_half_mirror
  }
  if constexpr (LPR >= 16) {
    if (gl >= 16) v = op(v, dpp_mov<0x140>(v));  // row_mirror
  }
  if constexpr (LPR >= 32) {
    if (gl >= 32) {
      const LanePair p = lane_pair16(v);  // lanes i and i ^ 16
      v = op(p.lo, p.hi);
    }
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

// Parameters of one quantization group from its reductions: amax (largest
// magnitude bits), kmin / kmax (order keys of the minimum and maximum).
struct GroupParams {
  float scale, r, lo;
  uint32_t s16, lo16;  // binary16 metadata
  bool zero;           // all codes zero (non-finite, zero a or range, binary16 underflow)
};

__device__ __forceinline__ GroupParams group_params(uint32_t amax, uint32_t kmin, uint32_t kmax, int tr, int32_t q) {
  const bool asym = (q & kQuantAsym) != 0, f16 = (q & kQuantFp16) != 0;
  const int Q = tr == kINT8 ? 127 : 7, M = tr == kINT8 ? 255 : 15;
  GroupParams g;
  g.scale = 0.0f;
  g.r = 0.0f;
  g.lo = 0.0f;
  g.s16 = 0;
  g.lo16 = key_to_half(kmin);
  g.zero = false;
  if (amax >= 0x7C00u) {  // the group holds an inf/NaN
    g.scale = __builtin_bit_cast(float, 0x7FC00000u);
    g.lo = g.scale;
    g.s16 = g.lo16 = 0x7E00u;
    g.zero = true;
  } else if (!asym) {
    if (amax == 0u) {
      g.zero = true;
    } else {
      const float a = half_lo(amax);
      g.scale = scale_of(a, static_cast<float>(Q), Q == 127 ? 1.0f / 127.0f : 1.0f / 7.0f);
      if (f16) {
        g.s16 = __builtin_bit_cast(uint16_t, static_cast<_Float16>(g.scale));
        g.scale = half_lo(g.s16);
        g.zero = g.s16 == 0u;
        // RN32(1/s) by reciprocal + one correction: correctly rounded for
        // every positive binary16 s (checked exhaustively in exact arithmetic)
        g.r = g.zero ? 0.0f : recip_scale_of(g.scale, 1.0f);
      } else {
        g.r = recip_scale_of(a, static_cast<float>(Q));
      }
    }
  } else {
    g.lo = half_lo(g.lo16);
    const float range = half_lo(key_to_half(kmax)) - g.lo;
    if (range == 0.0f) {
      g.zero = true;
    } else {
      // RN32(range / M) and RN32(M / range) without a division: correctly
      // rounded for every binary32 range (checked exhaustively)
      const float Mf = static_cast<float>(M);
      g.scale = scale_of(range, Mf, M == 255 ? 1.0f / 255.0f : 1.0f / 15.0f);
      if (f16) {
        g.s16 = __builtin_bit_cast(uint16_t, static_cast<_Float16>(g.scale));
        g.scale = half_lo(g.s16);
        g.zero = g.s16 == 0u;
        g.r = g.zero ? 0.0f : recip_scale_of(g.scale, 1.0f);  // as above
      } else {
        g.r = recip_scale_of_f32(range, Mf);
      }
    }
  }
  return g;
}

// Code of x in a group (as the float-magic integer base + code, clamped).
// clamp = false only where the clamp provably never binds, i.e. with fp32
// metadata: symmetric, r = RN32(Q/a) keeps |RN32(x r)| < Q + 1/2 for every
// |x| <= a (exhaustive over binary16 a); asymmetric, 0 <= RN32(x - lo) <=
// range and RN32(range RN32(M/range)) < M + 1/2 for every binary32 range
// (exhaustive), so the code lies in [0, M].
__device__ __forceinline__ uint32_t group_code(float x, float r, float lo, bool zero, bool asym, int tr,
                                               bool clamp = true) {
  const int Q = tr == kINT8 ? 127 : 7, M = tr == kINT8 ? 255 : 15;
  const int32_t base = 0x4B400000;
  const int32_t cmin = asym ? base : base - Q, cmax = asym ? base + M : base + Q;
  const float y = asym ? (x - lo) * r : x * r;
  int32_t c = __builtin_bit_cast(int32_t, y + 12582912.0f);
  if (clamp) c = min(max(c, cmin), cmax);
  return static_cast<uint32_t>(zero ? base : c);
}

// Writes a group's metadata entry (s, then lo if asymmetric; fp32 or binary16).
__device__ __forceinline__ void store_entry(uint8_t* e, const GroupParams& g, int32_t q) {
  const bool asym = (q & kQuantAsym) != 0;
  if (q & kQuantFp16) {
    reinterpret_cast<uint16_t*>(e)[0] = static_cast<uint16_t>(g.s16);
    if (asym) reinterpret_cast<uint16_t*>(e)[1] = static_cast<uint16_t>(g.lo16);
  } else {
    store_u32_as_halves(e, __builtin_bit_cast(uint32_t, g.scale));
    if (asym) store_u32_as_halves(e + 4, __builtin_bit_cast(uint32_t, g.lo));
  }
}

__device__ __forceinline__ uint32_t entry_bytes(int32_t q) {
  return ((q & kQuantAsym) ? 2u : 1u) * ((q & kQuantFp16) ? 2u : 4u);
}

// Order keys of the two binary16 values of a word at once: h ^ 0x8000, and
// the other 15 bits flipped too when the sign is set (order_key16 per half).
__device__ __forceinline__ u16x2 order_key16x2(uint32_t w) {
  const uint32_t neg = ((w >> 15) & 0x00010001u) * 0x7FFFu;  // 0x7FFF in each negative half
  return __builtin_bit_cast(u16x2, w ^ 0x80008000u ^ neg);
}

// Order-key minimum and maximum of the lane's 8 elements (packed 16-bit
// integer minimum / maximum over the two halves of each word).
__device__ __forceinline__ void lane_key_range(u32x4 x, uint32_t& kmin, uint32_t& kmax) {
  const u16x2 k0 = order_key16x2(x.x), k1 = order_key16x2(x.y), k2 = order_key16x2(x.z), k3 = order_key16x2(x.w);
  const u16x2 lo = __builtin_elementwise_min(__builtin_elementwise_min(k0, k1), __builtin_elementwise_min(k2, k3));
  const u16x2 hi = __builtin_elementwise_max(__builtin_elementwise_max(k0, k1), __builtin_elementwise_max(k2, k3));
  kmin = min(static_cast<uint32_t>(lo.x), static_cast<uint32_t>(lo.y));
  kmax = max(static_cast<uint32_t>(hi.x), static_cast<uint32_t>(hi.y));
}

// Quantizes the lane's 8 elements of a row at tier tr under descriptor q and
// writes the group's metadata at meta (the row's metadata) from the group's
// first lane.  All lanes of the wavefront call it (reductions).
template <int LPR>
__device__ __forceinline__ LaneCodes quantize_lane_var(u32x4 x, int tr, int32_t q, int lane, uint8_t* meta,
                                                       bool write_meta) {
  constexpr int D = LPR * 8;
  const int gl = var_group_lanes(q, D);
  const bool asym = (q & kQuantAsym) != 0;  // uniform over the row's lanes
  const uint32_t lane_amax = absmax_bits8(x);
  uint32_t amax, kmin = 0xFFFFu, kmax = 0u;
  if (asym) {
    // minimum and maximum only; an inf or NaN sorts outside the finite keys
    // [0x0400, 0xFBFF], which is all group_params needs of amax here
    lane_key_range(x, kmin, kmax);
    kmin = group_reduce<LPR, false>(kmin, gl);
    kmax = group_reduce<LPR, true>(kmax, gl);
    amax = (kmin < 0x0400u || kmax > 0xFBFFu) ? 0x7C00u : 0u;
  } else {
    amax = group_reduce<LPR, true>(lane_amax, gl);
  }
  const GroupParams g = group_params(amax, kmin, kmax, tr, q);

  LaneCodes out;
  {
    // some group of the row holds an inf/NaN: one ballot over the wavefront,
    // masked to the row's aligned lanes
    const uint64_t nf = __ballot(lane_amax >= 0x7C00u);
    const int first = (threadIdx.x & 63) & ~(LPR - 1);
    const uint64_t row_lanes = (LPR >= 64 ? ~0ull : ((1ull << LPR) - 1ull)) << first;
    out.nonfinite = (nf & row_lanes) != 0ull;
  }
  out.scale = g.scale;
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  if (!(q & kQuantFp16)) {  // uniform per row: with fp32 metadata the clamp cannot bind
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out.c[2 * i] = group_code(half_lo(w[i]), g.r, g.lo, g.zero, asym, tr, false);
      out.c[2 * i + 1] = group_code(half_hi(w[i]), g.r, g.lo, g.zero, asym, tr, false);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out.c[2 * i] = group_code(half_lo(w[i]), g.r, g.lo, g.zero, asym, tr);
      out.c[2 * i + 1] = group_code(half_hi(w[i]), g.r, g.lo, g.zero, asym, tr);
    }
  }
  if (write_meta && (lane % gl) == 0) store_entry(meta + (lane / gl) * entry_bytes(q), g, q);
  return out;
}

// Per-channel K parameters of one chunk (descriptor bit SKV_QUANT_CHANNEL):
// channel c of tier t uses r[t][c], lo[t][c], zero[t][c] (t = 0 INT8, 1 INT4).
template <int D>
struct ChanLds {
  uint32_t amax[2][D], kmin[2][D], kmax[2][D];
  float r[2][D], lo[2][D];
  uint32_t zero[2][D];
  uint32_t rows[2];
};

// Row-width units and metadata bytes of one token (scan value of the variant
// layout: units | metadata bytes << 12).
__device__ __forceinline__ uint32_t var_scan_value(int tr, const VarCfg& v) {
  if (tr == kAbsent) return 0u;
  const uint32_t eb = tr == kINT8 ? v.e8 : tr == kINT4 ? v.e4 : 0u;
  return tier_units(tr) | (eb << 12);
}

// chunk_layout for the variant layout: s.q receives the byte offset of the
// row's metadata inside its segment's metadata.  cidx_entry: {units, quantized
// rows, V-side metadata bytes, K-side metadata bytes (0 unless a tier is
// per-channel)} of the chunk; meta_word selects the side (2 or 3).  Contains
// __syncthreads().
template <int D>
__device__ __forceinline__ void chunk_layout_var(ChunkLds& s, int tr, const uint32_t* cidx_entry, int meta_word,
                                                 const VarCfg& v) {
  uint32_t total;
  const uint32_t ex = block_exclusive_scan_256(var_scan_value(tr, v), s.scan, &total);
  s.tier[threadIdx.x] = static_cast<uint8_t>(tr);
  s.off[threadIdx.x] = (cidx_entry[0] + (ex & 0xFFFu)) * static_cast<uint32_t>(D / 2);
  s.q[threadIdx.x] = cidx_entry[meta_word] + (ex >> 12);
}

// Per-thread partial reductions of the per-channel tiers (t = 0 INT8, 1 INT4)
// over the rows the thread holds, for its 8 channels: symmetric tiers keep the
// largest magnitude bits in a, asymmetric tiers the order-key minimum in a and
// maximum in b.
struct ChanAcc {
  u16x2 a[2][4], b[2][4];  // channels 2i (low half) and 2i + 1 (high half) of the lane
  uint32_t rows[2];
};

__device__ __forceinline__ void chan_acc_init(ChanAcc& acc, const VarCfg& v) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const bool asym = ((t == 0 ? v.q8 : v.q4) & kQuantAsym) != 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc.a[t][e] = asym ? u16x2{0xFFFFu, 0xFFFFu} : u16x2{0u, 0u};
      acc.b[t][e] = u16x2{0u, 0u};
    }
    acc.rows[t] = 0u;
  }
}

// Two channels per packed 16-bit integer minimum / maximum.
template <int T>
__device__ __forceinline__ void chan_acc_row_t(ChanAcc& acc, u32x4 x, bool asym) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  ++acc.rows[T];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (asym) {
      const u16x2 k = order_key16x2(w[e]);
      acc.a[T][e] = __builtin_elementwise_min(acc.a[T][e], k);
      acc.b[T][e] = __builtin_elementwise_max(acc.b[T][e], k);
    } else {
      acc.a[T][e] = __builtin_elementwise_max(acc.a[T][e], __builtin_bit_cast(u16x2, w[e] & 0x7FFF7FFFu));
    }
  }
}

// Adds the row x of tier tr to acc if tr is a per-channel tier.
__device__ __forceinline__ void chan_acc_row(ChanAcc& acc, u32x4 x, int tr, const VarCfg& v) {
  if (tr == kINT8 && (v.q8 & kQuantChannel)) chan_acc_row_t<0>(acc, x, (v.q8 & kQuantAsym) != 0);
  else if (tr == kINT4 && (v.q4 & kQuantChannel)) chan_acc_row_t<1>(acc, x, (v.q4 & kQuantAsym) != 0);
}

// Clears the shared reduction arrays (before any chan_combine; the caller
// synchronizes).
template <int D>
__device__ __forceinline__ void chan_lds_init(ChanLds<D>& c) {
  for (int i = threadIdx.x; i < 2 * D; i += kRowThreads) {
    (&c.amax[0][0])[i] = 0u;
    (&c.kmin[0][0])[i] = 0xFFFFu;
    (&c.kmax[0][0])[i] = 0u;
  }
  if (threadIdx.x < 2) c.rows[threadIdx.x] = 0u;
}

// Combines every thread's partials into c with shared-memory integer max/min
// atomics (order-independent, so deterministic), then derives each channel's
// parameters and writes its entry (INT8 at blk8, INT4 at blk4; zeros for a
// tier without rows in the chunk).  Contains __syncthreads().
template <int D>
__device__ __forceinline__ void chan_finish(ChanLds<D>& c, const ChanAcc& acc, int lane, const VarCfg& v,
                                            uint8_t* blk8, uint8_t* blk4) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int32_t q = t == 0 ? v.q8 : v.q4;
    if (!(q & kQuantChannel)) continue;
    if (q & kQuantAsym) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        atomicMin(&c.kmin[t][lane * 8 + e], static_cast<uint32_t>(acc.a[t][e / 2][e & 1]));
        atomicMax(&c.kmax[t][lane * 8 + e], static_cast<uint32_t>(acc.b[t][e / 2][e & 1]));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) atomicMax(&c.amax[t][lane * 8 + e], static_cast<uint32_t>(acc.a[t][e / 2][e & 1]));
    }
    if (lane == 0 && acc.rows[t]) atomicAdd(&c.rows[t], acc.rows[t]);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 2 * D; i += kRowThreads) {
    const int t = i / D, ch = i % D;
    const int32_t q = t == 0 ? v.q8 : v.q4;
    if (!(q & kQuantChannel)) continue;
    uint32_t amax = c.amax[t][ch];
    const uint32_t kmin = c.kmin[t][ch], kmax = c.kmax[t][ch];
    // asymmetric groups track order keys only: an inf/NaN is a key beyond +-inf's
    if (q & kQuantAsym) amax = (kmax >= 0xFC00u || kmin <= 0x03FFu) ? 0x7C00u : 0u;
    GroupParams g = group_params(amax, kmin, kmax, t == 0 ? kINT8 : kINT4, q);
    if (c.rows[t] == 0u) {  // no row of the tier in this chunk: zero entry
      g.scale = g.r = g.lo = 0.0f;
      g.s16 = g.lo16 = 0u;
      g.zero = true;
    }
    c.r[t][ch] = g.r;
    c.lo[t][ch] = g.lo;
    c.zero[t][ch] = g.zero ? 1u : 0u;
    store_entry((t == 0 ? blk8 : blk4) + ch * entry_bytes(q), g, q);
  }
  __syncthreads();
}

// Per-channel parameters of a chunk whose rows are re-read from src (the
// rows of a thread do not fit its registers at d = 256).  Contains
// __syncthreads().
template <int D>
__device__ __forceinline__ void channel_params(const ChunkLds& s, ChanLds<D>& c, const uint16_t* __restrict__ src,
                                               int t0, const VarCfg& v, uint8_t* blk8, uint8_t* blk4) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
  chan_lds_init<D>(c);
  ChanAcc acc;
  chan_acc_init(acc, v);
#pragma unroll 4
  for (int it = 0; it < ITERS; ++it) {
    const int row = it * RPI + rsub;
    const int tr = s.tier[row];  // rows at or beyond n are DROP
    const bool take = (tr == kINT8 && (v.q8 & kQuantChannel)) || (tr == kINT4 && (v.q4 & kQuantChannel));
    if (!take) continue;
    chan_acc_row(acc, *reinterpret_cast<const u32x4*>(src + static_cast<size_t>(t0 + row) * D + lane * 8), tr, v);
  }
  __syncthreads();  // shared arrays cleared before any atomic
  chan_finish<D>(c, acc, lane, v, blk8, blk4);
}

// Quantizes and stores one row held by this lane (x: its 8 elements).  CHAN:
// rows of a per-channel tier take their codes from c and write no per-row
// metadata.  Every lane of the wavefront calls it (reductions).
template <int D, bool NT, bool CHAN>
__device__ __forceinline__ void pack_row_var(const ChunkLds& s, const ChanLds<D>* c, u32x4 x, int row,
                                             uint8_t* __restrict__ dst, uint8_t* __restrict__ meta,
                                             uint32_t* nonfinite, const VarCfg& v, int lane) {
  constexpr int LPR = D / 8;
  const int tr = s.tier[row];
  const bool quant = tr == kINT8 || tr == kINT4;
  const int32_t q = tr == kINT8 ? v.q8 : v.q4;
  const bool chan = CHAN && quant && (q & kQuantChannel) != 0;
  LaneCodes qc;
  // a row's lanes are one aligned group, so this branch is uniform per row and
  // the cross-lane reductions below stay inside active lanes
  if (chan) {
    const int t = tr == kINT8 ? 0 : 1;
    const bool asym = (q & kQuantAsym) != 0;
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    qc.nonfinite = group_max<LPR>(absmax_bits8(x)) >= 0x7C00u;
    qc.scale = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ch = lane * 8 + e;
      const float xv = (e & 1) ? half_hi(w[e / 2]) : half_lo(w[e / 2]);
      qc.c[e] = group_code(xv, c->r[t][ch], c->lo[t][ch], c->zero[t][ch] != 0u, asym, tr);
    }
  } else {
    qc = quantize_lane_var<LPR>(x, tr, q, lane, meta + s.q[row], quant);
  }
  if (tr == kFP16) {
    store16<NT>(dst + s.off[row] + lane * 16, x);
  } else if (quant) {
    if (qc.nonfinite && lane == 0) atomicAdd(nonfinite, 1u);
    uint8_t* out_row = dst + s.off[row];
    if (tr == kINT8) store8<NT>(out_row + lane * 8, pack_int8(qc));
    else store4<NT>(out_row + lane * 4, pack_int4(qc));
  }
}

// Packs one chunk of a segment under the variant descriptors.  CHAN: a K
// segment with a per-channel tier whose parameters are already in c.
template <int D, int ROWS_IN_FLIGHT, bool NT, bool CHAN>
__device__ __forceinline__ void pack_chunk_var(const ChunkLds& s, const ChanLds<D>* c, const uint16_t* __restrict__ src,
                                               uint8_t* __restrict__ dst, uint8_t* __restrict__ meta,
                                               uint32_t* nonfinite, int t0, int n, const VarCfg& v) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
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
    for (int u = 0; u < U; ++u)
      pack_row_var<D, NT, CHAN>(s, c, x[u], (it + u) * RPI + rsub, dst, meta, nonfinite, v, lane);
  }
}

// Quantizes and stores a row of a per-channel tier (tr) with its chunk's
// channel parameters in c: the lane's 8 channels are contiguous, so their
// scales and minimums are two 16-byte shared-memory reads each.  zero_bits:
// bit 8 t + e marks channel lane * 8 + e of tier t as all-zero codes.  Every
// lane of the row's group calls it.
template <int D, bool NT>
__device__ __forceinline__ void pack_row_chan(const ChunkLds& s, const ChanLds<D>& c, uint32_t zero_bits, u32x4 x,
                                              int row, int tr, bool asym, uint8_t* __restrict__ dst,
                                              uint32_t* nonfinite, int lane) {
  constexpr int LPR = D / 8;
  const int t = tr == kINT8 ? 0 : 1;
  const f32x4* rp = reinterpret_cast<const f32x4*>(&c.r[t][lane * 8]);
  const f32x4* lp = reinterpret_cast<const f32x4*>(&c.lo[t][lane * 8]);
  const f32x4 r0 = rp[0], r1 = rp[1], l0 = lp[0], l1 = lp[1];
  const float rs[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
  const float ls[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  LaneCodes qc;
  qc.nonfinite = group_max<LPR>(absmax_bits8(x)) >= 0x7C00u;
  qc.scale = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float xv = (e & 1) ? half_hi(w[e / 2]) : half_lo(w[e / 2]);
    qc.c[e] = group_code(xv, rs[e], ls[e], ((zero_bits >> (8 * t + e)) & 1u) != 0u, asym, tr);
  }
  if (qc.nonfinite && lane == 0) atomicAdd(nonfinite, 1u);
  uint8_t* out_row = dst + s.off[row];
  if (tr == kINT8) store8<NT>(out_row + lane * 8, pack_int8(qc));
  else store4<NT>(out_row + lane * 4, pack_int4(qc));
}

// K segment with a per-channel tier, d <= 128: the thread's rows of the chunk
// (at most 16) are loaded once into registers, reduced per channel, and then
// quantized from the same registers.  Contains __syncthreads().
template <int D, bool NT>
__device__ __forceinline__ void pack_chunk_chan(const ChunkLds& s, ChanLds<D>& c, const uint16_t* __restrict__ src,
                                                uint8_t* __restrict__ dst, uint8_t* __restrict__ meta,
                                                uint32_t* nonfinite, int t0, int n, const VarCfg& v, uint8_t* blk8,
                                                uint8_t* blk4) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  static_assert(ITERS <= 16, "rows of a thread held in registers");
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
  u32x4 x[ITERS];
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int row = it * RPI + rsub;
    const int t = t0 + row;
    x[it] = u32x4{0u, 0u, 0u, 0u};
    if (t < n && s.tier[row] != kDROP) x[it] = ld_nt16(src + static_cast<size_t>(t) * D + lane * 8);
  }
  chan_lds_init<D>(c);
  ChanAcc acc;
  chan_acc_init(acc, v);
#pragma unroll
  for (int it = 0; it < ITERS; ++it) chan_acc_row(acc, x[it], s.tier[it * RPI + rsub], v);
  __syncthreads();  // shared arrays cleared before any atomic
  chan_finish<D>(c, acc, lane, v, blk8, blk4);
  // the thread's 8 channels are the same in all its rows: their all-zero
  // flags of both tiers, as bits
  uint32_t zero_bits = 0u;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) zero_bits |= (c.zero[t][lane * 8 + e] != 0u ? 1u : 0u) << (8 * t + e);
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int row = it * RPI + rsub;
    const int tr = s.tier[row];
    const int32_t q = tr == kINT8 ? v.q8 : v.q4;
    if ((tr == kINT8 || tr == kINT4) && (q & kQuantChannel))  // uniform per row
      pack_row_chan<D, NT>(s, c, zero_bits, x[it], row, tr, (q & kQuantAsym) != 0, dst, nonfinite, lane);
    else
      pack_row_var<D, NT, true>(s, &c, x[it], row, dst, meta, nonfinite, v, lane);
  }
}

// Two binary32 values rounded to binary16 and packed low|high, any NaN as the
// canonical 0x7E00 (a payload whose metadata was corrupted can make code * s
// + lo a NaN of any sign and payload; the decoded cache then still matches a
// reference that writes every NaN as 0x7E00).
__device__ __forceinline__ uint32_t pack_half2_canon(float a, float b) {
  const uint32_t ha = __builtin_isnan(a) ? 0x7E00u : __builtin_bit_cast(uint16_t, static_cast<_Float16>(a));
  const uint32_t hb = __builtin_isnan(b) ? 0x7E00u : __builtin_bit_cast(uint16_t, static_cast<_Float16>(b));
  return ha | (hb << 16);
}

// The scale and minimum (0 if symmetric) of the lane's group of a quantized
// row under descriptor q, read from the row's metadata entry.
// A lane's group metadata as stored, kept as bits so that its loads stay in
// flight until the row is decoded: binary16 entries in a (the scale in the
// low half, an asymmetric group's minimum in the high half), binary32 entries
// in a (scale) and b (minimum); unused bits are zero.
struct LaneMeta {
  uint32_t a, b;
};
// Byte offset of a lane's group entry inside a row's metadata.
template <int LPR>
__device__ __forceinline__ uint32_t lane_meta_offset(int32_t q, int lane) {
  constexpr int D = LPR * 8;
  return static_cast<uint32_t>(lane / var_group_lanes(q, D)) * entry_bytes(q);
}
// 32 bits at a 2-byte aligned address (one load; global memory takes
// unaligned dword loads).
typedef uint32_t u32_align2 __attribute__((aligned(2)));
__device__ __forceinline__ uint32_t load_u32_align2(const uint8_t* p) {
  return *reinterpret_cast<const u32_align2*>(p);
}
// e: the lane's entry (row metadata + lane_meta_offset)
__device__ __forceinline__ LaneMeta load_lane_meta(int32_t q, const uint8_t* e) {
  const bool asym = (q & kQuantAsym) != 0;
  LaneMeta m{0u, 0u};
  if (q & kQuantFp16) {
    m.a = asym ? load_u32_align2(e) : static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(e)[0]);
  } else {
    m.a = load_u32_align2(e);
    if (asym) m.b = load_u32_align2(e + 4);
  }
  return m;
}

// The lane's 8 outputs of a quantized row under descriptor q, with its
// group's metadata m.
__device__ __forceinline__ u32x4 decode_lane_var(int tr, int32_t q, u32x4 raw, LaneMeta m) {
  const bool asym = (q & kQuantAsym) != 0;
  const bool f16 = (q & kQuantFp16) != 0;
  const float s = f16 ? half_lo(m.a) : __builtin_bit_cast(float, m.a);
  const float lo = f16 ? half_hi(m.a) : __builtin_bit_cast(float, m.b);
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
    f[i] = static_cast<float>(code) * s;  // no fused conversion here (a directed test checks)
    if (asym) f[i] = f[i] + lo;
  }
  // with a finite scale and minimum, code * s + lo is finite or an infinity:
  // only non-finite metadata can make a NaN to canonicalize
  if (__builtin_isfinite(s) && __builtin_isfinite(lo))
    return u32x4{pack_half2(f[0], f[1]), pack_half2(f[2], f[3]), pack_half2(f[4], f[5]), pack_half2(f[6], f[7])};
  return u32x4{pack_half2_canon(f[0], f[1]), pack_half2_canon(f[2], f[3]), pack_half2_canon(f[4], f[5]),
               pack_half2_canon(f[6], f[7])};
}

// Per-channel K parameters of one chunk on the decode side: scale and
// minimum of channel c of tier t (0 INT8, 1 INT4).
template <int D>
struct ChanDecLds {
  float s[2][D], lo[2][D];
};

// Loads the chunk's per-channel entries (INT8 at blk8, INT4 at blk4) into c;
// returns, to every thread, whether all of them are finite (then no decoded
// value can be a NaN).  Contains a block barrier.
template <int D>
__device__ __forceinline__ bool load_channel_params(ChanDecLds<D>& c, const uint8_t* blk8, const uint8_t* blk4,
                                                    const VarCfg& v) {
  int bad = 0;
  for (int i = threadIdx.x; i < 2 * D; i += kRowThreads) {
    const int t = i / D, ch = i % D;
    const int32_t q = t == 0 ? v.q8 : v.q4;
    float sc = 0.0f, lo = 0.0f;
    if (q & kQuantChannel) {
      const uint8_t* e = (t == 0 ? blk8 : blk4) + ch * entry_bytes(q);
      const bool asym = (q & kQuantAsym) != 0;
      if (q & kQuantFp16) {
        sc = half_lo(reinterpret_cast<const uint16_t*>(e)[0]);
        if (asym) lo = half_lo(reinterpret_cast<const uint16_t*>(e)[1]);
      } else {
        sc = __builtin_bit_cast(float, load_u32_from_halves(e));
        if (asym) lo = __builtin_bit_cast(float, load_u32_from_halves(e + 4));
      }
    }
    c.s[t][ch] = sc;
    c.lo[t][ch] = lo;
    bad |= !(__builtin_isfinite(sc) && __builtin_isfinite(lo));
  }
  return __syncthreads_or(bad) == 0;
}

// The lane's 8 outputs of a per-channel K row: element e of channel
// lane * 8 + e decoded with that channel's scale and minimum (NaN scale:
// 0x7E00).
template <int LPR>
__device__ __forceinline__ u32x4 decode_lane_chan(int tr, int32_t q, u32x4 raw, const float* sc, const float* lo,
                                                  int lane, bool finite) {
  const bool asym = (q & kQuantAsym) != 0;
  uint32_t h[8];
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
    const float s = sc[lane * 8 + i];
    float f = static_cast<float>(code) * s;
    if (asym) f = f + lo[lane * 8 + i];
    const uint32_t hv = __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
    h[i] = (!finite && __builtin_isnan(f)) ? 0x7E00u : hv;
  }
  return u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
}

template <int D, int ROWS_IN_FLIGHT, bool NT, bool CHAN>
__device__ __forceinline__ void unpack_chunk_var(const ChunkLds& s, const ChanDecLds<D>* c, bool chan_finite,
                                                 const uint8_t* __restrict__ src, const uint8_t* __restrict__ meta,
                                                 uint16_t* __restrict__ cache, int H, const VarCfg& v) {
  constexpr int LPR = D / 8;
  constexpr int RPI = kRowThreads / LPR;
  constexpr int ITERS = kChunkTokens / RPI;
  constexpr int U = ITERS < ROWS_IN_FLIGHT ? ITERS : ROWS_IN_FLIGHT;
  static_assert(ITERS % U == 0, "rows in flight must divide a thread's rows of the chunk");
  const int lane = threadIdx.x % LPR;
  const int rsub = threadIdx.x / LPR;
  const uint32_t moff8 = lane_meta_offset<LPR>(v.q8, lane), moff4 = lane_meta_offset<LPR>(v.q4, lane);
#pragma unroll 1
  for (int it = 0; it < ITERS; it += U) {
    u32x4 raw[U];
    LaneMeta mt[U];  // per-row metadata, loaded with the codes
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s.tier[r];
      const uint8_t* row = src + s.off[r];
      raw[u] = u32x4{0u, 0u, 0u, 0u};
      mt[u] = LaneMeta{0u, 0u};
      if (tr == kFP16) {
        raw[u] = ld_nt16(row + lane * 16);
      } else if (tr == kINT8) {
        const u32x2 cc = ld_nt8(row + lane * 8);
        raw[u].x = cc.x;
        raw[u].y = cc.y;
      } else if (tr == kINT4) {
        raw[u].x = ld_nt4(row + lane * 4);
      }
      if (tr == kINT8 || tr == kINT4) {
        const int32_t q = tr == kINT8 ? v.q8 : v.q4;
        if (!(CHAN && (q & kQuantChannel))) mt[u] = load_lane_meta(q, meta + s.q[r] + (tr == kINT8 ? moff8 : moff4));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = (it + u) * RPI + rsub;
      const int tr = s.tier[r];
      if (tr == kAbsent) continue;
      u32x4 o = raw[u];  // FP16 verbatim, DROP zeros
      if (tr == kINT8 || tr == kINT4) {
        const int32_t q = tr == kINT8 ? v.q8 : v.q4;
        if (CHAN && (q & kQuantChannel)) {
          const int t = tr == kINT8 ? 0 : 1;
          o = decode_lane_chan<LPR>(tr, q, raw[u], c->s[t], c->lo[t], lane, chan_finite);
        } else {
          o = decode_lane_var(tr, q, raw[u], mt[u]);
        }
      }
      store16<NT>(cache + static_cast<size_t>(s.pos[r]) * H * D + lane * 8, o);
    }
  }
}

}  // namespace skv
