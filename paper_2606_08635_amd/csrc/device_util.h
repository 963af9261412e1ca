// Device-side helpers for gfx950 (CDNA4, 64-lane wavefronts).
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace skv {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

enum : int { kFP16 = 0, kINT8 = 1, kINT4 = 2, kDROP = 3 };

// Row width in units of d/2 bytes and "is quantized" flag of each tier.
__device__ __forceinline__ uint32_t tier_units(int tr) {
  return tr == kFP16 ? 4u : tr == kINT8 ? 2u : tr == kINT4 ? 1u : 0u;
}
__device__ __forceinline__ uint32_t tier_quant(int tr) { return (tr == kINT8 || tr == kINT4) ? 1u : 0u; }

// Streaming (non-temporal) 16/8/4-byte global accesses.
__device__ __forceinline__ u32x4 ld_nt16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x2 ld_nt8(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
__device__ __forceinline__ uint32_t ld_nt4(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
}
__device__ __forceinline__ void st_nt16(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}
__device__ __forceinline__ void st_nt8(void* p, u32x2 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x2*>(p));
}
__device__ __forceinline__ void st_nt4(void* p, uint32_t v) {
  __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(p));
}

// Stores that are streaming (non-temporal) or ordinary, chosen at build time.
template <bool NT>
__device__ __forceinline__ void store16(void* p, u32x4 v) {
  if constexpr (NT) st_nt16(p, v); else *reinterpret_cast<u32x4*>(p) = v;
}
template <bool NT>
__device__ __forceinline__ void store8(void* p, u32x2 v) {
  if constexpr (NT) st_nt8(p, v); else *reinterpret_cast<u32x2*>(p) = v;
}
template <bool NT>
__device__ __forceinline__ void store4(void* p, uint32_t v) {
  if constexpr (NT) st_nt4(p, v); else *reinterpret_cast<uint32_t*>(p) = v;
}

// DPP lane move inside 16-lane rows (row_mask/bank_mask all set).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xF, 0xF, true));
}

// The values of lanes i and i ^ 16 (lane_pair16) or i and i ^ 32
// (lane_pair32), the lower lane's as lo, in both lanes: gfx950's
// v_permlane16_swap / v_permlane32_swap, one vector instruction each instead
// of a shuffle through the LDS unit and its address arithmetic.  The lanes
// exchanged stay inside aligned groups of 32 (lane_pair16) or the wave
// (lane_pair32), and every lane of such a group in use must be active.
struct LanePair {
  uint32_t lo, hi;
};
__device__ __forceinline__ LanePair lane_pair16(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return LanePair{r[0], r[1]};
}
__device__ __forceinline__ LanePair lane_pair32(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return LanePair{r[0], r[1]};
}

// Maximum over aligned groups of G consecutive lanes (G = 4, 8, 16 or 32);
// every lane of a group receives the group's maximum.  Must be called with
// every lane of each group active.
template <int G>
__device__ __forceinline__ uint32_t group_max(uint32_t v) {
  static_assert(G == 4 || G == 8 || G == 16 || G == 32, "group size");
  if constexpr (G == 32) {
    const LanePair p = lane_pair16(v);  // lanes i and i ^ 16
    v = max(p.lo, p.hi);
  }
  if constexpr (G >= 16) v = max(v, dpp_mov<0x140>(v));  // row_mirror: lane i <-> 15-i
  if constexpr (G >= 8) v = max(v, dpp_mov<0x141>(v));   // row_half_mirror: i <-> 7-i
  v = max(v, dpp_mov<0xB1>(v));                          // quad_perm [1,0,3,2]
  v = max(v, dpp_mov<0x4E>(v));                          // quad_perm [2,3,0,1]
  return v;
}

// Largest |x| of 8 binary16 values as a magnitude bit pattern (bits & 0x7FFF).
// For finite values the order of magnitude patterns is the order of |x|; any
// pattern >= 0x7C00 means an infinity or NaN is present.
__device__ __forceinline__ uint32_t absmax_bits8(u32x4 x) {
  const u16x2 m0 = __builtin_bit_cast(u16x2, x.x & 0x7FFF7FFFu);
  const u16x2 m1 = __builtin_bit_cast(u16x2, x.y & 0x7FFF7FFFu);
  const u16x2 m2 = __builtin_bit_cast(u16x2, x.z & 0x7FFF7FFFu);
  const u16x2 m3 = __builtin_bit_cast(u16x2, x.w & 0x7FFF7FFFu);
  const u16x2 m = __builtin_elementwise_max(__builtin_elementwise_max(m0, m1),
                                            __builtin_elementwise_max(m2, m3));
  return max(static_cast<uint32_t>(m.x), static_cast<uint32_t>(m.y));
}

__device__ __forceinline__ float half_lo(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xFFFFu)));
}
__device__ __forceinline__ float half_hi(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}
// Two binary32 values rounded (nearest-even) to binary16 and packed low|high.
__device__ __forceinline__ uint32_t pack_half2(float lo, float hi) {
  const uint16_t a = __builtin_bit_cast(uint16_t, static_cast<_Float16>(lo));
  const uint16_t b = __builtin_bit_cast(uint16_t, static_cast<_Float16>(hi));
  return static_cast<uint32_t>(a) | (static_cast<uint32_t>(b) << 16);
}

// Exclusive prefix sum of one 32-bit value per thread over a 256-thread
// block (4 wavefronts).  `scratch` holds at least 4 words of shared memory.
// Returns the exclusive sum; *total receives the block total.  Contains
// __syncthreads(); every thread of the block must call it.
__device__ __forceinline__ uint32_t block_exclusive_scan_256(uint32_t x, uint32_t* scratch,
                                                             uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = static_cast<uint32_t>(__shfl_up(static_cast<int>(inc), o));
    if (lane >= o) inc += y;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  uint32_t base = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) base += (w < wave) ? scratch[w] : 0u;
  *total = scratch[0] + scratch[1] + scratch[2] + scratch[3];
  __syncthreads();  // scratch may be reused after return
  return base + inc - x;
}

}  // namespace skv
