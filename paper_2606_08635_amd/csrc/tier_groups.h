// Tier-map bookkeeping shared by pack (which writes the map and the chunk
// index) and unpack (which checks them): one thread reads the codes of a
// group of 16 consecutive tokens; the 16 groups of a 256-token chunk sit in
// 16 consecutive lanes, so chunk sums are a 16-lane reduction.
#pragma once

#include "device_util.h"
#include "skv_internal.h"

namespace skv {

constexpr int kGroupTokens = 16;
constexpr int kGroupsPerChunk = kChunkTokens / kGroupTokens;  // 16

struct TierGroup {
  uint32_t units;   // sum of row widths in units of d/2 bytes
  uint32_t quant;   // number of INT8/INT4 rows
  uint32_t map2;    // the 16 codes, 2 bits each (token 16g+j at bits 2j..2j+1)
  uint32_t cnt[4];  // tokens per tier
  bool bad;         // a code outside 0..3 (byte input only)
};

__device__ __forceinline__ void tally(TierGroup& gi, uint32_t code, int j) {
  gi.map2 |= (code & 3u) << (2 * j);
  if (code > 3u) {
    gi.bad = true;
    return;
  }
  gi.cnt[code]++;
  gi.units += tier_units(static_cast<int>(code));
  gi.quant += tier_quant(static_cast<int>(code));
}

__device__ __forceinline__ TierGroup empty_group() {
  TierGroup gi;
  gi.units = gi.quant = gi.map2 = 0;
  gi.cnt[0] = gi.cnt[1] = gi.cnt[2] = gi.cnt[3] = 0;
  gi.bad = false;
  return gi;
}

// Codes from a uint8[n] tier array (16-byte aligned).
__device__ __forceinline__ TierGroup group_from_bytes(const uint8_t* __restrict__ tier, int n, int g) {
  TierGroup gi = empty_group();
  const int t0 = g * kGroupTokens;
  if (t0 + kGroupTokens <= n) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(tier + t0);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int j = 0; j < 16; ++j) tally(gi, (ws[j >> 2] >> (8 * (j & 3))) & 0xFFu, j);
  } else {
    for (int j = 0; j < kGroupTokens && t0 + j < n; ++j) tally(gi, tier[t0 + j], j);
  }
  return gi;
}

// Codes from the payload's 2-bit tier map; codes of tokens >= n are ignored.
__device__ __forceinline__ TierGroup group_from_map(const uint8_t* __restrict__ map, int n, int g) {
  TierGroup gi = empty_group();
  const int t0 = g * kGroupTokens;
  const uint32_t w = *reinterpret_cast<const uint32_t*>(map + 4 * g);
#pragma unroll
  for (int j = 0; j < kGroupTokens; ++j)
    if (t0 + j < n) tally(gi, (w >> (2 * j)) & 3u, j);
  return gi;
}

// Sum over aligned 16-lane groups; every lane gets its group's sum.
__device__ __forceinline__ uint32_t sum16(uint32_t v) {
  v += static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 1));
  v += static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 2));
  v += static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 4));
  v += static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 8));
  return v;
}

// Exclusive prefix sum of one 64-bit value per thread over a 1024-thread
// block.  `scratch` holds at least 16 words of shared memory.  Every thread
// must call it; contains __syncthreads().
__device__ __forceinline__ uint64_t block_exclusive_scan_1024(uint64_t x, uint64_t* scratch) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  uint64_t base = 0;
  for (int w = 0; w < wave; ++w) base += scratch[w];
  __syncthreads();
  return base + inc - x;
}

}  // namespace skv
